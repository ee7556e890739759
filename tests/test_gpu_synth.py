"""The device generator writes the same bytes as the host generator (GPU)."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import say, torch_to_bits

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name,over,layers", [
    ("C1", {}, (0,)),
    ("C2", dict(n_layers=3), (1,)),
    ("C3", dict(n_layers=2, n_q_heads=4, n_kv_heads=4, T=2048, window=409), (0, 1)),
    ("C5", dict(n_layers=2, n_q_heads=8, n_kv_heads=2, T=8192, window=819, hh_count=16, hh_hi=8192 - 32), (1,)),
    ("X1", dict(n_layers=2, batch=2, n_q_heads=4, n_kv_heads=4), (1,)),
])
def test_device_generator_matches_host(name, over, layers):
    w = synth.get(name).with_(**over)
    say(f"[synth] {name} {over}")
    sp = synth.spec(w)
    rope_h = synth.rope_table(w.T, w.head_dim, w.rope_base) if w.rope else None
    rope_d = torch.from_numpy(rope_h).cuda() if w.rope else None
    qd = synth.qwin_dev(sp, w.dtype, 0, w.n_layers, rope_d)
    kd, vd = synth.kv_dev(sp, w.dtype, 0, w.n_layers, qd, rope_d)
    q_dec = synth.dq_dev(sp, w.dtype, 3)
    torch.cuda.synchronize()
    for l in layers:
        qh, kh, vh = synth.prefill_host(w, l)
        np.testing.assert_array_equal(torch_to_bits(qd[l], w.dtype), qh)
        np.testing.assert_array_equal(torch_to_bits(kd[l], w.dtype), kh)
        np.testing.assert_array_equal(torch_to_bits(vd[l], w.dtype), vh)
    np.testing.assert_array_equal(torch_to_bits(q_dec, w.dtype), synth.dq_host(sp, 3, w.dtype))
