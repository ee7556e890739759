"""GPU selection against the oracle when many scores are exactly equal.

Representatives and queries hold small integers, so every similarity score is an exact integer in
fp64 on both sides and large groups of clusters tie exactly; ties are broken by the lower index on
both sides, so the selections must be identical (no tie allowance). Covers the
workgroup-per-head and wave-per-head kernels, sets spanning several ranking slots per lane, and
the degenerate all-equal case (zero query).
"""
import zlib

import numpy as np
import pytest
import torch

import oracle
from gpu_util import bits_to_torch, say, torch_to_bits

pytestmark = pytest.mark.gpu


def _int_inputs(rng, L, B, Hq, Hkv, d, C, S, dtype, R, zero_q):
    rows = (R, d) if R > 1 else (d,)
    cent = rng.integers(-1, 2, size=(L, B, Hkv, C) + rows).astype(np.float32)
    scent = rng.integers(-1, 2, size=(L, B, Hkv, S) + rows).astype(np.float32)
    qv = np.zeros((L, B, Hq, d)) if zero_q else rng.integers(-2, 3, size=(L, B, Hq, d))
    td = {"bf16": torch.bfloat16, "fp16": torch.float16, "fp32": torch.float32}[dtype]
    q = torch_to_bits(torch.from_numpy(qv).to(td), dtype)
    return q, cent, scent


CASES = [
    # name, L, B, Hq, Hkv, d, dtype, s, f, C, k_super, k_clusters, sim, zero_q
    ("block-bf16-S128-NC512", 2, 1, 32, 8, 128, "bf16", 16, 8, 1024, 64, 40, "linear", False),
    ("block-zero-query", 2, 1, 32, 8, 128, "bf16", 16, 8, 1024, 64, 40, "linear", True),
    ("block-maxprod", 2, 1, 16, 4, 64, "fp16", 16, 4, 300, 50, 33, "maxprod", False),
    ("block-fp32-S1024", 1, 1, 4, 4, 64, "fp32", 8, 2, 2047, 500, 300, "linear", False),
    ("wave-fp16-S128-NC128", 4, 4, 32, 32, 64, "fp16", 16, 4, 512, 32, 20, "linear", False),
    ("wave-zero-query", 4, 4, 32, 32, 64, "fp16", 16, 4, 512, 32, 20, "mean", True),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_select_exact_ties(case):
    name, L, B, Hq, Hkv, d, dtype, s, f, C, k_super, k_clusters, sim, zero_q = case
    say(f"[select ties] {name}: L={L} B={B} Hq={Hq} Hkv={Hkv} d={d} {dtype} C={C} f={f} "
        f"k_super={k_super} k_clusters={k_clusters} {sim}")
    import paper_2501_06807_amd as M
    S = -(-C // f)
    Ts = C * s
    R = oracle.rep_rows(sim)
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    q, cent, scent = _int_inputs(rng, L, B, Hq, Hkv, d, C, S, dtype, R, zero_q)
    sel_ref, _ = oracle.select_clusters(q, cent, scent, dtype, Ts=Ts, cluster=s, fanout=f, k_super=k_super,
                                        k_clusters=k_clusters, share_period=1, similarity=sim)
    cfg = M.select_cfg(s, f, k_super, k_clusters, 0.6, 1, similarity=sim)
    sel = torch.full(sel_ref.shape, -7, dtype=torch.int32, device="cuda")
    for rep in range(2):  # the second call sees the first call's outputs in place
        M.mpc_select_clusters(bits_to_torch(q, dtype), torch.from_numpy(cent).cuda(), torch.from_numpy(scent).cuda(),
                              sel, cfg, Ts=Ts)
        torch.cuda.synchronize()
        got = sel.cpu().numpy()
        bad = np.argwhere((got != sel_ref).any(-1))
        assert len(bad) == 0, f"{len(bad)} heads differ, first {bad[0].tolist()}: {got[tuple(bad[0])][:8]} vs " \
                              f"{sel_ref[tuple(bad[0])][:8]}"
    if zero_q:  # every score ties: the lowest candidate ids of the lowest super-clusters
        assert np.all(sel_ref == np.arange(k_clusters, dtype=np.int32))
