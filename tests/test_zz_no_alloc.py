"""The entry point that allocates nothing (mpc_static_evict_noalloc, its workspace a static device
array) gives what mpc_static_evict with a caller workspace gives, bit for bit, on two calls in a row,
the second on a smaller block (the refusal of a block beyond the array is a host-side check in
test_abi.py)."""
import math

import numpy as np
import pytest
import torch

import synth
from gpu_util import bits_to_torch, say

pytestmark = pytest.mark.gpu


def _inputs(w):
    qs, ks, vs = [], [], []
    for l in range(w.n_layers):
        qw, k, v = synth.prefill_host(w, l)
        qs.append(qw)
        ks.append(k)
        vs.append(v)
    dt = w.dtype
    return bits_to_torch(np.stack(qs), dt), bits_to_torch(np.stack(ks), dt), bits_to_torch(np.stack(vs), dt)


def _evict(M, w, q_win, k, v, noalloc, stream=None):
    L, B, Hkv, T, d = k.shape
    kept = torch.full((L, B, Hkv, w.keep), -1, dtype=torch.int32, device="cuda")
    k_out = torch.zeros((L, B, Hkv, w.keep, d), dtype=k.dtype, device="cuda")
    v_out = torch.zeros_like(k_out)
    score = torch.zeros((L, B, Hkv, T), dtype=torch.float32, device="cuda")
    lse = torch.zeros((L, B, q_win.shape[2], q_win.shape[3]), dtype=torch.float32, device="cuda")
    kw = dict(keep=w.keep, local_keep=w.local_keep, sm_scale=1.0 / math.sqrt(d), share_period=w.share_period,
              share_start=w.share_start, token_score=score, row_lse=lse)
    if noalloc:
        if stream is not None:  # the outputs' fills above ran on the current stream
            stream.wait_stream(torch.cuda.current_stream())
        M.mpc_static_evict_noalloc(q_win, k, v, kept, k_out, v_out, stream=stream, **kw)
    else:
        M.mpc_static_evict(q_win, k, v, kept, k_out, v_out, **kw)
    torch.cuda.synchronize()
    return kept, k_out, v_out, score, lse


def _same(a, b):
    return all(torch.equal(x.view(torch.int32) if x.dtype == torch.float32 else x.view(torch.int16)
                           if x.dtype in (torch.bfloat16, torch.float16) else x,
                           y.view(torch.int32) if y.dtype == torch.float32 else y.view(torch.int16)
                           if y.dtype in (torch.bfloat16, torch.float16) else y) for x, y in zip(a, b))


def test_noalloc_static_evict_matches_the_workspace_call_twice():
    import paper_2501_06807_amd as M
    limit = M.noalloc_limit()
    # first call: 8K prompt, four layers of 8 kv heads with sharing; second: a smaller GQA block
    first = synth.get("C3").with_(n_layers=4, n_q_heads=8, n_kv_heads=8)
    second = synth.get("C2").with_(n_layers=3)
    # the second call runs on a stream of its own (default priority): the scratch address is that
    # of the stream's device
    side = torch.cuda.Stream()
    for w, stream in ((first, None), (second, side)):
        q_win, k, v = _inputs(w)
        dims = M.dims_of(q_win, k)
        cfg = M.MpcEvictCfg(window=w.window, keep=w.keep, local_keep=w.local_keep, sm_scale=1.0, causal=1,
                            share_period=w.share_period, share_start=w.share_start)
        need = M.workspace_bytes(M.MPC_OP_STATIC_EVICT, dims, w.T, cfg)
        say(f"[noalloc] {w.name} L={w.n_layers}: workspace {need} of {limit} scratch bytes")
        assert 0 < need <= limit
        ref = _evict(M, w, q_win, k, v, noalloc=False)
        got = _evict(M, w, q_win, k, v, noalloc=True, stream=stream)
        assert _same(ref, got), f"{w.name}: the no-allocation call differs from the workspace call"
        assert (got[0] >= 0).all()

