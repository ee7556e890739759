"""GPU parity of look-once static eviction (window scoring, top-k, gather) against the oracle."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_sets_tie_equal, bits_to_torch, boundary_score, say, torch_to_bits

pytestmark = pytest.mark.gpu


def _prefill(w, layer0=0):
    qs, ks, vs = [], [], []
    for l in range(w.n_layers):
        qw, k, v = synth.prefill_host(w, layer0 + l)
        qs.append(qw)
        ks.append(k)
        vs.append(v)
    return np.stack(qs), np.stack(ks), np.stack(vs)


def _run_gpu(w, qw, k, v, layer0=0, kept_in=None, causal=True, sm=None):
    import paper_2501_06807_amd as M
    L, B, Hkv = k.shape[:3]
    dt = w.dtype
    kept = (torch.zeros((L, B, Hkv, w.keep), dtype=torch.int32, device="cuda") if kept_in is None
            else torch.from_numpy(kept_in).cuda())
    k_out = torch.empty((L, B, Hkv, w.keep, w.head_dim), dtype=synth.torch_dtype(dt), device="cuda")
    v_out = torch.empty_like(k_out)
    score = torch.zeros((L, B, Hkv, w.T), dtype=torch.float32, device="cuda")
    row_lse = torch.zeros((L, B, w.n_q_heads, w.window), dtype=torch.float32, device="cuda")
    M.mpc_static_evict(bits_to_torch(qw, dt), bits_to_torch(k, dt), bits_to_torch(v, dt), kept, k_out, v_out,
                       keep=w.keep, local_keep=w.local_keep,
                       sm_scale=1.0 / math.sqrt(w.head_dim) if sm is None else sm, causal=causal,
                       layer0=layer0, share_period=w.share_period, share_start=w.share_start,
                       token_score=score, row_lse=row_lse)
    torch.cuda.synchronize()
    return (kept.cpu().numpy(), torch_to_bits(k_out, dt), torch_to_bits(v_out, dt), score.cpu().numpy(),
            row_lse.cpu().numpy())


def _check(w, qw, k, v, got, layer0=0, score_rtol=2e-5):
    kept_g, ko_g, vo_g, sc_g, lse_g = got
    sm = 1.0 / math.sqrt(w.head_dim)
    kept_r, ko_r, vo_r, sc_r = oracle.static_evict(qw, k, v, w.dtype, keep=w.keep, local_keep=w.local_keep,
                                                   sm_scale=sm, layer0=layer0, share_period=w.share_period,
                                                   share_start=w.share_start, with_scores=True)
    G = w.group
    loc = min(w.local_keep, w.keep)
    swaps = 0
    worst = 0.0
    for l in range(w.n_layers):
        owner = oracle.owner_layer(layer0 + l, w.share_period, w.share_start) == layer0 + l
        for b in range(w.batch):
            for h in range(w.n_kv_heads):
                got_k = kept_g[l, b, h]
                assert np.all(np.diff(got_k) > 0), "kept set must be ascending and unique"
                if loc:
                    np.testing.assert_array_equal(got_k[-loc:], np.arange(w.T - loc, w.T))
                if owner:
                    worst = max(worst, float(np.max(np.abs(sc_g[l, b, h] - sc_r[l, b, h]) / sc_r[l, b, h])))
                    np.testing.assert_allclose(sc_g[l, b, h], sc_r[l, b, h], rtol=score_rtol)
                    assert abs(sc_g[l, b, h].astype(np.float64).sum() - G * w.window) < 1e-5 * G * w.window
                    bnd = boundary_score(sc_r[l, b, h, :w.T - loc], w.keep - loc)
                    swaps += assert_sets_tie_equal(got_k, kept_r[l, b, h], sc_r[l, b, h], bnd,
                                                   f"layer {l} b {b} h {h}")
                # the gather is a bit copy of the kept rows
                np.testing.assert_array_equal(ko_g[l, b, h], k[l, b, h, got_k])
                np.testing.assert_array_equal(vo_g[l, b, h], v[l, b, h, got_k])
            if not owner:
                o = oracle.owner_layer(layer0 + l, w.share_period, w.share_start) - layer0
                if o >= 0:
                    np.testing.assert_array_equal(kept_g[l], kept_g[o])
    return swaps, worst


def _row_lse_check(w, qw, k, lse_g, layer0=0, rows=8):
    sm = 1.0 / math.sqrt(w.head_dim)
    rng = np.random.default_rng(7)
    for l in range(w.n_layers):
        if oracle.owner_layer(layer0 + l, w.share_period, w.share_start) != layer0 + l:
            continue
        for _ in range(rows):
            b, hq, t = rng.integers(w.batch), rng.integers(w.n_q_heads), rng.integers(w.window)
            ref = oracle.row_lse(qw[l, b, hq, t], int(t), w.window, k[l, b, hq // w.group], w.dtype, sm)
            assert abs(lse_g[l, b, hq, t] - ref) <= 2e-6 * max(1.0, abs(ref)), (l, b, hq, t)


CASES = {
    # name: overrides of the workload (fewer heads / shorter prompts so the oracle finishes quickly)
    "C1": {},
    "C2": dict(n_layers=4),
    "C3": dict(n_layers=1, n_q_heads=4, n_kv_heads=4),
    "C4": dict(n_layers=1, batch=2, n_q_heads=2, n_kv_heads=2, T=4096, window=409, keep=1216),
    "C5": dict(n_layers=1, n_q_heads=8, n_kv_heads=2, T=4096, window=409, keep=1024, hh_count=8,
               hh_hi=4096 - 32),
    "X1": dict(n_layers=2, batch=2, n_q_heads=4, n_kv_heads=4),
    # the other element types at the other head dim, ragged window rows and key blocks
    "C3-fp16": dict(n_layers=1, n_q_heads=4, n_kv_heads=2, dtype="fp16", T=2000, window=400, keep=1024),
    "C3-fp32": dict(n_layers=1, n_q_heads=2, n_kv_heads=2, dtype="fp32", T=1500, window=300, keep=768),
    "C2-bf16": dict(n_layers=2, n_q_heads=4, n_kv_heads=2, dtype="bf16", T=1300, window=260, keep=640),
    # the most layers one call takes (256): owners on both sides of every 64-layer boundary
    "C2-L256": dict(n_layers=256, n_q_heads=2, n_kv_heads=1, T=160, window=32, keep=80, share_period=3),
}


@pytest.mark.parametrize("name", list(CASES))
def test_static_evict_matches_oracle(name):
    w = synth.get(name.split("-")[0]).with_(**CASES[name])  # "C3-fp16": workload C3, overridden
    say(f"[evict] {name} L={w.n_layers} B={w.batch} Hq={w.n_q_heads} Hkv={w.n_kv_heads} T={w.T} "
        f"W={w.window} keep={w.keep} {w.dtype}")
    qw, k, v = _prefill(w)
    got = _run_gpu(w, qw, k, v)
    swaps, worst = _check(w, qw, k, v, got)
    _row_lse_check(w, qw, k, got[4])
    say(f"  tie swaps {swaps}, worst score relative error {worst:.2e}")


# Edges of the scoring passes' register blocks (for 16-bit inputs a wave holds 64 window rows in the
# row pass and 64 keys in the column pass as four groups of 16, tiles of 64 keys / rows are staged
# per barrier, and a workgroup covers 256 rows / keys; fp32 inputs use one 32-row block per wave):
# windows that end inside a wave's groups or just past a workgroup, key ranges that end inside a
# staged tile, both element sizes and head dims, grouped heads.
EDGE_CASES = {
    "W20-T1000": dict(base="C3", n_q_heads=4, n_kv_heads=1, T=1000, window=20, keep=512),
    "W33-T993-fp16": dict(base="C3", n_q_heads=2, n_kv_heads=2, dtype="fp16", T=993, window=33, keep=480),
    "W64-T1088": dict(base="C3", n_q_heads=4, n_kv_heads=2, T=1088, window=64, keep=544),
    "W65-T1057-d64": dict(base="C2", n_layers=1, n_q_heads=4, n_kv_heads=4, dtype="bf16", T=1057, window=65, keep=528),
    "W257-T1285": dict(base="C3", n_q_heads=2, n_kv_heads=1, T=1285, window=257, keep=640),
    "W100-T700-fp32": dict(base="C3", n_q_heads=2, n_kv_heads=2, dtype="fp32", T=700, window=100, keep=352),
    # degenerate sizes: every token kept, the window the whole prompt; a one-row window and no recent
    # tokens kept by rule; more recent tokens asked for than kept (the last `keep` tokens, the top-k
    # choosing none)
    "keep-all-W=T": dict(base="C3", n_q_heads=2, n_kv_heads=1, T=300, window=300, keep=300),
    "W1-local0": dict(base="C2", n_layers=2, n_q_heads=2, n_kv_heads=2, T=500, window=1, keep=100, local_keep=0),
    "local-above-keep": dict(base="C3", n_q_heads=2, n_kv_heads=2, T=500, window=50, keep=40, local_keep=64),
}


@pytest.mark.parametrize("name", list(EDGE_CASES))
def test_static_evict_block_edges(name):
    o = dict(EDGE_CASES[name])
    w = synth.get(o.pop("base")).with_(n_layers=o.pop("n_layers", 1), **o)
    say(f"[evict edge] {name} Hq={w.n_q_heads} Hkv={w.n_kv_heads} d={w.head_dim} T={w.T} W={w.window} "
        f"keep={w.keep} {w.dtype}")
    qw, k, v = _prefill(w)
    got = _run_gpu(w, qw, k, v)
    swaps, worst = _check(w, qw, k, v, got)
    _row_lse_check(w, qw, k, got[4], rows=16)
    say(f"  tie swaps {swaps}, worst score relative error {worst:.2e}")


# All-zero window queries: every score is 0, so every block of the row pass sums four terms of
# exactly 1 and goes through its offset check's slow path, and the accumulated attention has a
# closed form: key j receives 1 / (T - W + t + 1) from every window row t that sees it, once per
# query head of its group, and row t's log-sum-exp is ln(T - W + t + 1). Most older tokens tie.
EQUAL_CASES = {
    "bf16-d128": dict(base="C3", n_q_heads=4, n_kv_heads=2, T=1100, window=200, keep=560),
    "fp16-d64": dict(base="C2", n_q_heads=4, n_kv_heads=2, dtype="fp16", T=777, window=150, keep=400),
}


@pytest.mark.parametrize("name", list(EQUAL_CASES))
def test_static_evict_equal_scores(name):
    o = dict(EQUAL_CASES[name])
    w = synth.get(o.pop("base")).with_(n_layers=1, **o)
    say(f"[evict equal scores] {name} Hq={w.n_q_heads} Hkv={w.n_kv_heads} d={w.head_dim} T={w.T} "
        f"W={w.window} keep={w.keep} {w.dtype}")
    qw, k, v = _prefill(w)
    qw = np.zeros_like(qw)
    got = _run_gpu(w, qw, k, v)
    T, W = w.T, w.window
    seen = T - W + np.arange(W) + 1                       # keys row t attends
    tail = np.cumsum((1.0 / seen)[::-1])[::-1]            # tail[t] = sum over rows t' >= t of 1 / seen
    first = np.clip(np.arange(T) - (T - W), 0, None)      # first window row that sees key j
    exact = w.group * tail[first]
    for b in range(w.batch):
        for h in range(w.n_kv_heads):
            np.testing.assert_allclose(got[3][0, b, h], exact, rtol=1e-6)
        for hq in range(w.n_q_heads):
            np.testing.assert_allclose(got[4][0, b, hq], np.log(seen), rtol=1e-6)
    swaps, worst = _check(w, qw, k, v, got)
    say(f"  closed form ok; tie swaps {swaps}, worst score relative error {worst:.2e}")


def test_static_evict_block_whose_first_owner_precedes_it():
    w = synth.get("C2").with_(n_layers=3, T=700, window=140, keep=320, n_q_heads=4, n_kv_heads=4)
    say("[evict] layer block starting at 3 (layer 3 follows layer 2)")
    qw, k, v = _prefill(w, layer0=3)
    # layer 3's owner is layer 2 (outside the block): its kept set is an input
    prev = np.tile(np.sort(np.random.default_rng(0).choice(700, 320, replace=False)).astype(np.int32),
                   (3, 1, 4, 1))
    got = _run_gpu(w, qw, k, v, layer0=3, kept_in=prev)
    np.testing.assert_array_equal(got[0][0], prev[0])
    np.testing.assert_array_equal(got[1][0, 0, 1], k[0, 0, 1, prev[0, 0, 1]])
    kept_r, _, _ = oracle.static_evict(qw, k, v, w.dtype, keep=w.keep, local_keep=w.local_keep,
                                       sm_scale=1 / 8, layer0=3, share_period=2, kept_in=prev)
    sc_r = oracle.static_evict(qw, k, v, w.dtype, keep=w.keep, local_keep=w.local_keep, sm_scale=1 / 8,
                               layer0=3, share_period=2, kept_in=prev, with_scores=True)[3]
    for h in range(4):
        bnd = boundary_score(sc_r[1, 0, h, :w.T - 32], w.keep - 32)
        assert_sets_tie_equal(got[0][1, 0, h], kept_r[1, 0, h], sc_r[1, 0, h], bnd, f"h {h}")
    np.testing.assert_array_equal(got[0][2], got[0][1])  # layer 5 follows layer 4


def test_identity_budget_keeps_everything():
    w = synth.get("C1").with_(keep=512)
    say("[evict] keep = T")
    qw, k, v = _prefill(w)
    kept, ko, vo, _, _ = _run_gpu(w, qw, k, v)
    assert np.all(kept == np.arange(512))
    np.testing.assert_array_equal(ko, k)
    np.testing.assert_array_equal(vo, v)


@pytest.mark.parametrize("name", ["C1", "C2"])
def test_literal_algorithm_readings(name):
    """Alg. 3 read literally: no causal mask, no 1/sqrt(d) in the window scores, and the pairing
    l % 2 of layers (sharing from layer 0). The kept sets follow the oracle under the tie rule;
    token scores are compared against the largest one (sharper softmaxes underflow the smallest)."""
    w = synth.get(name).with_(share_start=0, **({"n_layers": 4} if name == "C2" else {}))
    say(f"[evict literal] {name} causal=0 sm_scale=1 share_start=0 P={w.share_period}")
    qw, k, v = _prefill(w)
    kept_g, ko_g, vo_g, sc_g, _ = _run_gpu(w, qw, k, v, causal=False, sm=1.0)
    kept_r, _, _, sc_r = oracle.static_evict(qw, k, v, w.dtype, keep=w.keep, local_keep=w.local_keep, sm_scale=1.0,
                                             causal=False, share_period=w.share_period, share_start=0,
                                             with_scores=True)
    loc = min(w.local_keep, w.keep)
    for l in range(w.n_layers):
        o = oracle.owner_layer(l, w.share_period, 0)
        for b in range(w.batch):
            for h in range(w.n_kv_heads):
                if o == l:
                    top = float(sc_r[l, b, h].max())
                    np.testing.assert_allclose(sc_g[l, b, h], sc_r[l, b, h], rtol=2e-5, atol=1e-6 * top)
                    bnd = boundary_score(sc_r[l, b, h, :w.T - loc], w.keep - loc)
                    assert_sets_tie_equal(kept_g[l, b, h], kept_r[l, b, h], sc_r[l, b, h], bnd, f"l {l} h {h}")
                else:
                    np.testing.assert_array_equal(kept_g[l, b, h], kept_g[o, b, h])
                np.testing.assert_array_equal(ko_g[l, b, h], k[l, b, h, kept_g[l, b, h]])
