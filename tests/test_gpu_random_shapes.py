"""GPU parity of the whole decode path on seeded random shapes.

Each case draws its own shape from a seeded generator: element type, head dim, grouped heads,
sequences, layers and first layer of the block, sharing period and start, cluster size, fan-out,
a kept length that may end inside a cluster and a super-cluster, both budgets, the similarity
measure and the grouped-query rule. The cluster build must equal the oracle bit for bit, the
selection must equal it except where the oracle's scores tie at a level boundary (within 1e-6
relative), the attention over the GPU's selection must match the oracle's attention over the same
selection within the element type's tolerance, and the one-launch step must give the two separate
calls' selection and output bit for bit. The drawn shapes reach the kernels' other paths than the
fixed workloads do (counting versus tournament ranking, register ranking, workgroup- versus
wave-per-unit selection, split-K attention, ragged tails).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_out_close, bits_to_torch, boundary_score, say, torch_to_bits

pytestmark = pytest.mark.gpu

N_CASES = 24


def _draw(i):
    """Shape of case i (seeded; every draw satisfies the entry points' documented limits)."""
    rng = np.random.default_rng(0x5EED0000 + i)
    d = int(rng.choice([64, 128]))
    dtype = str(rng.choice(["bf16", "fp16", "fp32"]))
    G = int(rng.choice([1, 2, 4, 8]))
    Hkv = int(rng.integers(1, 4))
    B = int(rng.integers(1, 3))
    L = int(rng.integers(1, 7))
    layer0 = int(rng.integers(0, 5))
    period = int(rng.choice([1, 2, 3, 4]))
    start = int(rng.choice([0, 2]))
    s = int(rng.choice([4, 8, 16, 32, 64]))
    f = int(rng.choice([2, 3, 4, 8]))
    C = int(rng.integers(f + 1, 260))
    Ts = C * s - int(rng.integers(0, s))          # may end inside the last cluster
    S = -(-C // f)
    k_super = int(rng.integers(1, S + 1))
    last = C - (S - 1) * f                         # members of the last (maybe partial) super-cluster
    smallest = k_super * f - (f - last)            # fewest candidates any choice of k_super can give
    k_clusters = int(rng.integers(1, max(1, min(smallest, 48)) + 1))
    sim = str(rng.choice(["linear", "maxprod", "mean"]))
    rule = str(rng.choice(["sum", "max", "head"])) if G > 1 else "sum"
    base = "C2" if d == 64 else "C3"
    w = synth.get(base).with_(n_layers=L, batch=B, n_q_heads=G * Hkv, n_kv_heads=Hkv, head_dim=d, dtype=dtype,
                              keep=Ts, cluster=s, fanout=f, k_super=k_super, k_clusters=k_clusters,
                              share_period=period, share_start=start, seed=synth.workloads.SEED_BASE + 100 + i)
    return w, layer0, sim, rule


def _check_selection(w, layer0, q, cent, scent, sel_gpu, sel_ref, rule, sim):
    """Equal selections (ascending), except swaps where the oracle's scores tie at a level boundary;
    sharing layers hold their owner's selection."""
    C, f, G = cent.shape[3], w.fanout, w.group
    swaps = 0
    for l in range(w.n_layers):
        o = oracle.owner_layer(layer0 + l, w.share_period, w.share_start) - layer0
        if o != l:
            if o >= 0:
                np.testing.assert_array_equal(sel_gpu[l], sel_gpu[o])
            continue
        for b in range(w.batch):
            for h in range(sel_ref.shape[2]):
                got, exp = sel_gpu[l, b, h], sel_ref[l, b, h]
                assert np.all(np.diff(got) > 0), "selection must be ascending"
                if np.array_equal(got, exp):
                    continue
                heads = [h] if rule == "head" else list(range(h * G, (h + 1) * G))
                kvh = h // G if rule == "head" else h
                grp = "max" if rule == "max" else "sum"
                qg = q[l, b, heads]
                s1 = oracle.cluster_scores(qg, scent[l, b, kvh], w.dtype, sim, group=grp)
                s_all = oracle.cluster_scores(qg, cent[l, b, kvh], w.dtype, sim, group=grp)
                b1 = boundary_score(s1, w.k_super)
                top1 = set(np.argsort(-s1, kind="stable")[:w.k_super].tolist())
                ok_super = {c for c in range(C) if abs(s1[c // f] - b1) <= 1e-6 * abs(b1)}
                cand = [c for c in range(C) if c in ok_super or c // f in top1]
                b2 = boundary_score(s_all[cand], w.k_clusters)
                bad = [c for c in set(got.tolist()) ^ set(exp.tolist())
                       if c not in ok_super and abs(s_all[c] - b2) > 1e-6 * abs(b2)]
                assert not bad, f"layer {l} b {b} unit {h}: non-tie differences {bad}"
                swaps += 1
    return swaps


@pytest.mark.parametrize("i", range(N_CASES))
def test_random_shape_decode_path(i):
    import paper_2501_06807_amd as M
    w, layer0, sim, rule = _draw(i)
    C = -(-w.keep // w.cluster)
    S = -(-C // w.fanout)
    say(f"[random {i}] {w.dtype} d={w.head_dim} L={w.n_layers}@{layer0} B={w.batch} Hq={w.n_q_heads} "
        f"Hkv={w.n_kv_heads} P={w.share_period}/{w.share_start} Ts={w.keep} s={w.cluster} f={w.fanout} C={C} "
        f"S={S} k_super={w.k_super} k_clusters={w.k_clusters} {sim} {rule}")
    ks, vs = zip(*[synth.cache_host(w, layer0 + l, T=w.keep) for l in range(w.n_layers)])
    k, v = np.stack(ks), np.stack(vs)
    q = synth.dq_host(synth.spec(w, n_layers=layer0 + w.n_layers), 1, w.dtype)[layer0:]

    # cluster build: bit-exact
    cent, scent = oracle.build_clusters(k, w.dtype, cluster=w.cluster, fanout=w.fanout, alpha=0.6, layer0=layer0,
                                        share_period=w.share_period, share_start=w.share_start, similarity=sim)
    cfg = M.select_cfg(w.cluster, w.fanout, w.k_super, w.k_clusters, 0.6, w.share_period, w.share_start,
                       similarity=sim, group=rule)
    qd, kd, vd = (bits_to_torch(x, w.dtype) for x in (q, k, v))
    cd = torch.zeros(cent.shape, dtype=torch.float32, device="cuda")
    sd = torch.zeros(scent.shape, dtype=torch.float32, device="cuda")
    M.mpc_build_clusters(kd, cd, sd, cfg, layer0=layer0)
    torch.cuda.synchronize()
    owned = [l for l in range(w.n_layers)
             if oracle.owner_layer(layer0 + l, w.share_period, w.share_start) == layer0 + l]
    for l in owned:
        np.testing.assert_array_equal(cd[l].cpu().numpy(), cent[l])
        np.testing.assert_array_equal(sd[l].cpu().numpy(), scent[l])
    cd, sd = torch.from_numpy(cent).cuda(), torch.from_numpy(scent).cuda()

    # selection: equal to the oracle up to boundary ties; layers owned before the block are inputs
    sel_ref, _ = oracle.select_clusters(q, cent, scent, w.dtype, Ts=w.keep, cluster=w.cluster, fanout=w.fanout,
                                        k_super=w.k_super, k_clusters=w.k_clusters, layer0=layer0,
                                        share_period=w.share_period, share_start=w.share_start, similarity=sim,
                                        group=rule)
    given = [l for l in range(w.n_layers) if oracle.owner_layer(layer0 + l, w.share_period, w.share_start) < layer0]
    sel_in = np.full(sel_ref.shape, -7, dtype=np.int32)
    for l in given:  # the caller's selection for layers owned before the block: any valid list
        sel_in[l] = np.arange(w.k_clusters, dtype=np.int32) * (C // w.k_clusters)
        sel_ref[l] = sel_in[l]
    sel = torch.from_numpy(sel_in).cuda()
    M.mpc_select_clusters(qd, cd, sd, sel, cfg, Ts=w.keep, layer0=layer0)
    torch.cuda.synchronize()
    sel_g = sel.cpu().numpy()
    for l in given:
        np.testing.assert_array_equal(sel_g[l], sel_in[l])
    swaps = _check_selection(w, layer0, q, cent, scent, sel_g, sel_ref, rule, sim)

    # attention over the GPU's selection: within the element type's tolerance of the oracle's
    sm = 1.0 / math.sqrt(w.head_dim)
    dt = synth.torch_dtype(w.dtype)
    out = torch.empty(q.shape, dtype=dt, device="cuda")
    lse = torch.empty(q.shape[:-1], dtype=torch.float32, device="cuda")
    M.mpc_sparse_decode_attn(qd, kd, vd, sel, out, cluster_size=w.cluster, sm_scale=sm, lse=lse, layer0=layer0)
    torch.cuda.synchronize()
    ref, lse_ref = oracle.sparse_decode_attn(q, k, v, sel_g, w.dtype, cluster=w.cluster, sm_scale=sm)
    worst = assert_out_close(out.double().cpu().numpy(), ref, w.dtype, f"random case {i}")
    np.testing.assert_allclose(lse.cpu().numpy(), lse_ref, rtol=1e-5, atol=1e-5)

    # one launch: the two calls' selection and output bit for bit
    sel1 = torch.from_numpy(sel_in).cuda()
    out1 = torch.empty_like(out)
    M.mpc_decode_step(qd, cd, sd, kd, vd, sel1, out1, cfg, sm_scale=sm, layer0=layer0)
    torch.cuda.synchronize()
    assert torch.equal(sel1, sel), "one-launch selection differs from mpc_select_clusters"
    assert torch.equal(out1.view(torch.uint8), out.view(torch.uint8)), "one-launch output differs"
    say(f"  tie swaps {swaps}, worst attention relative error {worst:.2e}")


N_EVICT_CASES = 16


def _draw_evict(i):
    """Shape of static-eviction case i: element type, head dim, grouped heads, sequences, layer block
    and sharing, prompt length, window rows (ending anywhere inside the scoring passes' register
    blocks), kept and recent counts."""
    rng = np.random.default_rng(0xE71C0000 + i)
    d = int(rng.choice([64, 128]))
    dtype = str(rng.choice(["bf16", "fp16", "fp32"]))
    G = int(rng.choice([1, 2, 4]))
    Hkv = int(rng.integers(1, 3))
    B = int(rng.integers(1, 3))
    L = int(rng.integers(1, 5))
    layer0 = int(rng.integers(0, 4))
    period = int(rng.choice([1, 2, 4]))
    start = int(rng.choice([0, 2]))
    T = int(rng.integers(64, 1400))
    W = int(rng.integers(1, min(T, 300) + 1))
    local = int(rng.integers(0, 65))
    keep = int(rng.integers(max(local, 1), T + 1))
    s = int(rng.choice([4, 8, 16, 32]))
    f = int(rng.choice([2, 4, 8]))
    sim = str(rng.choice(["linear", "maxprod", "mean"]))
    base = "C2" if d == 64 else "C3"
    w = synth.get(base).with_(n_layers=L, batch=B, n_q_heads=G * Hkv, n_kv_heads=Hkv, head_dim=d, dtype=dtype, T=T,
                              window=W, keep=keep, local_keep=local, cluster=s, fanout=f, share_period=period,
                              share_start=start, seed=synth.workloads.SEED_BASE + 200 + i)
    return w, layer0, sim


@pytest.mark.parametrize("i", range(N_EVICT_CASES))
def test_random_shape_static_eviction_and_prefill(i):
    """Static eviction against the oracle (token scores within 2e-5, kept sets equal up to boundary
    ties, gathered rows a bit copy, row log-sum-exp sampled) and the one-call prefill equal to
    eviction followed by the cluster build, bit for bit."""
    import paper_2501_06807_amd as M
    from test_gpu_evict import _check, _row_lse_check
    w, layer0, sim = _draw_evict(i)
    say(f"[random evict {i}] {w.dtype} d={w.head_dim} L={w.n_layers}@{layer0} B={w.batch} Hq={w.n_q_heads} "
        f"Hkv={w.n_kv_heads} P={w.share_period}/{w.share_start} T={w.T} W={w.window} keep={w.keep} "
        f"local={w.local_keep} s={w.cluster} f={w.fanout} {sim}")
    parts = [synth.prefill_host(w, layer0 + l) for l in range(w.n_layers)]
    qw, k, v = (np.stack([p[j] for p in parts]) for j in range(3))
    # layers owned before the block arrive with their kept set
    kept_in = np.zeros((w.n_layers, w.batch, w.n_kv_heads, w.keep), dtype=np.int32)
    given = [l for l in range(w.n_layers) if oracle.owner_layer(layer0 + l, w.share_period, w.share_start) < layer0]
    loc = min(w.local_keep, w.keep)
    for l in given:  # a kept set of the method's form: older tokens, then the recent window
        older = np.sort(np.random.default_rng(i).choice(w.T - loc, w.keep - loc, replace=False))
        kept_in[l] = np.concatenate([older, np.arange(w.T - loc, w.T)]).astype(np.int32)
    dt = w.dtype
    qd, kd, vd = bits_to_torch(qw, dt), bits_to_torch(k, dt), bits_to_torch(v, dt)
    R = 2 if sim == "maxprod" else 1
    C = -(-w.keep // w.cluster)
    S = -(-C // w.fanout)
    cfg = M.select_cfg(w.cluster, w.fanout, 1, 1, 0.6, w.share_period, w.share_start, sim)
    sm = 1.0 / math.sqrt(w.head_dim)

    def run(fused):
        kept = torch.from_numpy(kept_in).cuda()
        k_out = torch.zeros((w.n_layers, w.batch, w.n_kv_heads, w.keep, w.head_dim), dtype=synth.torch_dtype(dt),
                            device="cuda")
        v_out = torch.zeros_like(k_out)
        cent = torch.zeros((w.n_layers, w.batch, w.n_kv_heads, C, R, w.head_dim), dtype=torch.float32, device="cuda")
        scent = torch.zeros((w.n_layers, w.batch, w.n_kv_heads, S, R, w.head_dim), dtype=torch.float32,
                            device="cuda")
        score = torch.zeros((w.n_layers, w.batch, w.n_kv_heads, w.T), dtype=torch.float32, device="cuda")
        lse = torch.zeros((w.n_layers, w.batch, w.n_q_heads, w.window), dtype=torch.float32, device="cuda")
        kw = dict(keep=w.keep, local_keep=w.local_keep, sm_scale=sm, layer0=layer0, share_period=w.share_period,
                  share_start=w.share_start, token_score=score, row_lse=lse)
        if fused:
            M.mpc_prefill(qd, kd, vd, kept, k_out, v_out, cent, scent, cfg, **kw)
        else:
            M.mpc_static_evict(qd, kd, vd, kept, k_out, v_out, **kw)
            M.mpc_build_clusters(k_out, cent, scent, cfg, Ts=w.keep, layer0=layer0)
        torch.cuda.synchronize()
        return [kept.cpu().numpy(), torch_to_bits(k_out, dt), torch_to_bits(v_out, dt), score.cpu().numpy(),
                lse.cpu().numpy(), cent.cpu().numpy(), scent.cpu().numpy()]

    two = run(False)
    one = run(True)
    for a, b, name in zip(two, one, ["kept", "k_out", "v_out", "token_score", "row_lse", "cent", "scent"]):
        if name == "cent" or name == "scent":  # representatives exist for the selection's owner layers
            owners = [l for l in range(w.n_layers)
                      if oracle.owner_layer(layer0 + l, w.share_period, w.share_start) == layer0 + l]
            a, b = a[owners], b[owners]
        assert np.array_equal(a, b), f"one-call prefill differs from the two calls in {name}"
    for l in given:
        np.testing.assert_array_equal(two[0][l], kept_in[l])
    # scores and kept sets of the layers owned inside the block; every layer's gathered rows
    swaps, worst = _check(w, qw, k, v, two[:5], layer0=layer0)
    _row_lse_check(w, qw, k, two[4], layer0=layer0, rows=6)
    say(f"  tie swaps {swaps}, worst score relative error {worst:.2e}")
