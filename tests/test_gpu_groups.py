"""GPU parity of the grouped-query selection rules, per-q-head attention lists and the
layer-commonality score against the oracle.

Rules (the paper states the selection for one query head): "sum" (the q-heads of a kv head share
one selection scored by the sum of their similarities), "max" (scored by the largest), "head" (every
q-head selects its own clusters and attends only them). Inputs are the seeded workload generators'
caches and queries; each stage gets the oracle's upstream outputs.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_out_close, bits_to_torch, boundary_score, random_sel, say

pytestmark = pytest.mark.gpu

# (workload, overrides): GQA shapes spanning the workgroup-per-unit and wave-per-unit kernels
CASES = {
    "C5-L6": ("C5", dict(n_layers=6)),                                          # G = 4, bf16, d = 128
    "C2-G2": ("C2", dict(n_layers=4, n_q_heads=12, n_kv_heads=6)),              # G = 2, fp16, d = 64
    # 512 selection units: the wave-per-unit kernel (per q-head for "head", per kv head for "max")
    "C5-wide": ("C5", dict(n_layers=4, batch=4, keep=8192, k_super=8, share_period=1)),
    "C4-G2": ("C4", dict(n_layers=4, n_q_heads=64, n_kv_heads=32, keep=2048, k_super=4, k_clusters=8,
                         share_period=1)),
}


def _case(name):
    base, kw = CASES[name]
    return synth.get(base).with_(**kw)


def _inputs(w, step=0, sim="linear"):
    ks = [synth.cache_host(w, l, T=w.keep)[0] for l in range(w.n_layers)]
    k = np.stack(ks)
    cent, scent = oracle.build_clusters(k, w.dtype, cluster=w.cluster, fanout=w.fanout, alpha=0.6,
                                        share_period=w.share_period, similarity=sim)
    q = synth.dq_host(synth.spec(w), step, w.dtype)
    return k, q, cent, scent


def _check(w, q, cent, scent, sel_gpu, sel_ref, rule, sim):
    """Equal selections, except swaps where the oracle's scores tie at a level boundary."""
    C, f, G = cent.shape[3], w.fanout, w.group
    swaps = 0
    for l in range(w.n_layers):
        o = oracle.owner_layer(l, w.share_period, w.share_start)
        if o != l:
            np.testing.assert_array_equal(sel_gpu[l], sel_gpu[o])
            continue
        for b in range(w.batch):
            for h in range(sel_ref.shape[2]):
                got, exp = sel_gpu[l, b, h], sel_ref[l, b, h]
                assert np.all(np.diff(got) > 0)
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


@pytest.mark.parametrize("rule", ["max", "head"])
@pytest.mark.parametrize("sim", ["linear", "maxprod"])
@pytest.mark.parametrize("name", list(CASES))
def test_select_group_rule_matches_oracle(name, sim, rule):
    import paper_2501_06807_amd as M
    w = _case(name)
    say(f"[select {rule}] {name} {sim} L={w.n_layers} B={w.batch} Hq={w.n_q_heads} Hkv={w.n_kv_heads} "
        f"Ts={w.keep} k_super={w.k_super} k_clusters={w.k_clusters}")
    k, q, cent, scent = _inputs(w, 1, sim)
    sel_ref, _ = oracle.select_clusters(q, cent, scent, w.dtype, Ts=w.keep, cluster=w.cluster, fanout=w.fanout,
                                        k_super=w.k_super, k_clusters=w.k_clusters, share_period=w.share_period,
                                        similarity=sim, group=rule)
    cfg = M.select_cfg(w.cluster, w.fanout, w.k_super, w.k_clusters, 0.6, w.share_period, similarity=sim,
                       group=rule)
    sel = torch.full(sel_ref.shape, -7, dtype=torch.int32, device="cuda")
    M.mpc_select_clusters(bits_to_torch(q, w.dtype), torch.from_numpy(cent).cuda(), torch.from_numpy(scent).cuda(),
                          sel, cfg, Ts=w.keep)
    torch.cuda.synchronize()
    swaps = _check(w, q, cent, scent, sel.cpu().numpy(), sel_ref, rule, sim)
    say(f"  tie swaps {swaps}")


@pytest.mark.parametrize("name", ["C5-L6", "C2-G2"])
def test_per_head_attention_matches_oracle(name):
    import paper_2501_06807_amd as M
    w = _case(name)
    C = -(-w.keep // w.cluster)
    say(f"[attn per q-head] {name} L={w.n_layers} Hq={w.n_q_heads} Hkv={w.n_kv_heads} Ts={w.keep}")
    ks, vs = zip(*[synth.cache_host(w, l, T=w.keep) for l in range(w.n_layers)])
    k, v = np.stack(ks), np.stack(vs)
    q = synth.dq_host(synth.spec(w), 0, w.dtype)
    rng = np.random.default_rng(77)
    sel = random_sel(rng, w.n_layers * w.batch * w.n_q_heads, C, w.k_clusters).reshape(
        w.n_layers, w.batch, w.n_q_heads, w.k_clusters)
    sm = 1.0 / math.sqrt(w.head_dim)
    ref, lse_ref = oracle.sparse_decode_attn(q, k, v, sel, w.dtype, cluster=w.cluster, sm_scale=sm)
    out = torch.empty(q.shape, dtype=synth.torch_dtype(w.dtype), device="cuda")
    lse = torch.empty(q.shape[:-1], dtype=torch.float32, device="cuda")
    M.mpc_sparse_decode_attn(bits_to_torch(q, w.dtype), bits_to_torch(k, w.dtype), bits_to_torch(v, w.dtype),
                             torch.from_numpy(sel).cuda(), out, cluster_size=w.cluster, sm_scale=sm, lse=lse)
    torch.cuda.synchronize()
    worst = assert_out_close(out.double().cpu().numpy(), ref, w.dtype, "per-head attention")
    np.testing.assert_allclose(lse.double().cpu().numpy(), lse_ref, rtol=1e-5, atol=1e-5)
    say(f"  worst relative error {worst:.2e}")


@pytest.mark.parametrize("rule", ["max", "head"])
def test_decode_step_group_rule_equals_two_calls_and_oracle(rule):
    """mpc_decode_step (one launch for "max", the two kernels in sequence for "head") against the
    two separate calls bit for bit, and against the oracle's selection and attention."""
    import paper_2501_06807_amd as M
    w = _case("C5-L6")
    say(f"[decode step {rule}] C5 L={w.n_layers} Hq={w.n_q_heads} Hkv={w.n_kv_heads}")
    k, q, cent, scent = _inputs(w, 2)
    _, v = zip(*[synth.cache_host(w, l, T=w.keep) for l in range(w.n_layers)])
    v = np.stack(v)
    dt = synth.torch_dtype(w.dtype)
    cfg = M.select_cfg(w.cluster, w.fanout, w.k_super, w.k_clusters, 0.6, w.share_period, group=rule)
    H = M.sel_heads(cfg, w.n_q_heads, w.n_kv_heads)
    qd, kd, vd = (bits_to_torch(x, w.dtype) for x in (q, k, v))
    cd, sd = torch.from_numpy(cent).cuda(), torch.from_numpy(scent).cuda()
    sm = 1.0 / math.sqrt(w.head_dim)
    shape = (w.n_layers, w.batch, H, w.k_clusters)
    sel_a, sel_b = (torch.zeros(shape, dtype=torch.int32, device="cuda") for _ in range(2))
    out_a, out_b = (torch.empty(q.shape, dtype=dt, device="cuda") for _ in range(2))
    ws = None
    for _ in range(2):  # the second call reuses the workspace the first left
        ws = M.mpc_decode_step(qd, cd, sd, kd, vd, sel_a, out_a, cfg, sm_scale=sm, ws=ws)
    M.mpc_select_clusters(qd, cd, sd, sel_b, cfg, Ts=w.keep)
    M.mpc_sparse_decode_attn(qd, kd, vd, sel_b, out_b, cluster_size=w.cluster, sm_scale=sm)
    torch.cuda.synchronize()
    assert torch.equal(sel_a, sel_b)
    assert torch.equal(out_a.view(torch.int16), out_b.view(torch.int16))
    sel_ref, _ = oracle.select_clusters(q, cent, scent, w.dtype, Ts=w.keep, cluster=w.cluster, fanout=w.fanout,
                                        k_super=w.k_super, k_clusters=w.k_clusters, share_period=w.share_period,
                                        group=rule)
    sel_g = sel_a.cpu().numpy()
    _check(w, q, cent, scent, sel_g, sel_ref, rule, "linear")
    ref, _ = oracle.sparse_decode_attn(q, k, v, sel_g, w.dtype, cluster=w.cluster, sm_scale=sm)
    assert_out_close(out_a.double().cpu().numpy(), ref, w.dtype, f"decode step ({rule})")


@pytest.mark.parametrize("L,units,k,m", [(32, 8, 10, 1), (32, 8, 10, 3), (12, 96, 8, 2), (5, 3, 300, 4), (4, 7, 64, 0)])
def test_commonality_matches_oracle_exactly(L, units, k, m):
    import paper_2501_06807_amd as M
    say(f"[commonality] L={L} units={units} k={k} m={m}")
    rng = np.random.default_rng(L * 1000 + units + k + m)
    n = max(2 * k, 24)
    idx = np.stack([np.stack([np.sort(rng.choice(n, k, replace=False)) for _ in range(units)])
                    for _ in range(L)]).astype(np.int32)
    if L > 6:  # some layers repeat their predecessor, so long intersections occur too
        idx[3] = idx[2]
        idx[4] = idx[2]
    ref = oracle.commonality(idx, m)
    out = torch.zeros(units, dtype=torch.float64, device="cuda")
    M.mpc_commonality(torch.from_numpy(idx).cuda(), out, m)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy(), ref)
