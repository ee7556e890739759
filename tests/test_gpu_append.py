"""GPU parity of decode-time cache growth (mpc_append_kv) and of the decode step over a grown cache.

A kept cache of Ts0 rows (a multiple of the cluster size s) sits in buffers with room for more;
one token is appended per decode step for a little over two clusters' worth of steps, so the tail
is sealed into new clusters twice. After every append:
  - the cache state (Ts, n_tail) follows the oracle's rule;
  - the representatives of owner layers equal, bit for bit, the oracle's cluster build over the
    clustered rows [0, Ts), and the slots past the clustered ones stay untouched;
  - the decode step (two calls and one launch, identical bit for bit) matches the oracle: the
    selection with the tie rule, the attention over the selected clusters plus the tail rows.
The appended tokens continue the prompt with the same generator (positions after the kept rows).
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_out_close, bits_to_torch, say, to_f64
from test_gpu_decode import _check_selection

pytestmark = pytest.mark.gpu

# name -> (workload, overrides, similarity)
CASES = {
    "C1-fp32": ("C1", dict(), "linear"),
    "C2-fp16": ("C2", dict(n_layers=4), "linear"),
    "C3-bf16": ("C3", dict(n_layers=6, n_kv_heads=4, n_q_heads=4, keep=1024, k_super=2, k_clusters=6), "linear"),
    # 8 layers x 32 kv heads = 256 units: the one-launch decode step runs over the grown cache
    "C3-bf16-L8": ("C3", dict(n_layers=8, keep=1024, k_super=2, k_clusters=6), "linear"),
    "C5-bf16-gqa": ("C5", dict(n_layers=5, n_kv_heads=2, n_q_heads=8, keep=2048, k_super=2, k_clusters=4),
                    "linear"),
    "C3-bf16-maxprod": ("C3", dict(n_layers=3, n_kv_heads=2, n_q_heads=4, keep=1024, k_super=2, k_clusters=6),
                        "maxprod"),
    "C2-fp16-mean": ("C2", dict(n_layers=3), "mean"),
}


def _owner(w, l):
    return oracle.owner_layer(l, w.share_period, w.share_start) == l


@pytest.mark.parametrize("case", list(CASES))
def test_append_and_decode_over_grown_cache(case):
    name, kw, sim = CASES[case]
    w = synth.get(name).with_(**kw)
    s, Ts0 = w.cluster, w.keep
    assert Ts0 % s == 0
    n_app = 2 * s + 3
    cap = Ts0 + n_app + 5
    say(f"[append] {case}: L={w.n_layers} B={w.batch} Hq={w.n_q_heads} Hkv={w.n_kv_heads} d={w.head_dim} "
        f"{w.dtype} s={s} f={w.fanout} Ts0={Ts0} appends={n_app} capacity={cap} {sim}")
    ks, vs = [], []
    for l in range(w.n_layers):
        k, v = synth.cache_host(w, l, T=Ts0 + n_app)
        ks.append(k)
        vs.append(v)
    k_all, v_all = np.stack(ks), np.stack(vs)

    import paper_2501_06807_amd as M
    dt = synth.torch_dtype(w.dtype)
    path = M.MPCachePath(n_layers=w.n_layers, batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                         head_dim=w.head_dim, dtype=dt, T=Ts0, window=1, keep=Ts0, local_keep=0, cluster=s,
                         fanout=w.fanout, k_super=w.k_super, k_clusters=w.k_clusters, share_period=w.share_period,
                         share_start=w.share_start, similarity=sim, capacity=cap)
    path.k_s[:, :, :, :Ts0] = bits_to_torch(k_all[:, :, :, :Ts0], w.dtype)
    path.v_s[:, :, :, :Ts0] = bits_to_torch(v_all[:, :, :, :Ts0], w.dtype)
    M.mpc_build_clusters(path.k_s, path.cent, path.scent, path.cfg, Ts=Ts0)
    k_new_d = bits_to_torch(np.ascontiguousarray(k_all.transpose(3, 0, 1, 2, 4)), w.dtype)  # [step][L][B][Hkv][d]
    v_new_d = bits_to_torch(np.ascontiguousarray(v_all.transpose(3, 0, 1, 2, 4)), w.dtype)
    sm = 1.0 / math.sqrt(w.head_dim)
    sp = synth.spec(w)
    owners = [l for l in range(w.n_layers) if _owner(w, l)]
    Ts, nt = Ts0, 0
    seals = 0
    for e in range(n_app):
        path.append(k_new_d[Ts0 + e], v_new_d[Ts0 + e])
        Ts_ref, nt_ref = oracle.append_state(Ts, nt, s)
        seals += Ts_ref != Ts
        Ts, nt = Ts_ref, nt_ref
        assert (path.Ts, path.n_tail) == (Ts, nt)
        assert Ts + nt == Ts0 + e + 1
        # representatives: the oracle's build over the clustered rows
        C = Ts // s
        S = -(-C // w.fanout)
        cent_ref, scent_ref = oracle.build_clusters(k_all[:, :, :, :Ts], w.dtype, cluster=s, fanout=w.fanout,
                                                    alpha=0.6, share_period=w.share_period,
                                                    share_start=w.share_start, similarity=sim)
        cent_g, scent_g = path.cent.cpu().numpy(), path.scent.cpu().numpy()
        for l in owners:
            np.testing.assert_array_equal(cent_g[l, :, :, :C], cent_ref[l])
            np.testing.assert_array_equal(scent_g[l, :, :, :S], scent_ref[l])
        assert not cent_g[:, :, :, C:].any() and not scent_g[:, :, :, S:].any()
        # the cache rows: kept rows and appended rows in order
        if e in (0, n_app - 1):
            got = path.k_s[:, :, :, :Ts + nt].cpu()
            exp = bits_to_torch(k_all[:, :, :, :Ts + nt], w.dtype, "cpu")
            assert torch.equal(got.view(torch.int16 if dt != torch.float32 else torch.int32),
                               exp.view(torch.int16 if dt != torch.float32 else torch.int32))
        # decode step over the grown cache
        q = synth.dq_host(sp, e, w.dtype)
        qd = bits_to_torch(q, w.dtype)
        path.decode(qd)
        torch.cuda.synchronize()
        sel0, sc0, out0, lse0 = (t.cpu().clone() for t in (path.sel, path.sel_score, path.out, path.lse))
        path.decode_fused(qd)
        torch.cuda.synchronize()
        assert torch.equal(sel0, path.sel.cpu()) and torch.equal(sc0, path.sel_score.cpu())
        assert torch.equal(out0.float(), path.out.cpu().float()) and torch.equal(lse0, path.lse.cpu())
        sel_ref, _ = oracle.select_clusters(q, cent_ref, scent_ref, w.dtype, Ts=Ts, cluster=s, fanout=w.fanout,
                                            k_super=w.k_super, k_clusters=w.k_clusters,
                                            share_period=w.share_period, share_start=w.share_start,
                                            similarity=sim)
        w_now = w.with_(keep=Ts)
        swaps = _check_selection(w_now, 0, q, cent_ref, scent_ref, sel0.numpy(), sel_ref.copy(), sc0.numpy(), sim)
        ref, lse_ref = oracle.sparse_decode_attn(q, k_all[:, :, :, :Ts + nt], v_all[:, :, :, :Ts + nt],
                                                 np.ascontiguousarray(sel0.numpy()), w.dtype, cluster=s,
                                                 sm_scale=sm, n_tail=nt)
        worst = assert_out_close(to_f64(out0), ref, w.dtype, f"{case} step {e}")
        np.testing.assert_allclose(lse0.numpy(), lse_ref, rtol=1e-5, atol=1e-5)
        if e % 16 == 0 or e == n_app - 1:
            say(f"  step {e}: Ts={Ts} n_tail={nt} tie swaps {swaps} worst relative error {worst:.2e}")
    assert seals == 2
