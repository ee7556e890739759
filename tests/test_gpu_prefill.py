"""GPU: the one-call prefill (static eviction, then cluster representatives of the kept rows, the
selection owners' rows gathered inside the build) gives the results of the two calls it replaces
bit for bit, and its representatives are the oracle's over the rows it kept."""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import bits_to_torch, say, torch_to_bits

pytestmark = pytest.mark.gpu


def _inputs(w, layer0):
    parts = [synth.prefill_host(w, layer0 + l) for l in range(w.n_layers)]
    return tuple(np.stack([p[i] for p in parts]) for i in range(3))


def _buffers(w, cap, sim, kept_in):
    L, B, Hkv, d = w.n_layers, w.batch, w.n_kv_heads, w.head_dim
    R = 2 if sim == "maxprod" else 1
    C = -(-cap // w.cluster)
    S = -(-C // w.fanout)
    kept = (torch.zeros((L, B, Hkv, w.keep), dtype=torch.int32, device="cuda") if kept_in is None
            else torch.from_numpy(kept_in).cuda())
    k_out = torch.zeros((L, B, Hkv, cap, d), dtype=synth.torch_dtype(w.dtype), device="cuda")
    return dict(kept=kept, k_out=k_out, v_out=torch.zeros_like(k_out),
                cent=torch.zeros((L, B, Hkv, C, R, d), dtype=torch.float32, device="cuda"),
                scent=torch.zeros((L, B, Hkv, S, R, d), dtype=torch.float32, device="cuda"),
                score=torch.zeros((L, B, Hkv, w.T), dtype=torch.float32, device="cuda"),
                lse=torch.zeros((L, B, w.n_q_heads, w.window), dtype=torch.float32, device="cuda"))


def _run(w, qw, k, v, *, sim, layer0, cap, sel_period, kept_in, fused):
    import paper_2501_06807_amd as M
    dt = w.dtype
    out = _buffers(w, cap, sim, kept_in)
    cfg = M.select_cfg(w.cluster, w.fanout, 1, 1, 0.6, sel_period, w.share_start, sim)
    q_d, k_d, v_d = bits_to_torch(qw, dt), bits_to_torch(k, dt), bits_to_torch(v, dt)
    kw = dict(keep=w.keep, local_keep=w.local_keep, sm_scale=1.0 / math.sqrt(w.head_dim), layer0=layer0,
              share_period=w.share_period, share_start=w.share_start, token_score=out["score"],
              row_lse=out["lse"])
    if fused:
        M.mpc_prefill(q_d, k_d, v_d, out["kept"], out["k_out"], out["v_out"], out["cent"], out["scent"], cfg, **kw)
    else:
        M.mpc_static_evict(q_d, k_d, v_d, out["kept"], out["k_out"], out["v_out"], **kw)
        M.mpc_build_clusters(out["k_out"], out["cent"], out["scent"], cfg, Ts=w.keep, layer0=layer0)
    torch.cuda.synchronize()
    return {n: (torch_to_bits(t, dt) if n in ("k_out", "v_out") else t.cpu().numpy()) for n, t in out.items()}


CASES = {
    # name: (workload, overrides, similarity, layer0, extra kv rows, selection sharing period)
    "C1-linear": ("C1", {}, "linear", 0, 0, None),
    "C2-maxprod": ("C2", dict(n_layers=4), "maxprod", 0, 0, None),
    "C2-mean-capacity": ("C2", dict(n_layers=3, T=1000, window=200, keep=500), "mean", 0, 37, None),
    "C5-gqa": ("C5", dict(n_layers=2, n_q_heads=8, n_kv_heads=2, T=4096, window=409, keep=1024,
                          hh_count=8, hh_hi=4096 - 32), "linear", 0, 0, None),
    "X1": ("X1", dict(n_layers=3, batch=2, n_q_heads=4, n_kv_heads=4), "linear", 0, 0, None),
    # every layer builds its own representatives while pairs of layers share one kept set
    "C2-sel-unshared": ("C2", dict(n_layers=4, T=1000, window=200, keep=480), "linear", 0, 0, 1),
    # kept sets unshared, representatives shared by pairs of layers
    "C2-evict-unshared": ("C2", dict(n_layers=4, T=1000, window=200, keep=480, share_period=1), "maxprod", 0,
                          0, 2),
    # the block's first layer is owned by a layer before it: its kept set arrives in place
    "C2-owner-before": ("C2", dict(n_layers=3, T=700, window=140, keep=320, n_q_heads=4, n_kv_heads=4),
                        "linear", 3, 0, None),
    # every token kept, the window the whole prompt, no recent tokens kept by rule
    "C2-keep-all": ("C2", dict(n_layers=3, T=300, window=300, keep=300, local_keep=0), "maxprod", 0, 0, None),
    # the most layers one call takes (256): the gather's mask of layers left to the build spans four
    # 64-layer words; kept sets shared by threes, representatives by fives
    "C2-L256": ("C2", dict(n_layers=256, n_q_heads=2, n_kv_heads=1, T=160, window=32, keep=80, share_period=3),
                "linear", 0, 0, 5),
}


@pytest.mark.parametrize("name", list(CASES))
def test_prefill_equals_evict_then_build(name):
    base, over, sim, layer0, extra, sel_period = CASES[name]
    w = synth.get(base).with_(**over)
    sel_period = w.share_period if sel_period is None else sel_period
    say(f"prefill {name}: L={w.n_layers} B={w.batch} Hq/Hkv={w.n_q_heads}/{w.n_kv_heads} T={w.T} keep={w.keep} "
        f"s={w.cluster} f={w.fanout} {sim} layer0={layer0}")
    qw, k, v = _inputs(w, layer0)
    kept_in = None
    if layer0 > 0:  # the preceding owner's kept set, from the oracle
        wp = w.with_(n_layers=1)
        qp, kp, vp = _inputs(wp, layer0 - 1)
        kept_in = np.repeat(oracle.static_evict(qp, kp, vp, w.dtype, keep=w.keep, local_keep=w.local_keep,
                                                sm_scale=1.0 / math.sqrt(w.head_dim))[0], w.n_layers, axis=0)
    cap = w.keep + extra
    args = dict(sim=sim, layer0=layer0, cap=cap, sel_period=sel_period, kept_in=kept_in)
    two = _run(w, qw, k, v, fused=False, **args)
    one = _run(w, qw, k, v, fused=True, **args)
    for n in ("kept", "score", "lse", "cent", "scent"):
        np.testing.assert_array_equal(one[n], two[n], err_msg=n)
    for n in ("k_out", "v_out"):
        np.testing.assert_array_equal(one[n][:, :, :, :w.keep], two[n][:, :, :, :w.keep], err_msg=n)
    # every layer's kept rows are a bit copy of the prompt rows
    kept = one["kept"]
    for l in range(w.n_layers):
        for b in range(w.batch):
            for h in range(w.n_kv_heads):
                np.testing.assert_array_equal(one["k_out"][l, b, h, :w.keep], k[l, b, h, kept[l, b, h]])
                np.testing.assert_array_equal(one["v_out"][l, b, h, :w.keep], v[l, b, h, kept[l, b, h]])
    # the representatives of the selection's owner layers are the oracle's over the kept rows
    cent_r, scent_r = oracle.build_clusters(one["k_out"][:, :, :, :w.keep], w.dtype, cluster=w.cluster,
                                            fanout=w.fanout, alpha=0.6, layer0=layer0, share_period=sel_period,
                                            share_start=w.share_start, similarity=sim)
    C, S = cent_r.shape[3], scent_r.shape[3]
    shape = (w.n_layers, w.batch, w.n_kv_heads)
    cent_g = one["cent"][:, :, :, :C].reshape(shape + cent_r.shape[3:])
    scent_g = one["scent"][:, :, :, :S].reshape(shape + scent_r.shape[3:])
    owners = [l for l in range(w.n_layers)
              if oracle.owner_layer(layer0 + l, sel_period, w.share_start) == layer0 + l]
    assert owners
    np.testing.assert_array_equal(cent_g[owners], cent_r[owners])
    np.testing.assert_array_equal(scent_g[owners], scent_r[owners])
    others = [l for l in range(w.n_layers) if l not in owners]
    assert not np.any(one["cent"][others]) and not np.any(one["scent"][others])
