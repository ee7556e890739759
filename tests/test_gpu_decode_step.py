"""GPU parity of the one-launch decode step (mpc_decode_step).

The step must give bit for bit what mpc_select_clusters followed by mpc_sparse_decode_attn give,
and both are checked against the oracle: the selection with the tie rule, the attention output
recomputed by the oracle from the selection the GPU made. Cases are chosen so that both one-launch
kernels run: the self-selecting one (at most one (layer, sequence, kv head) unit per compute unit:
every workgroup computes its owner head's selection) and the claiming one (more units: the first
consumer of an owner head selects, the others wait for it), with per-head and per-wave selection,
owners inside and before the block, and the sequential fallback of small blocks.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import assert_out_close, bits_to_torch, random_sel, say, to_f64
from test_gpu_decode import _check_selection

pytestmark = pytest.mark.gpu

# name -> (workload, overrides, layer0)
CASES = {
    # 8 layers x 32 kv heads = 256 units (self-selecting); owners 0, 1, 2, 6
    "C3-L8": ("C3", dict(n_layers=8), 0),
    # 16 layers: 512 units (claiming); owners 0, 1, 2, 6, 10, 14
    "C3-L16": ("C3", dict(n_layers=16), 0),
    # layers 3..10: layers 3-5 are owned by layer 2 (before the block) -> their selection is an input
    "C3-L8@3": ("C3", dict(n_layers=8), 3),
    # 512 owner heads -> one wave per head
    "C4-L8": ("C4", dict(n_layers=8, keep=2048, k_super=4, k_clusters=8), 0),
    # GQA group 4, 32 layers x 8 kv heads = 256 units
    "C5-L32": ("C5", dict(keep=8192, k_super=8), 0),
    # small blocks: the two kernels in sequence
    "C1": ("C1", dict(), 0),
    "C2": ("C2", dict(), 0),
    # the other similarity measures in one launch (four heads per group for the bound)
    "C5-L32-maxprod": ("C5", dict(keep=8192, k_super=8), 0, "maxprod"),
    "C3-L8-mean": ("C3", dict(n_layers=8), 0, "mean"),
    # clusters of 4 tokens, fan-out 2: 1280 owner heads (one wave each), 2048 attention units
    "X1-L8": ("X1", dict(n_layers=8), 0),
    # the dynamic ratio read against the prompt length (40 clusters per selection)
    "C5-T-L32": ("C5-T", dict(keep=8192, k_super=8), 0),
    # degenerate budgets: one partial cluster of 10 tokens (one super-cluster, three of its four
    # member slots empty); every cluster of every super-cluster selected (256 units, self-selecting)
    "C2-one-cluster": ("C2", dict(keep=10, k_super=1, k_clusters=1), 0),
    "C2-all-selected": ("C2", dict(n_layers=32, n_q_heads=8, n_kv_heads=8, keep=512, k_super=8, k_clusters=32), 0),
    # the most layers one call takes (256): one kv head -> 256 units (self-selecting); two kv heads
    # from layer 5 -> 512 units (claiming), layer 5 owned by layer 4 before the block
    "C2-L256": ("C2", dict(n_layers=256, n_q_heads=1, n_kv_heads=1, keep=512), 0),
    "C2-L256x2@5": ("C2", dict(n_layers=256, n_q_heads=2, n_kv_heads=2, keep=512), 5),
}


def _setup(case):
    name, kw, layer0 = CASES[case][:3]
    sim = CASES[case][3] if len(CASES[case]) > 3 else "linear"
    w = synth.get(name).with_(**kw)
    ks, vs = [], []
    for l in range(w.n_layers):
        k, v = synth.cache_host(w, layer0 + l, T=w.keep)
        ks.append(k)
        vs.append(v)
    k, v = np.stack(ks), np.stack(vs)
    cent, scent = oracle.build_clusters(k, w.dtype, cluster=w.cluster, fanout=w.fanout, alpha=0.6, layer0=layer0,
                                        share_period=w.share_period, similarity=sim)
    return w, layer0, k, v, cent, scent, sim


def _queries(w, layer0, step):
    sp = synth.spec(w, n_layers=layer0 + w.n_layers)
    return synth.dq_host(sp, step, w.dtype)[layer0:]


def _sync_state(ws, n_heads):
    """Error word, and the per-owner-head state and consumer words (256-byte aligned regions)."""
    words = ws.view(torch.int32).cpu()
    region = -(-n_heads * 4 // 256) * 256 // 4
    return int(words[0]), words[64:64 + 2 * region]


@pytest.mark.parametrize("case", list(CASES))
def test_decode_step_equals_two_calls_and_oracle(case):
    w, layer0, k, v, cent, scent, sim = _setup(case)
    import paper_2501_06807_amd as M
    units = w.n_layers * w.batch * w.n_kv_heads
    say(f"[step] {case}: L={w.n_layers}@{layer0} B={w.batch} Hq={w.n_q_heads} Hkv={w.n_kv_heads} Ts={w.keep} "
        f"s={w.cluster} f={w.fanout} k_super={w.k_super} k_clusters={w.k_clusters} units={units}")
    dt = synth.torch_dtype(w.dtype)
    cfg = M.select_cfg(w.cluster, w.fanout, w.k_super, w.k_clusters, 0.6, w.share_period, similarity=sim)
    kd, vd = bits_to_torch(k, w.dtype), bits_to_torch(v, w.dtype)
    cent_d, scent_d = torch.from_numpy(cent).cuda(), torch.from_numpy(scent).cuda()
    shape_sel = (w.n_layers, w.batch, w.n_kv_heads, w.k_clusters)
    shape_out = (w.n_layers, w.batch, w.n_q_heads, w.head_dim)
    sm = 1.0 / math.sqrt(w.head_dim)
    dims = M.dims_of(torch.empty(shape_out, dtype=dt), kd, layer0)
    ws = M.workspace(M.workspace_bytes(M.MPC_OP_DECODE_STEP, dims, w.keep, cfg), "cuda")
    ws_attn = M.workspace(M.workspace_bytes(M.MPC_OP_DECODE_ATTN, dims, w.keep), "cuda")
    # layers owned before the block arrive with a selection made upstream (here: random, ascending)
    C = -(-w.keep // w.cluster)
    sel_in = random_sel(np.random.default_rng(11), w.n_layers * w.batch * w.n_kv_heads, C,
                        w.k_clusters).reshape(shape_sel)
    owners = [l for l in range(w.n_layers)
              if oracle.owner_layer(layer0 + l, w.share_period, w.share_start) == layer0 + l]
    n_heads = len(owners) * w.batch * w.n_kv_heads
    for step in range(3):
        q = _queries(w, layer0, step)
        qd = bits_to_torch(q, w.dtype)
        sel_ref, _ = oracle.select_clusters(q, cent, scent, w.dtype, Ts=w.keep, cluster=w.cluster, fanout=w.fanout,
                                            k_super=w.k_super, k_clusters=w.k_clusters, layer0=layer0,
                                            share_period=w.share_period, sel_in=sel_in, similarity=sim)
        outs = []
        for fused in (False, True):
            sel = torch.from_numpy(np.ascontiguousarray(sel_ref)).cuda()
            for l in range(w.n_layers):
                if oracle.owner_layer(layer0 + l, w.share_period, w.share_start) >= layer0:
                    sel[l] = -7
            sc = torch.zeros(shape_sel, dtype=torch.float32, device="cuda")
            out = torch.full(shape_out, 3.0, dtype=dt, device="cuda")
            lse = torch.zeros(shape_out[:-1], dtype=torch.float32, device="cuda")
            if fused:
                M.mpc_decode_step(qd, cent_d, scent_d, kd, vd, sel, out, cfg, sm_scale=sm, sel_score=sc, lse=lse,
                                  ws=ws, layer0=layer0)
            else:
                M.mpc_select_clusters(qd, cent_d, scent_d, sel, cfg, Ts=w.keep, sel_score=sc, layer0=layer0)
                M.mpc_sparse_decode_attn(qd, kd, vd, sel, out, cluster_size=w.cluster, sm_scale=sm, lse=lse,
                                         ws=ws_attn, layer0=layer0)
            torch.cuda.synchronize()
            outs.append((sel.cpu(), sc.cpu(), out.cpu(), lse.cpu()))
        (s0, c0, o0, l0), (s1, c1, o1, l1) = outs
        assert torch.equal(s0, s1), "selection differs from the two-call path"
        assert torch.equal(c0, c1), "selection scores differ from the two-call path"
        assert torch.equal(o0.view(torch.int16 if dt != torch.float32 else torch.int32),
                           o1.view(torch.int16 if dt != torch.float32 else torch.int32)), "output differs"
        assert torch.equal(l0, l1), "lse differs"
        # no unit gave up waiting; every head's state and consumer count back at zero
        err, words = _sync_state(ws, n_heads)
        assert err == 0 and not words.any(), f"error {err}, non-zero head words {words.nonzero().flatten()[:8]}"
        # oracle: selection (tie rule) and attention over the selection the GPU made
        sel_g = s1.numpy()
        swaps = _check_selection(w, layer0, q, cent, scent, sel_g, sel_ref.copy(), c1.numpy(), sim)
        ref, lse_ref = oracle.sparse_decode_attn(q, k, v, np.ascontiguousarray(sel_g), w.dtype, cluster=w.cluster,
                                                 sm_scale=sm)
        worst = assert_out_close(to_f64(o1), ref, w.dtype, case)
        np.testing.assert_allclose(l1.numpy(), lse_ref, rtol=1e-5, atol=1e-5)
        say(f"  step {step}: identical to two calls; tie swaps {swaps}; worst relative error {worst:.2e}")


def test_decode_step_unit_that_gives_up_is_reported():
    """A selection that is never published (forced from the host: one owner head's state word is
    set to "being selected" before the launch, which no workgroup then computes) makes its consuming
    units give up after their bounded poll: the error word reports it, those units' outputs are NaN,
    every other unit matches the normal step, and the head's words are back at zero afterwards.
    Every workgroup exits normally."""
    w, layer0, k, v, cent, scent, sim = _setup("C3-L16")  # 512 units: the claiming kernel
    import paper_2501_06807_amd as M
    say("[step give-up] C3-L16: owner head (layer 2, b 0, h 0) marked claimed before the launch")
    dt = synth.torch_dtype(w.dtype)
    cfg = M.select_cfg(w.cluster, w.fanout, w.k_super, w.k_clusters, 0.6, w.share_period, similarity=sim)
    kd, vd = bits_to_torch(k, w.dtype), bits_to_torch(v, w.dtype)
    cent_d, scent_d = torch.from_numpy(cent).cuda(), torch.from_numpy(scent).cuda()
    shape_sel = (w.n_layers, w.batch, w.n_kv_heads, w.k_clusters)
    shape_out = (w.n_layers, w.batch, w.n_q_heads, w.head_dim)
    sm = 1.0 / math.sqrt(w.head_dim)
    dims = M.dims_of(torch.empty(shape_out, dtype=dt), kd, layer0)
    ws = M.workspace(M.workspace_bytes(M.MPC_OP_DECODE_STEP, dims, w.keep, cfg), "cuda")
    qd = bits_to_torch(_queries(w, layer0, 0), w.dtype)
    owners = [l for l in range(w.n_layers) if oracle.owner_layer(l, w.share_period, w.share_start) == l]
    n_heads = len(owners) * w.batch * w.n_kv_heads

    def step():
        sel = torch.zeros(shape_sel, dtype=torch.int32, device="cuda")
        out = torch.zeros(shape_out, dtype=dt, device="cuda")
        lse = torch.zeros(shape_out[:-1], dtype=torch.float32, device="cuda")
        M.mpc_decode_step(qd, cent_d, scent_d, kd, vd, sel, out, cfg, sm_scale=sm, lse=lse, ws=ws)
        torch.cuda.synchronize()
        return out.float().cpu(), lse.cpu()

    o_ref, l_ref = step()
    assert M.mpc_decode_step_status(ws) == 0
    # owner index 2 is layer 2, whose head (b 0, h 0) serves layers 2..5
    o_idx = owners.index(2)
    head = (o_idx * w.batch + 0) * w.n_kv_heads + 0
    ws.view(torch.int32)[64 + head] = 1
    torch.cuda.synchronize()
    o_bad, l_bad = step()
    assert M.mpc_decode_step_status(ws) == 1
    layers = [l for l in range(w.n_layers) if oracle.owner_layer(l, w.share_period, w.share_start) == 2]
    G = w.group
    hit = torch.zeros(shape_out[:-1], dtype=torch.bool)
    for l in layers:
        hit[l, 0, 0:G] = True
    assert torch.isnan(o_bad[hit]).all() and torch.isnan(l_bad[hit]).all()
    assert torch.equal(o_bad[~hit], o_ref[~hit]) and torch.equal(l_bad[~hit], l_ref[~hit])
    err, words = _sync_state(ws, n_heads)
    assert err == 1 and not words.any()
    # clearing the word; the next step is normal again
    assert M.mpc_decode_step_status(ws, clear=True) == 1
    assert M.mpc_decode_step_status(ws) == 0
    o2, l2 = step()
    assert torch.equal(o2, o_ref) and torch.equal(l2, l_ref)
    assert M.mpc_decode_step_status(ws) == 0
    say(f"  {int(hit.sum())} q-head outputs NaN after the give-up; error word cleared; next step identical")
