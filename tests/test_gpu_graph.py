"""GPU: the decode step and the prefill captured as HIP graphs (torch.cuda.CUDAGraph) and replayed.
Every replay equals the eager call bit for bit. Between replays the test refills the input
buffers, clears the outputs with eager kernels of its own and synchronises."""
import pytest
import torch

import synth
from gpu_util import say

pytestmark = pytest.mark.gpu

CASES = {
    # 144 units: the one-launch step takes the two kernels in turn, the attention split over workgroups
    "C2": ("C2", {}),
    # 256 units: the self-selecting one-launch kernel
    "C3-L8": ("C3", dict(n_layers=8)),
    # 512 units: the claiming one-launch kernel (its workspace words back at zero after every launch)
    "C3-L16": ("C3", dict(n_layers=16)),
}


def _inputs(w, steps=3):
    sp = synth.spec(w)
    rope = synth.rope_dev(w.T, w.head_dim, w.rope_base) if w.rope else None
    q_win = synth.qwin_dev(sp, w.dtype, 0, w.n_layers, rope)
    k, v = synth.kv_dev(sp, w.dtype, 0, w.n_layers, q_win, rope)
    return q_win, k, v, [synth.dq_dev(sp, w.dtype, e) for e in range(steps)]


def _path(w, **kw):
    import paper_2501_06807_amd as M
    return M.MPCachePath(n_layers=w.n_layers, batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                         head_dim=w.head_dim, dtype=synth.torch_dtype(w.dtype), T=w.T, window=w.window,
                         keep=w.keep, local_keep=w.local_keep, cluster=w.cluster, fanout=w.fanout,
                         k_super=w.k_super, k_clusters=w.k_clusters, share_period=w.share_period,
                         share_start=w.share_start, **kw)


def _bits(t):
    return t.view(torch.int32) if t.dtype == torch.float32 else t.view(torch.int16)


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("case", list(CASES))
def test_decode_graph_replays_equal_eager(case, fused):
    name, over = CASES[case]
    w = synth.get(name).with_(**over)
    say(f"[graph decode] {case} fused={fused} L={w.n_layers} Hkv={w.n_kv_heads} Ts={w.keep}")
    q_win, k, v, qs = _inputs(w)
    path = _path(w)
    path.prefill(q_win, k, v)
    step = path.decode_fused if fused else path.decode
    ref = []
    for q in qs:
        step(q)
        torch.cuda.synchronize()
        ref.append((path.sel.clone(), path.sel_score.clone(), path.out.clone(), path.lse.clone()))
    q_buf = qs[0].clone()
    g = path.capture(step, q_buf)
    for rep in range(2):
        for i, q in enumerate(qs):
            q_buf.copy_(q)
            path.sel.fill_(-1)
            path.sel_score.zero_()
            path.out.fill_(float("nan"))
            path.lse.zero_()
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            sel, sc, out, lse = ref[i]
            assert torch.equal(path.sel, sel), (rep, i, "selection")
            assert torch.equal(_bits(path.sel_score), _bits(sc)), (rep, i, "selection scores")
            assert torch.equal(_bits(path.out), _bits(out)), (rep, i, "output")
            assert torch.equal(_bits(path.lse), _bits(lse)), (rep, i, "lse")
    say("  6 replays equal to the eager steps")


@pytest.mark.parametrize("case", ["C2", "C3-L8"])
def test_prefill_graph_replays_equal_eager(case):
    name, over = CASES[case]
    w = synth.get(name).with_(**over)
    say(f"[graph prefill] {case} L={w.n_layers} T={w.T} W={w.window} keep={w.keep}")
    q_win, k, v, qs = _inputs(w, steps=1)
    path = _path(w, keep_scores=True)
    outs = lambda: [path.kept, path.k_s, path.v_s, path.cent, path.scent, path.token_score, path.row_lse]
    path.prefill(q_win, k, v)
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs()]
    g = path.capture(path.prefill, q_win, k, v)
    for rep in range(3):
        for t in outs():
            t.zero_()
        path.decode(qs[0])  # eager work of the program between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for n, (t, r) in enumerate(zip(outs(), ref)):
            assert torch.equal(_bits(t) if t.dtype != torch.int32 else t, _bits(r) if r.dtype != torch.int32 else r), \
                (rep, n)
    say("  3 replays equal to the eager prefill")


def test_noalloc_eviction_graph_replays_equal_eager():
    """The static eviction without allocation, captured as a graph (its scratch address is looked
    up by an eager call first): every replay equals the eager workspace call."""
    import math
    import paper_2501_06807_amd as M
    w = synth.get("C2").with_(n_layers=4)
    say(f"[graph noalloc] C2 L={w.n_layers} T={w.T} W={w.window} keep={w.keep}")
    q_win, k, v, _ = _inputs(w, steps=1)
    L, B, Hkv = w.n_layers, w.batch, w.n_kv_heads
    dt = synth.torch_dtype(w.dtype)
    kw = dict(keep=w.keep, local_keep=w.local_keep, sm_scale=1.0 / math.sqrt(w.head_dim), share_period=w.share_period,
              share_start=w.share_start)

    def buffers():
        return dict(kept=torch.zeros((L, B, Hkv, w.keep), dtype=torch.int32, device="cuda"),
                    k_out=torch.zeros((L, B, Hkv, w.keep, w.head_dim), dtype=dt, device="cuda"),
                    v_out=torch.zeros((L, B, Hkv, w.keep, w.head_dim), dtype=dt, device="cuda"),
                    score=torch.zeros((L, B, Hkv, w.T), dtype=torch.float32, device="cuda"),
                    lse=torch.zeros((L, B, w.n_q_heads, w.window), dtype=torch.float32, device="cuda"))

    def call(o, noalloc):
        fn = M.mpc_static_evict_noalloc if noalloc else M.mpc_static_evict
        fn(q_win, k, v, o["kept"], o["k_out"], o["v_out"], token_score=o["score"], row_lse=o["lse"], **kw)

    ref = buffers()
    call(ref, False)
    got = buffers()
    call(got, True)  # eager: the scratch address of this device is looked up here
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(got, True)
    for rep in range(3):
        for t in got.values():
            t.zero_()
        call(buffers(), False)  # eager work of the program between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for n in ref:
            a, b = got[n], ref[n]
            assert torch.equal(a if a.dtype == torch.int32 else _bits(a), b if b.dtype == torch.int32 else _bits(b)), \
                (rep, n)
    say("  3 replays equal to the eager workspace call")
