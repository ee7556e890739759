#!/usr/bin/env python3
"""Benchmark of the MPCache hot path on one MI355X.

One timed step = one full pass of the path over one batch of synthetic input already resident in
HBM: look-once static eviction of the prompt cache (window scoring, top-k, gather), cluster
representatives, then every decode step of the workload (two-level selection with layer sharing +
sparse attention over all layers). The reported metric is the decode step's latency per layer
(select + attention), measured with HIP events on the stream the kernels run on, with its
effective HBM bandwidth against the 8 TB/s peak. Prefill figures are reported beside it, and so is
the decode step in the other mode (two kernels, or one launch of mpc_decode_step). Measured
ceilings give the fractions a scale: a random-order chunk read (the attention's access pattern) over
2 GiB and over exactly the attention's bytes of each workload (one launch, fixed costs included), a
matrix-core throughput kernel, a device copy; the CPU oracle is timed on a bounded sample, on all
host threads and on one.

Prints one JSON line. Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload C4]
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-step select+sparse-attn latency (µs/layer) & achieved HBM GB/s vs peak"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "fp16": 2500.0, "fp32": 157.3}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=3)
    p.add_argument("--warmup", type=int, default=1)
    p.add_argument("--workload", default="C4")
    p.add_argument("--decode-steps", type=int, default=None, help="decode steps per pass (default: workload's)")
    p.add_argument("--decode-mode", choices=("auto", "split", "fused"), default="auto",
                   help="timed decode step: selection and attention as two kernels (split) or one launch of "
                        "mpc_decode_step (fused); auto (default): one launch when the block has at most one "
                        "(layer, sequence, kv head) unit per compute unit, where every workgroup selects for its "
                        "own unit, else two kernels")
    p.add_argument("--similarity", choices=("linear", "maxprod", "mean"), default="linear",
                   help="cluster similarity: the paper's linear form (default), the max-product bound (Eq. 2) "
                        "or the cluster average")
    p.add_argument("--group", choices=("sum", "max", "head"), default="sum",
                   help="grouped q-heads: one selection per kv head scored by the sum (default) or the maximum of "
                        "its q-heads' similarities, or one selection per q-head")
    p.add_argument("--extra", default="C3,C5,C5-T",
                   help="comma-separated workloads whose decode step is also measured (same pass structure, "
                        "reported under other_workloads; C5-T: the level-2 budget read against the prompt); "
                        "'' for none")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--copy-calibration", action="store_true",
                   help="accepted for recorded profiling commands; the 1 GiB reference copy always runs")
    return p.parse_args()


DECODE_STEP_SOURCES = ("fused.hip", "fused.h", "decode_dev.h", "select_dev.h", "decode_attn.h", "select.h",
                       "common.h")
SPARSE_DECODE_SOURCES = ("decode_attn.hip", "decode_attn.h", "decode_dev.h", "common.h")


NUM_CU = 256  # compute units of an MI355X


def resolve_mode(mode, path):
    """The decode mode a run times: `auto` takes the one launch where mpc_decode_step runs its
    self-selecting kernel (at most one attention unit per compute unit: faster there than two
    kernels), and the two kernels elsewhere (faster than the claiming one-launch kernel)."""
    if mode != "auto":
        return mode
    return "fused" if path.L * path.B * path.Hsel <= NUM_CU else "split"


def source_digest(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2501_06807_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload, digest):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it was taken on the
    current kernel source; None otherwise."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_digest") != digest:
        return None
    return rec.get("bytes_per_launch")


def decode_bytes(w, owners, sel, C, S, rep_rows=1):
    """Algorithmic bytes of one decode step: reads of representatives (rep_rows rows of d floats
    each), queries, gathered K/V rows and selections; writes of selections and outputs. Every
    byte is counted once. sel [L][B][H][k] has one list per kv head or one per q-head."""
    d, e = w.head_dim, w.elt
    H = sel.shape[2]  # selection lists per (layer, sequence)
    Gu = w.n_q_heads // H  # q-heads per list
    n_own = len(owners)
    sel_read = n_own * w.batch * H * ((S + w.k_super * w.fanout) * rep_rows * d * 4 + Gu * d * e)
    sel_write = w.n_layers * w.batch * H * w.k_clusters * 8
    # exact gathered token count (a partial last cluster holds fewer rows)
    last = w.keep - (C - 1) * w.cluster
    n_tok = int(w.n_layers * w.batch * H * w.k_clusters * w.cluster - (sel == C - 1).sum() * (w.cluster - last))
    attn_read = n_tok * d * e * 2 + w.n_layers * w.batch * (w.n_q_heads * d * e + H * w.k_clusters * 4)
    attn_write = w.n_layers * w.batch * w.n_q_heads * (d * e + 4)
    return sel_read + sel_write, attn_read + attn_write


def measure_read_ceiling(dev, chunk_bytes=16384, per_wg=24, total=2 << 30):
    """Read rate of a kernel that reads every 16 KB chunk of a 2 GiB buffer once, in random order
    (the sparse attention's access pattern: whole clusters of rows): the practical ceiling the
    decode kernels are compared with, beside the published peak."""
    import ctypes

    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2501_06807_amd", "libmpc_ceiling.so"))
    lib.mpc_read_ceiling.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                                     ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    n_chunks = total // chunk_bytes
    grid = n_chunks // per_wg
    buf = torch.empty(total, dtype=torch.uint8, device=dev).fill_(3)
    gen = torch.Generator(device=dev)
    gen.manual_seed(7)
    order = torch.randperm(n_chunks, generator=gen, device=dev, dtype=torch.int32)[:grid * per_wg].contiguous()
    sink = torch.empty(grid * 256, dtype=torch.int32, device=dev)
    st = torch.cuda.current_stream(dev)

    def launch():
        rc = lib.mpc_read_ceiling(buf.data_ptr(), n_chunks, chunk_bytes, order.data_ptr(), grid, per_wg,
                                  sink.data_ptr(), st.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"read-ceiling kernel failed to launch ({rc})")

    launch()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(st)
    for _ in range(5):
        launch()
    b.record(st)
    torch.cuda.synchronize()
    gbs = 5 * grid * per_wg * chunk_bytes / (a.elapsed_time(b) * 1e-3) / 1e9
    del buf, order, sink
    return {"GBps": round(gbs, 1), "frac_of_peak": round(gbs / HBM_PEAK_GBS, 4),
            "note": "every 16 KB chunk of 2 GiB read once in random order, 16-byte non-temporal loads (the "
                    "sparse attention's pattern)"}


def measure_read_time(dev, nbytes, chunk_bytes=16384, total=2 << 30):
    """Time of the same chunk-read kernel reading about `nbytes` (a decode step's attention bytes)
    as 16 KB chunks in random order, the best of three grid shapes (1024 / 2560 / 5120 workgroups
    of four waves), each the per-launch average of five back-to-back launches: what one launch that
    only reads this many bytes the attention's way takes on this GPU, fixed costs included."""
    import ctypes

    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2501_06807_amd", "libmpc_ceiling.so"))
    lib.mpc_read_ceiling.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                                     ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    n_chunks = total // chunk_bytes
    want = max(1, min(n_chunks, round(nbytes / chunk_bytes)))
    buf = torch.empty(total, dtype=torch.uint8, device=dev).fill_(3)
    gen = torch.Generator(device=dev)
    gen.manual_seed(11)
    perm = torch.randperm(n_chunks, generator=gen, device=dev, dtype=torch.int32)
    st = torch.cuda.current_stream(dev)
    best = None
    for g in (1024, 2560, 5120):
        per_wg = max(1, want // g)
        grid = max(1, want // per_wg)
        order = perm[:grid * per_wg].contiguous()
        sink = torch.empty(grid * 256, dtype=torch.int32, device=dev)

        def launch():
            rc = lib.mpc_read_ceiling(buf.data_ptr(), n_chunks, chunk_bytes, order.data_ptr(), grid, per_wg,
                                      sink.data_ptr(), st.cuda_stream)
            if rc != 0:
                raise RuntimeError(f"read kernel failed to launch ({rc})")

        launch()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        for _ in range(5):
            launch()
        b.record(st)
        torch.cuda.synchronize()
        us = a.elapsed_time(b) * 1e3 / 5
        nb = grid * per_wg * chunk_bytes
        if best is None or nb / us > best[0] / best[1]:
            best = (nb, us, grid)
    del buf, perm
    nb, us, grid = best
    return {"bytes": nb, "us": round(us, 3), "GBps": round(nb / us / 1e3, 1), "workgroups": grid}


def measure_mfma_ceiling(dev, grid=2048, iters=2048):
    """bf16 matrix-core throughput of a kernel that does nothing but chains of the 32x32x16
    instruction the scoring passes use (four independent accumulators per wave)."""
    import ctypes

    import torch
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2501_06807_amd", "libmpc_ceiling.so"))
    lib.mpc_mfma_ceiling.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    sink = torch.empty(grid * 256, dtype=torch.float32, device=dev)
    st = torch.cuda.current_stream(dev)

    def launch():
        rc = lib.mpc_mfma_ceiling(grid, iters, sink.data_ptr(), st.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"matrix-core ceiling kernel failed to launch ({rc})")

    launch()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(st)
    for _ in range(3):
        launch()
    b.record(st)
    torch.cuda.synchronize()
    flop = 3.0 * grid * 4 * iters * 4 * 32768
    tf = flop / (a.elapsed_time(b) * 1e-3) / 1e12
    return {"TFLOPs": round(tf, 1), "frac_of_peak": round(tf / MFMA_PEAK_TFLOPS["bf16"], 4),
            "note": "chains of v_mfma_f32_32x32x16_bf16 on registers, 4 accumulators per wave, 8192 waves"}


def prefill_flops(w, n_owner):
    """One causal pass of window scores q_t . k_j (2d flops each) over the owner layers."""
    rows = sum(w.T - w.window + t + 1 for t in range(w.window))
    return n_owner * w.batch * w.n_q_heads * rows * 2 * w.head_dim


def cpu_baseline(w, n_steps_sample, similarity="linear", group="sum", min_seconds=10.0, max_seconds=30.0):
    """The oracle's decode step (selection + sparse attention) on a sample of the workload: one
    sharing block of layers (2..2+P-1), every sequence and head, `n_steps_sample` fresh queries,
    repeated until at least `min_seconds` of CPU work (stopping at the first pass past
    `max_seconds`)."""
    import oracle
    import synth
    layer0 = w.share_start
    n_l = max(1, w.share_period)
    ws = w.with_(n_layers=n_l)
    ks, vs = [], []
    for l in range(n_l):
        k, v = synth.cache_host(w, layer0 + l)
        ks.append(k)
        vs.append(v)
    import numpy as np
    k, v = np.stack(ks), np.stack(vs)
    cent, scent = oracle.build_clusters(k, w.dtype, cluster=w.cluster, fanout=w.fanout, layer0=layer0,
                                        share_period=w.share_period, share_start=w.share_start,
                                        similarity=similarity)
    sp = synth.spec(w, n_layers=layer0 + n_l)
    qs = [synth.dq_host(sp, e, w.dtype)[layer0:] for e in range(n_steps_sample)]
    sm = 1.0 / math.sqrt(w.head_dim)

    def timed(min_s, max_s):
        steps = 0
        t0 = time.perf_counter()
        while True:
            for q in qs:
                sel, _ = oracle.select_clusters(q, cent, scent, w.dtype, Ts=w.keep, cluster=w.cluster,
                                                fanout=w.fanout, k_super=w.k_super, k_clusters=w.k_clusters,
                                                layer0=layer0, share_period=w.share_period,
                                                share_start=w.share_start, similarity=similarity, group=group)
                oracle.sparse_decode_attn(q, k, v, sel, w.dtype, cluster=w.cluster, sm_scale=sm)
                steps += 1
                if time.perf_counter() - t0 > max_s:
                    break
            dt = time.perf_counter() - t0
            if dt >= min_s:
                return dt, steps

    cores = oracle.threads()
    dt, steps = timed(min_seconds, max_seconds)
    oracle.set_threads(1)
    try:
        dt1, steps1 = timed(min_seconds / 3, max_seconds / 3)
    finally:
        oracle.set_threads(cores)
    return {"value": dt / (steps * n_l) * 1e6, "unit": "us/layer", "cores": cores,
            "kind": "oracle", "cpu": cpu_model(),
            "single_core_us_per_layer": round(dt1 / (steps1 * n_l) * 1e6, 1),
            "sample": f"{ws.name}: layers {layer0}..{layer0 + n_l - 1} (one sharing block), all {w.batch} "
                      f"sequences x {w.n_kv_heads} kv heads, {steps} decode steps over {len(qs)} distinct "
                      f"queries (selection + sparse attention), fp64, {dt:.2f} s total on {cores} threads; "
                      f"then {steps1} steps on one thread ({dt1:.2f} s)"}


def cpu_model():
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def commonality(w, path, q, args, M, torch, dev, mk):
    """Commonality score (m = 1, 2, 3) of the per-layer selections made without sharing, and the
    commonality kernel's time."""
    cfg = M.select_cfg(w.cluster, w.fanout, w.k_super, w.k_clusters, 0.6, 1, w.share_start,
                       similarity=args.similarity, group=args.group)
    cent = torch.zeros_like(path.cent)
    scent = torch.zeros_like(path.scent)
    M.mpc_build_clusters(path.k_s, cent, scent, cfg, Ts=w.keep)
    sel = torch.zeros_like(path.sel)
    M.mpc_select_clusters(q, cent, scent, sel, cfg, Ts=w.keep)
    out = torch.zeros(sel.shape[1] * sel.shape[2], dtype=torch.float64, device=dev)
    res = {}
    for m in (1, 2, 3):
        M.mpc_commonality(sel, out, m)
        res[f"m{m}"] = round(out.mean().item(), 4)
    a, b = mk(), mk()
    a.record()
    for _ in range(10):
        M.mpc_commonality(sel, out, 1)
    b.record()
    torch.cuda.synchronize()
    res["kernel_us"] = round(a.elapsed_time(b) / 10 * 1e3, 3)
    res["chance_level"] = round(w.k_clusters / path.C, 4)
    res["note"] = ("mean over (sequence, selection list) of the share of top-k clusters common to m+1 adjacent "
                   "layers, each layer selecting on its own (no sharing); the workloads' decode queries are "
                   "independent across layers, so it stays near chance (k / C)")
    return res


PLANTING = ("sinks k <- k - (k.u)u + 4 sqrt(d) u; heavy hitters k <- 3 sqrt(d) u + 0.3 n, u the unit mean of the "
            "group's window queries (the stated 0.7 q_mean + 0.3 noise makes them less attended than random keys)")


def make_state(w, args, M, synth, dev):
    """Device-resident inputs of one pass (window queries, prompt K/V, decode queries) and the
    preallocated path."""
    sp = synth.spec(w)
    rope = synth.rope_dev(w.T, w.head_dim, w.rope_base) if w.rope else None
    q_win = synth.qwin_dev(sp, w.dtype, 0, w.n_layers, rope)
    k, v = synth.kv_dev(sp, w.dtype, 0, w.n_layers, q_win, rope)
    del rope
    E = args.decode_steps or w.steps
    qs = [synth.dq_dev(sp, w.dtype, e) for e in range(E)]
    path = M.MPCachePath(n_layers=w.n_layers, batch=w.batch, n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads,
                         head_dim=w.head_dim, dtype=synth.torch_dtype(w.dtype), T=w.T, window=w.window,
                         keep=w.keep, local_keep=w.local_keep, cluster=w.cluster, fanout=w.fanout,
                         k_super=w.k_super, k_clusters=w.k_clusters, share_period=w.share_period,
                         share_start=w.share_start, similarity=args.similarity, group=args.group)
    return q_win, k, v, qs, path


def timed_passes(path, q_win, k, v, qs, step_fn, steps, warmup, torch):
    """`warmup` untimed passes, then `steps` timed passes (prefill, then every decode step back to
    back), with HIP events on the launch stream at the pass boundaries and after the prefill.
    Returns (prefill ms per pass, decode µs per step, wall seconds of the timed passes)."""
    E = len(qs)
    mk = lambda: torch.cuda.Event(enable_timing=True)

    def one_pass(ev=None):
        if ev:
            ev[0].record()
        path.prefill(q_win, k, v)
        if ev:
            ev[1].record()
        for e in range(E):
            step_fn(qs[e])
        if ev:
            ev[2].record()

    for _ in range(warmup):
        one_pass()
    torch.cuda.synchronize()
    evs = [(mk(), mk(), mk()) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(steps):
        one_pass(evs[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    pre_ms = [a.elapsed_time(b) for a, b, _ in evs]
    dec_us = sum(b.elapsed_time(c) / E for _, b, c in evs) / steps * 1e3
    return pre_ms, dec_us, wall


def kernel_times(path, qs, torch):
    """Per-launch averages of the selection and the attention kernel on the path's current state:
    each launched once per decode step, back to back, between two HIP events (the attention reads
    each step's own selection)."""
    E = len(qs)
    mk = lambda: torch.cuda.Event(enable_timing=True)

    def step_time(fn):
        a, b = mk(), mk()
        a.record()
        for e in range(E):
            fn(qs[e])
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / E * 1e3

    sels = []
    for e in range(E):
        path.select(qs[e])
        sels.append(path.sel.clone())
    calls = [path.attend_call(sv) for sv in sels]
    state = {"it": iter(())}

    def attend_next(q):
        next(state["it"])(q)

    step_time(path.select)
    sel_us = step_time(path.select)
    for _ in range(2):
        state["it"] = iter(calls)
        att_us = step_time(attend_next)
    return sel_us, att_us


def step_record(w, path, M, args, dec_us, sel_us, att_us):
    """Decode-step figures of one workload: latency per layer, algorithmic bytes, bandwidth."""
    owners = [l for l in range(w.n_layers) if M.owner_layer(l, w.share_period, w.share_start) == l]
    sel_b, att_b = decode_bytes(w, owners, path.sel.cpu().numpy(), path.C, path.S, M.rep_rows(args.similarity))
    gbs = (sel_b + att_b) / (dec_us * 1e-6) / 1e9
    att_gbs = att_b / (att_us * 1e-6) / 1e9
    return {"workload": f"{w.name}", "us_per_step": round(dec_us, 3), "us_per_layer": round(dec_us / w.n_layers, 4),
            "algorithmic_bytes": sel_b + att_b, "achieved_GBps": round(gbs, 1),
            "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4), "select_us": round(sel_us, 3),
            "attention_us": round(att_us, 3), "attention_algorithmic_bytes": att_b,
            "attention_frac_of_hbm_peak": round(att_gbs / HBM_PEAK_GBS, 4)}


def extra_workload(name, args, M, synth, torch, dev):
    """The decode step of another workload, timed with the same pass structure as the headline."""
    w = synth.get(name)
    q_win, k, v, qs, path = make_state(w, args, M, synth, dev)
    torch.cuda.synchronize()
    mode = resolve_mode(args.decode_mode, path)
    step_fn = path.decode_fused if mode == "fused" else path.decode
    pre_ms, dec_us, _ = timed_passes(path, q_win, k, v, qs, step_fn, max(3, args.steps), max(1, args.warmup), torch)
    del q_win, k, v
    sel_us, att_us = kernel_times(path, qs, torch)
    rec = step_record(w, path, M, args, dec_us, sel_us, att_us)
    rec["read_same_bytes"] = measure_read_time(dev, rec["attention_algorithmic_bytes"])
    rec["attention_us_over_read_us"] = round(att_us / rec["read_same_bytes"]["us"], 4)
    rec["decode_mode"] = mode
    rec["prefill_ms_per_pass"] = round(sum(pre_ms) / len(pre_ms), 3)
    rec["decode_steps_per_pass"] = len(qs)
    del path, qs
    torch.cuda.empty_cache()
    return rec


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the path shards by "
              f"(sequence, kv head) with no exchange, and no multi-GPU figure is measured here.",
              file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2501_06807_amd as M
    import synth

    w = synth.get(args.workload)
    E = args.decode_steps or w.steps
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    # measured stream-copy ceiling: a 1 GiB device-to-device copy (read + write bytes); with
    # --copy-calibration it is also the reference kernel for HBM counter scaling
    src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(2):
        dst.copy_(src)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(5):
        dst.copy_(src)
    c1.record()
    torch.cuda.synchronize()
    copy_gbs = 2 * (1 << 30) * 5 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    del src, dst
    read_ceiling = measure_read_ceiling(dev)
    mfma_ceiling = measure_mfma_ceiling(dev)

    # inputs, generated on the device
    q_win, k, v, qs, path = make_state(w, args, M, synth, dev)
    torch.cuda.synchronize()

    mode = resolve_mode(args.decode_mode, path)
    fused = mode == "fused"
    modes = {"split": path.decode, "fused": path.decode_fused}
    step_fn = modes[mode]
    mk = lambda: torch.cuda.Event(enable_timing=True)
    mean = lambda x: sum(x) / len(x)

    # timed region: events only at the pass boundaries and after the prefill, so that the decode
    # steps run back to back as a serving loop would issue them
    pre_ms, dec_us, wall = timed_passes(path, q_win, k, v, qs, step_fn, args.steps, args.warmup, torch)

    # the same prefill as two calls (eviction with every layer's gather, then the cluster build
    # re-reading the kept keys); same inputs and results, second of two runs
    for _ in range(2):
        a, b = mk(), mk()
        a.record()
        path.prefill(q_win, k, v, fused=False)
        b.record()
        torch.cuda.synchronize()
    pre_two_ms = a.elapsed_time(b)

    # per-kernel times on the same state and queries: each kernel launched E times back to back
    # (attention with every step's own selection), bracketed by HIP events on the launch stream
    def step_time(fn):
        a, b = mk(), mk()
        a.record()
        for e in range(E):
            fn(qs[e])
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / E * 1e3

    sel_us, att_us = kernel_times(path, qs, torch)
    alt = {}
    for name, fn in modes.items():  # every mode on the same state, E steps back to back
        if name != mode:
            step_time(fn)
            alt[name] = round(step_time(fn), 3)

    # cache state: each decode step alone between two events, once right after the previous step
    # (warm: L2 and the 256 MB memory-side cache hold what the earlier steps left) and once after a
    # read of 1 GiB of unrelated data (cold: nothing of the path's data is cached)
    flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)

    def single_steps(cold):
        t = []
        for e in range(E):
            if cold:
                flush.sum()
            a, b = mk(), mk()
            a.record()
            step_fn(qs[e])
            b.record()
            t.append((a, b))
        torch.cuda.synchronize()
        return mean([a.elapsed_time(b) for a, b in t]) * 1e3

    single_steps(False)
    cache = {"warm_us": round(single_steps(False), 3), "cold_us": round(single_steps(True), 3),
             "note": "one decode step between two HIP events (so launch latency is inside both); cold = "
                     "after reading 1 GiB of other data, which evicts L2 and the memory-side cache"}
    del flush

    # selection quality on the last step's queries: the share of each head's full softmax mass
    # (over every kept token) that falls on the selected clusters, exp(lse_selected - lse_all)
    path.decode(qs[E - 1])
    lse_sel = path.lse.clone()
    all_sel = torch.arange(path.C, dtype=torch.int32, device=dev).expand(*path.sel.shape[:3], path.C).contiguous()
    out_all = torch.empty_like(path.out)
    lse_all = torch.empty_like(path.lse)
    ws_all = M.workspace(M.workspace_bytes(M.MPC_OP_DECODE_ATTN, M.dims_of(path.out, path.k_s), w.keep), dev)
    M.mpc_sparse_decode_attn(qs[E - 1], path.k_s, path.v_s, all_sel, out_all, cluster_size=w.cluster,
                             sm_scale=path.sm_scale, lse=lse_all, ws=ws_all)
    recall = torch.exp(lse_sel.double() - lse_all.double())
    quality = {"attention_mass_recall_mean": round(recall.mean().item(), 4),
               "attention_mass_recall_min": round(recall.min().item(), 4),
               "note": "share of each head's softmax mass over all kept tokens that the selected clusters hold "
                       "(last decode step, every layer, sequence and query head)"}
    del all_sel, out_all, lse_all, ws_all

    # commonality of adjacent layers' unshared selections (Sec. 3, Observation 3) on the last
    # step's queries: representatives of every layer, one selection per layer, then the score
    common = commonality(w, path, qs[E - 1], args, M, torch, dev, mk)

    owners = [l for l in range(w.n_layers) if M.owner_layer(l, w.share_period, w.share_start) == l]
    sel_b, att_b = decode_bytes(w, owners, path.sel.cpu().numpy(), path.C, path.S, M.rep_rows(args.similarity))
    step_b = sel_b + att_b
    att_gbs = att_b / (att_us * 1e-6) / 1e9
    dec_gbs = step_b / (dec_us * 1e-6) / 1e9
    if fused:
        traffic = measured_traffic("decode_step", args.workload, source_digest(*DECODE_STEP_SOURCES))
        one = ("k_decode_self (every workgroup selects for its own unit, then gathers and attends)"
               if path.L * path.B * path.Hsel <= NUM_CU else
               "k_decode_step (first consumer of an owner head selects, the others wait)")
        roofline = {"kernel": one + ": two-level selection + gather + online-softmax attention, all layers, "
                                    "one launch",
                    "bound": "hbm", "achieved": round(dec_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(dec_gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
                    "algorithmic_bytes_per_launch": step_b, "avg_launch_us": round(dec_us, 3)}
    else:
        traffic = measured_traffic("sparse_decode", args.workload, source_digest(*SPARSE_DECODE_SOURCES))
        roofline = {"kernel": "k_sparse_decode (gather + online-softmax attention, all layers per launch)",
                    "bound": "hbm", "achieved": round(att_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(att_gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
                    "algorithmic_bytes_per_launch": att_b, "avg_launch_us": round(att_us, 3),
                    "whole_step": {"kernels": "k_select + k_sparse_decode", "achieved": round(dec_gbs, 1),
                                   "frac": round(dec_gbs / HBM_PEAK_GBS, 4), "algorithmic_bytes": step_b,
                                   "us": round(dec_us, 3)}}
    fl = prefill_flops(w, len(owners))
    pre_tflops = fl / (mean(pre_ms) * 1e-3) / 1e12
    read_same = measure_read_time(dev, att_b)

    rec = {
        "metric": METRIC,
        "value": round(dec_us / w.n_layers, 4),
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded generator, device-resident before timing)",
        "config": {"workload": f"{args.workload} {w.name}", "layers": w.n_layers, "batch": w.batch,
                   "q_heads": w.n_q_heads, "kv_heads": w.n_kv_heads, "head_dim": w.head_dim, "prompt_tokens": w.T,
                   "window_rows": w.window, "kept_tokens": w.keep, "cluster": w.cluster, "fanout": w.fanout,
                   "k_super": w.k_super, "k_clusters": w.k_clusters, "share_period": w.share_period,
                   "similarity": args.similarity, "group": args.group, "decode_steps_per_pass": E,
                   **({"planting": PLANTING} if w.n_sinks or w.hh_count else {})},
        "decode_step": {"mode": mode, "us": round(dec_us, 3), "algorithmic_bytes": step_b,
                        "achieved_GBps": round(dec_gbs, 1), "frac_of_hbm_peak": round(dec_gbs / HBM_PEAK_GBS, 4)},
        "kernels": {"select_us": round(sel_us, 3), "attention_us": round(att_us, 3),
                    "attention_algorithmic_bytes": att_b, "attention_GBps": round(att_gbs, 1),
                    "attention_frac_of_hbm_peak": round(att_gbs / HBM_PEAK_GBS, 4),
                    "read_same_bytes": read_same,
                    "attention_us_over_read_us": round(att_us / read_same["us"], 4),
                    "note": "each kernel launched once per decode step, back to back, between two HIP "
                            "events; per-launch average (attention reads each step's own selection); "
                            "read_same_bytes: one launch of the read-ceiling kernel reading the attention's "
                            "bytes as 16 KB chunks in random order, best of three grid shapes"},
        "decode_step_other_modes": alt,
        "decode_step_cache": cache,
        "selection_quality": quality,
        "commonality": common,
        "roofline": roofline,
        "copy_ceiling": {"GBps": round(copy_gbs, 1), "frac_of_peak": round(copy_gbs / HBM_PEAK_GBS, 4),
                         "note": "1 GiB device-to-device copy, read + write bytes"},
        "read_ceiling": dict(read_ceiling, attention_frac_of_ceiling=round(att_gbs / read_ceiling["GBps"], 4)),
        "mfma_ceiling": mfma_ceiling,
        "prefill": {"ms_per_pass": round(mean(pre_ms), 3), "owner_layers": len(owners),
                    "ms_per_owner_layer": round(mean(pre_ms) / len(owners), 3),
                    "algorithmic_TFLOP_per_pass": round(fl / 1e12, 3),
                    "achieved_TFLOPs": round(pre_tflops, 1),
                    "frac_of_mfma_peak": round(pre_tflops / MFMA_PEAK_TFLOPS[w.dtype], 4),
                    "ms_two_calls": round(pre_two_ms, 3),
                    "note": "one call (mpc_prefill): two score passes, top-k, gather of the layers without "
                            "representatives, cluster build gathering the other layers' rows; all layers"},
    }
    extra = [x for x in args.extra.split(",") if x and x != args.workload]
    if extra:
        # free the headline workload's prompt and kept caches before the other workloads
        del q_win, k, v, path, qs, modes, step_fn
        torch.cuda.empty_cache()
        rec["other_workloads"] = {x: extra_workload(x, args, M, synth, torch, dev) for x in extra}
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(w, min(E, 64), args.similarity, args.group)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
