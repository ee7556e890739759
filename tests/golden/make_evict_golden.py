"""Writes the oracle's static-eviction results for sampled heads of the 128K GQA workload at its
full window (13107 rows x 131072 keys per query head), too slow to recompute inside a GPU test.

Calls only the seeded input generator (``synth``) and the oracle (``oracle``). For each sampled
(layer, sequence, kv head) it stores the oracle's kept set, its boundary score (the score of rank
keep - local_keep among the older tokens, Sec. 3.2 / Alg. 3 step 1 ranking) and every older token
whose score lies within 1e-3 relative of that boundary, with its score. A GPU kept set that differs
from the stored one only by tokens of that band within 1e-6 of the boundary is a tie; any other
difference is a failure.

The window rows are split into chunks that run on separate threads: rows [t0, t1) of the window
are the rows of a window of t1 - t0 rows over the first T - W + t1 keys (under the causal mask no
later key is visible to them), so each chunk is one oracle call and the chunks' scores add up to
the whole window's.

    python tests/golden/make_evict_golden.py [--threads N]
"""
import argparse
import concurrent.futures as cf
import math
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import synth  # noqa: E402

# (workload, layer, [(sequence, kv head), ...])
CASES = [("C5", 30, [(0, 0), (0, 7)])]
BAND = 1e-3
OUT = os.path.join(HERE, "evict_{name}_layer{layer}.npz")


def head_scores(w, qw_group, k_head, chunk, threads):
    """Oracle token scores of one kv head: sum over its query heads and window-row chunks."""
    G, W, _ = qw_group.shape
    T = k_head.shape[0]
    sm = 1.0 / math.sqrt(w.head_dim)
    tasks = [(g, t0, min(W, t0 + chunk)) for g in range(G) for t0 in range(0, W, chunk)]

    def run(task):
        g, t0, t1 = task
        Tp = T - W + t1
        return oracle.token_scores(qw_group[g:g + 1, t0:t1], k_head[:Tp], w.dtype, sm)

    score = np.zeros(T, np.float64)
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        for (g, t0, t1), part in zip(tasks, ex.map(run, tasks)):
            score[:part.shape[0]] += part
    return score


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=os.cpu_count())
    ap.add_argument("--chunk", type=int, default=256)
    args = ap.parse_args()
    oracle.set_threads(1)
    for name, layer, heads in CASES:
        w = synth.get(name)
        t_start = time.time()
        qw, k, _ = synth.prefill_host(w, layer)
        G, loc, n_sel = w.group, w.local_keep, w.keep - w.local_keep
        rec = {}
        for b, h in heads:
            sc = head_scores(w, qw[b, h * G:(h + 1) * G], k[b, h], args.chunk, args.threads)
            kept = oracle.static_topk(sc, w.keep, loc)
            old = sc[:w.T - loc]
            order = np.lexsort((np.arange(old.shape[0]), -old))
            bnd = old[order[n_sel - 1]]
            band = np.nonzero(np.abs(old - bnd) <= BAND * bnd)[0].astype(np.int32)
            key = f"b{b}_h{h}"
            rec[key + "_kept"] = kept
            rec[key + "_boundary"] = np.array([bnd])
            rec[key + "_band_idx"] = band
            rec[key + "_band_score"] = old[band]
            rec[key + "_total"] = np.array([sc.sum()])
            print(f"{name} layer {layer} b {b} h {h}: boundary {bnd:.9e}, {band.size} tokens within "
                  f"{BAND:g}, total {sc.sum():.6f} (G*W = {G * w.window}), {time.time() - t_start:.0f} s", flush=True)
        np.savez_compressed(OUT.format(name=name, layer=layer), **rec)


if __name__ == "__main__":
    main()
