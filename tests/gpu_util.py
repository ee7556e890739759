"""Comparison rules and helpers for the GPU parity tests.

Index sets (kept tokens, selected clusters) must be equal, except that an element in the symmetric
difference is allowed when its oracle score ties the oracle's boundary score within 1e-6 relative.
Attention outputs: per (layer, sequence, q-head), ||o_gpu - o_ref||_inf <= tol * ||o_ref||_inf with
tol = 1e-4 for fp32 and 2e-2 for fp16 / bf16.
"""
import sys

import numpy as np
import torch

TIE_REL = 1e-6
OUT_TOL = {"fp32": 1e-4, "fp16": 2e-2, "bf16": 2e-2}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def bits_to_torch(a, dtype, device="cuda"):
    """numpy raw bits -> torch tensor of the element type on the device."""
    if dtype == "fp32":
        return torch.from_numpy(np.ascontiguousarray(a)).to(device)
    td = torch.bfloat16 if dtype == "bf16" else torch.float16
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(td).to(device)


def torch_to_bits(t, dtype):
    t = t.detach().cpu().contiguous()
    if dtype == "fp32":
        return t.numpy()
    return t.view(torch.int16).numpy().view(np.uint16)


def to_f64(t):
    return t.detach().to(torch.float64).cpu().numpy()


def boundary_score(score, k):
    """Score of the k-th element in (score desc, index asc) order."""
    order = np.lexsort((np.arange(len(score)), -np.asarray(score)))
    return score[order[k - 1]]


def assert_sets_tie_equal(got, exp, score, boundary, what):
    """Equal sets up to elements whose oracle score ties the boundary (1e-6 relative)."""
    g, e = set(np.asarray(got).tolist()), set(np.asarray(exp).tolist())
    diff = g ^ e
    tol = TIE_REL * abs(boundary)
    bad = [i for i in diff if abs(score[i] - boundary) > tol]
    assert not bad, f"{what}: {len(diff)} differing elements, {len(bad)} not ties (e.g. {bad[:5]})"
    return len(diff) // 2


def assert_out_close(out, ref, dtype, what):
    """out, ref: [..., d] float64 arrays; per-row relative inf-norm check."""
    err = np.abs(out - ref).max(axis=-1)
    scale = np.abs(ref).max(axis=-1)
    worst = float((err / np.maximum(scale, 1e-30)).max())
    assert worst <= OUT_TOL[dtype], f"{what}: worst relative error {worst:.3e} > {OUT_TOL[dtype]}"
    return worst


def random_sel(rng, n_units, C, k, include_last=True):
    """Ascending distinct cluster ids per unit; about half the units include the last cluster."""
    sel = np.empty((n_units, k), np.int32)
    for u in range(n_units):
        if include_last and u % 2 == 0 and k > 1:
            s = np.concatenate([rng.choice(C - 1, k - 1, replace=False), [C - 1]])
        else:
            s = rng.choice(C, k, replace=False)
        sel[u] = np.sort(s)
    return sel
