"""Seeded synthetic inputs shared by the CPU oracle tests and the GPU path.

The generator is a compiled module of its own (``libsynth.so``): host functions fill numpy
buffers, device functions fill torch CUDA tensors, and both produce the same bytes for the same
spec. Nothing here computes any step of the method.
"""
import ctypes
import os

import numpy as np

from .workloads import WORKLOADS, Workload, get  # noqa: F401

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

DTYPE_CODE = {"fp32": 0, "fp16": 1, "bf16": 2}
NP_STORAGE = {"fp32": np.float32, "fp16": np.uint16, "bf16": np.uint16}


class SynthSpec(ctypes.Structure):
    _fields_ = [
        ("seed", ctypes.c_uint64),
        ("seq_stride", ctypes.c_uint64),
        ("n_layers", ctypes.c_int32),
        ("batch", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("T", ctypes.c_int32),
        ("W", ctypes.c_int32),
        ("n_outlier", ctypes.c_int32),
        ("outlier_scale", ctypes.c_float),
        ("rope", ctypes.c_int32),
        ("rope_base", ctypes.c_float),
        ("n_sinks", ctypes.c_int32),
        ("hh_count", ctypes.c_int32),
        ("hh_span", ctypes.c_int32),
        ("hh_lo", ctypes.c_int32),
        ("hh_hi", ctypes.c_int32),
    ]


def lib():
    global _LIB
    if _LIB is None:
        # MPC_SANITIZE=1: the AddressSanitizer / UBSan build (tests/sanitize.sh)
        san = os.environ.get("MPC_SANITIZE") == "1"
        path = os.path.join(HERE, "libsynth_san.so" if san else "libsynth.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(path)
        P, I, V = ctypes.POINTER(SynthSpec), ctypes.c_int32, ctypes.c_void_p
        for name, args in {
            "synth_validate": [P],
            "synth_rope_table": [I, I, ctypes.c_double, V],
            "synth_outlier_channels": [P, I, I, I, V],
            "synth_hh_starts": [P, I, I, I, V],
            "synth_qwin_host": [P, I, V, V],
            "synth_unit_dir_host": [P, V, V],
            "synth_kv_host": [P, I, V, V, V, V],
            "synth_dq_host": [P, I, V],
            "synth_qwin_dev": [P, I, I, V, V, V],
            "synth_kv_dev": [P, I, I, V, V, V, V, V, V],
            "synth_dq_dev": [P, I, V, V],
        }.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        _LIB = L
    return _LIB


def spec(w: Workload, *, T=None, W=None, planting=True, n_layers=None) -> SynthSpec:
    """Generator spec for workload ``w``. ``T``/``W`` override the prompt / window lengths (used to
    generate a post-eviction cache directly); ``planting=False`` drops sinks and heavy hitters."""
    T = w.T if T is None else T
    W = w.window if W is None else W
    plant = planting and W > 0
    return SynthSpec(
        seed=w.seed, seq_stride=w.seq_stride,
        n_layers=w.n_layers if n_layers is None else n_layers, batch=w.batch,
        n_q_heads=w.n_q_heads, n_kv_heads=w.n_kv_heads, head_dim=w.head_dim,
        dtype=DTYPE_CODE[w.dtype], T=T, W=W, n_outlier=w.n_outlier,
        outlier_scale=w.outlier_scale, rope=int(w.rope), rope_base=w.rope_base,
        n_sinks=w.n_sinks if plant else 0, hh_count=w.hh_count if plant else 0,
        hh_span=w.hh_span, hh_lo=w.hh_lo, hh_hi=w.hh_hi if w.hh_count else 0,
    )


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"{what} failed with code {rc}")


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data)


def rope_table(T, d, base):
    out = np.empty((T, d // 2, 2), np.float64)
    _check(lib().synth_rope_table(T, d, float(base), _ptr(out)), "synth_rope_table")
    return out


def storage(dtype):
    return NP_STORAGE[dtype]


def qwin_host(sp: SynthSpec, layer: int, dtype: str, rope=None):
    out = np.empty((sp.batch, sp.n_q_heads, sp.W, sp.head_dim), storage(dtype))
    if sp.W == 0:
        return out
    r = None if rope is None else _ptr(rope)
    _check(lib().synth_qwin_host(ctypes.byref(sp), layer, r, _ptr(out)), "synth_qwin_host")
    return out


def kv_host(sp: SynthSpec, layer: int, dtype: str, qwin_layer=None, rope=None):
    shape = (sp.batch, sp.n_kv_heads, sp.T, sp.head_dim)
    k = np.empty(shape, storage(dtype))
    v = np.empty(shape, storage(dtype))
    q = None if qwin_layer is None else _ptr(np.ascontiguousarray(qwin_layer))
    r = None if rope is None else _ptr(rope)
    _check(lib().synth_kv_host(ctypes.byref(sp), layer, q, r, _ptr(k), _ptr(v)), "synth_kv_host")
    return k, v


def unit_dir_host(sp: SynthSpec, qwin_layer):
    u = np.empty((sp.batch, sp.n_kv_heads, sp.head_dim), np.float64)
    _check(lib().synth_unit_dir_host(ctypes.byref(sp), _ptr(np.ascontiguousarray(qwin_layer)), _ptr(u)),
           "synth_unit_dir_host")
    return u


def dq_host(sp: SynthSpec, step: int, dtype: str):
    q = np.empty((sp.n_layers, sp.batch, sp.n_q_heads, sp.head_dim), storage(dtype))
    _check(lib().synth_dq_host(ctypes.byref(sp), step, _ptr(q)), "synth_dq_host")
    return q


def outlier_channels(sp: SynthSpec, layer, b, kvh):
    ch = np.zeros(max(sp.n_outlier, 1), np.int32)
    _check(lib().synth_outlier_channels(ctypes.byref(sp), layer, b, kvh, _ptr(ch)), "outliers")
    return ch[: sp.n_outlier]


def hh_starts(sp: SynthSpec, layer, b, kvh):
    st = np.zeros(max(sp.hh_count, 1), np.int32)
    _check(lib().synth_hh_starts(ctypes.byref(sp), layer, b, kvh, _ptr(st)), "hh_starts")
    return st[: sp.hh_count]


def prefill_host(w: Workload, layer: int):
    """One layer of prefill inputs on the host: (q_win [B][Hq][W][d], k, v [B][Hkv][T][d])."""
    sp = spec(w)
    rope = rope_table(w.T, w.head_dim, w.rope_base) if w.rope else None
    qw = qwin_host(sp, layer, w.dtype, rope)
    k, v = kv_host(sp, layer, w.dtype, qw, rope)
    return qw, k, v


def cache_host(w: Workload, layer: int, T=None):
    """A post-eviction cache of ``T`` (default ``w.keep``) rows generated directly (no planting)."""
    T = w.keep if T is None else T
    sp = spec(w, T=T, W=0, planting=False)
    rope = rope_table(T, w.head_dim, w.rope_base) if w.rope else None
    return kv_host(sp, layer, w.dtype, None, rope)


# ------------------------------------------------------------------ device (torch) helpers
def _torch():
    import torch
    return torch


def torch_dtype(dtype):
    t = _torch()
    return {"fp32": t.float32, "fp16": t.float16, "bf16": t.bfloat16}[dtype]


def _stream_ptr():
    return ctypes.c_void_p(_torch().cuda.current_stream().cuda_stream)


def rope_dev(T, d, base, device="cuda"):
    return _torch().from_numpy(rope_table(T, d, base)).to(device)


def qwin_dev(sp: SynthSpec, dtype: str, layer0=0, n_layers=None, rope=None, device="cuda"):
    t = _torch()
    n = sp.n_layers if n_layers is None else n_layers
    out = t.empty((n, sp.batch, sp.n_q_heads, sp.W, sp.head_dim), dtype=torch_dtype(dtype), device=device)
    if sp.W:
        r = None if rope is None else ctypes.c_void_p(rope.data_ptr())
        _check(lib().synth_qwin_dev(ctypes.byref(sp), layer0, n, r, ctypes.c_void_p(out.data_ptr()),
                                    _stream_ptr()), "synth_qwin_dev")
    return out


def kv_dev(sp: SynthSpec, dtype: str, layer0=0, n_layers=None, qwin=None, rope=None, device="cuda",
           out=None):
    t = _torch()
    n = sp.n_layers if n_layers is None else n_layers
    shape = (n, sp.batch, sp.n_kv_heads, sp.T, sp.head_dim)
    if out is None:
        k = t.empty(shape, dtype=torch_dtype(dtype), device=device)
        v = t.empty(shape, dtype=torch_dtype(dtype), device=device)
    else:
        k, v = out
    u = t.empty((sp.batch, sp.n_kv_heads, sp.head_dim), dtype=t.float64, device=device)
    q = None if qwin is None else ctypes.c_void_p(qwin.data_ptr())
    r = None if rope is None else ctypes.c_void_p(rope.data_ptr())
    _check(lib().synth_kv_dev(ctypes.byref(sp), layer0, n, q, r, ctypes.c_void_p(u.data_ptr()),
                              ctypes.c_void_p(k.data_ptr()), ctypes.c_void_p(v.data_ptr()), _stream_ptr()),
           "synth_kv_dev")
    return k, v


def dq_dev(sp: SynthSpec, dtype: str, step: int, device="cuda"):
    t = _torch()
    q = t.empty((sp.n_layers, sp.batch, sp.n_q_heads, sp.head_dim), dtype=torch_dtype(dtype), device=device)
    _check(lib().synth_dq_dev(ctypes.byref(sp), step, ctypes.c_void_p(q.data_ptr()), _stream_ptr()),
           "synth_dq_dev")
    return q
