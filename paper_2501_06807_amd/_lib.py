"""ctypes binding of libmpcache.so: the entry points of the C ABI with the same names.

Argument marshalling only: shapes are read off torch CUDA tensors, pointers and the current
stream are handed to the library, and a non-zero status raises MpcError. Every step of the path
runs in the HIP kernels; there is no fallback.
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmpcache.so")

MPC_OK, MPC_EINVAL, MPC_ESHAPE, MPC_EUNSUPPORTED, MPC_EWORKSPACE, MPC_EHIP = range(6)
MPC_OP_STATIC_EVICT, MPC_OP_SELECT, MPC_OP_DECODE_ATTN, MPC_OP_DECODE_STEP = range(4)
DTYPE_CODE = {torch.float32: 0, torch.float16: 1, torch.bfloat16: 2}


class MpcDims(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("batch", "layer0", "n_layers", "n_q_heads", "n_kv_heads", "head_dim", "dtype", "kv_capacity")]


class MpcSelectCfg(ctypes.Structure):
    _fields_ = [("cluster_size", ctypes.c_int32), ("fanout", ctypes.c_int32),
                ("k_super", ctypes.c_int32), ("k_clusters", ctypes.c_int32),
                ("alpha", ctypes.c_float), ("share_period", ctypes.c_int32),
                ("share_start", ctypes.c_int32), ("similarity", ctypes.c_int32), ("group", ctypes.c_int32)]


class MpcEvictCfg(ctypes.Structure):
    _fields_ = [("window", ctypes.c_int32), ("keep", ctypes.c_int32),
                ("local_keep", ctypes.c_int32), ("sm_scale", ctypes.c_float),
                ("causal", ctypes.c_int32), ("share_period", ctypes.c_int32),
                ("share_start", ctypes.c_int32)]


class MpcError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__(f"{fn}: status {status} ({msg})")
        self.status = status


_LIB = None
EXPORTS = ("mpc_workspace_bytes", "mpc_static_evict", "mpc_static_evict_noalloc", "mpc_static_evict_noalloc_limit",
           "mpc_build_clusters", "mpc_prefill", "mpc_select_clusters",
           "mpc_sparse_decode_attn", "mpc_decode_step", "mpc_decode_step_status", "mpc_append_kv", "mpc_commonality",
           "mpc_owner_layer",
           "mpc_status_string", "mpc_last_error")


def lib():
    """Loads libmpcache.so; raises if it has not been built (no fallback path exists)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P, V, I, F = ctypes.POINTER, ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
        L.mpc_workspace_bytes.argtypes = [I, P(MpcDims), I, V]
        L.mpc_workspace_bytes.restype = ctypes.c_size_t
        L.mpc_static_evict.argtypes = [P(MpcDims), I, P(MpcEvictCfg)] + [V] * 8 + [V, ctypes.c_size_t, V]
        L.mpc_static_evict_noalloc.argtypes = [P(MpcDims), I, P(MpcEvictCfg)] + [V] * 8 + [V]
        L.mpc_static_evict_noalloc.restype = ctypes.c_int
        L.mpc_static_evict_noalloc_limit.argtypes = []
        L.mpc_static_evict_noalloc_limit.restype = ctypes.c_size_t
        L.mpc_build_clusters.argtypes = [P(MpcDims), I, P(MpcSelectCfg), V, V, V, V]
        L.mpc_prefill.argtypes = [P(MpcDims), I, P(MpcEvictCfg), P(MpcSelectCfg)] + [V] * 10 + [V, ctypes.c_size_t, V]
        L.mpc_select_clusters.argtypes = [P(MpcDims), I, P(MpcSelectCfg)] + [V] * 5 + [V, ctypes.c_size_t, V]
        L.mpc_sparse_decode_attn.argtypes = [P(MpcDims), I, I, I, V, V, V, V, I, I, F, V, V, V, ctypes.c_size_t, V]
        L.mpc_decode_step.argtypes = [P(MpcDims), I, I, P(MpcSelectCfg)] + [V] * 5 + [F] + [V] * 4 + [
            V, ctypes.c_size_t, V]
        L.mpc_append_kv.argtypes = [P(MpcDims), I, I, P(MpcSelectCfg)] + [V] * 6 + [P(I), P(I), V]
        L.mpc_decode_step_status.argtypes = [V, ctypes.c_size_t, I, P(I)]
        L.mpc_commonality.argtypes = [I, I, I, I, V, V, V]
        for fn in ("mpc_static_evict", "mpc_build_clusters", "mpc_prefill", "mpc_select_clusters", "mpc_sparse_decode_attn",
                   "mpc_decode_step", "mpc_decode_step_status", "mpc_append_kv", "mpc_commonality"):
            getattr(L, fn).restype = ctypes.c_int
        L.mpc_owner_layer.argtypes = [I, I, I]
        L.mpc_owner_layer.restype = I
        L.mpc_status_string.argtypes = [ctypes.c_int]
        L.mpc_status_string.restype = ctypes.c_char_p
        L.mpc_last_error.argtypes = []
        L.mpc_last_error.restype = ctypes.c_char_p
        _LIB = L
    return _LIB


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check(fn, status):
    if status != MPC_OK:
        raise MpcError(fn, status, lib().mpc_last_error().decode())


def dims_of(q_like, kv, layer0=0):
    """mpc_dims from a query-like tensor [L][B][Hq][..][d] and a cache [L][B][Hkv][Tcap][d]; the
    cache's row axis is its capacity."""
    if kv.dtype not in DTYPE_CODE:
        raise TypeError(f"unsupported dtype {kv.dtype}")
    cap = kv.shape[3] if kv.dim() == 5 else 0
    return MpcDims(batch=kv.shape[1], layer0=layer0, n_layers=kv.shape[0], n_q_heads=q_like.shape[2],
                   n_kv_heads=kv.shape[2], head_dim=kv.shape[-1], dtype=DTYPE_CODE[kv.dtype], kv_capacity=cap)


def _contig(*ts):
    for t in ts:
        if t is not None and not (t.is_cuda and t.is_contiguous()):
            raise ValueError("tensors must be contiguous CUDA tensors")


def owner_layer(layer, period, start=2):
    return lib().mpc_owner_layer(layer, period, start)


def workspace_bytes(op, dims, T_or_Ts, cfg=None):
    c = None if cfg is None else ctypes.byref(cfg)
    return lib().mpc_workspace_bytes(op, ctypes.byref(dims), T_or_Ts, c)


def workspace(nbytes, device="cuda"):
    """A zero-filled workspace buffer (the counters in it must start at zero)."""
    return torch.zeros(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def mpc_static_evict(q_win, k, v, kept_idx, k_out, v_out, *, keep, local_keep, sm_scale, causal=True,
                     layer0=0, share_period=1, share_start=2, token_score=None, row_lse=None, ws=None,
                     stream=None):
    """q_win [L][B][Hq][W][d], k/v [L][B][Hkv][T][d] -> kept_idx [L][B][Hkv][keep], k_out/v_out."""
    _contig(q_win, k, v, kept_idx, k_out, v_out, token_score, row_lse, ws)
    dims = dims_of(q_win, k, layer0)
    dims.kv_capacity = k_out.shape[3]
    T, W = k.shape[3], q_win.shape[3]
    cfg = MpcEvictCfg(window=W, keep=keep, local_keep=local_keep, sm_scale=sm_scale, causal=int(causal),
                      share_period=share_period, share_start=share_start)
    if ws is None:
        ws = workspace(workspace_bytes(MPC_OP_STATIC_EVICT, dims, T, cfg), k.device)
    _check("mpc_static_evict", lib().mpc_static_evict(
        ctypes.byref(dims), T, ctypes.byref(cfg), _ptr(q_win), _ptr(k), _ptr(v), _ptr(kept_idx), _ptr(k_out),
        _ptr(v_out), _ptr(token_score), _ptr(row_lse), _ptr(ws), ws.numel(), _stream(stream)))


def mpc_static_evict_noalloc(q_win, k, v, kept_idx, k_out, v_out, *, keep, local_keep, sm_scale, causal=True,
                             layer0=0, share_period=1, share_start=2, token_score=None, row_lse=None, stream=None):
    """mpc_static_evict with the library's static scratch array as its workspace (nothing is
    allocated); fails with MpcError (MPC_EWORKSPACE) when the block needs more than
    noalloc_limit() scratch bytes."""
    _contig(q_win, k, v, kept_idx, k_out, v_out, token_score, row_lse)
    dims = dims_of(q_win, k, layer0)
    dims.kv_capacity = k_out.shape[3]
    T, W = k.shape[3], q_win.shape[3]
    cfg = MpcEvictCfg(window=W, keep=keep, local_keep=local_keep, sm_scale=sm_scale, causal=int(causal),
                      share_period=share_period, share_start=share_start)
    _check("mpc_static_evict_noalloc", lib().mpc_static_evict_noalloc(
        ctypes.byref(dims), T, ctypes.byref(cfg), _ptr(q_win), _ptr(k), _ptr(v), _ptr(kept_idx), _ptr(k_out),
        _ptr(v_out), _ptr(token_score), _ptr(row_lse), _stream(stream)))


def noalloc_limit():
    """Bytes of the static scratch array behind mpc_static_evict_noalloc."""
    return lib().mpc_static_evict_noalloc_limit()


SIMILARITY = {"linear": 0, "maxprod": 1, "mean": 2}
GROUP = {"sum": 0, "max": 1, "head": 2}


def rep_rows(similarity):
    """Rows of d floats per cluster representative (r^max and r^min for the max-product bound)."""
    return 2 if SIMILARITY[similarity] == 1 else 1


def select_cfg(cluster, fanout, k_super, k_clusters, alpha=0.6, share_period=1, share_start=2,
               similarity="linear", group="sum"):
    """group: "sum" / "max" (the q-heads of a kv head share one selection scored by the sum / the
    maximum of their similarities) or "head" (one selection per q-head)."""
    return MpcSelectCfg(cluster_size=cluster, fanout=fanout, k_super=k_super, k_clusters=k_clusters,
                        alpha=alpha, share_period=share_period, share_start=share_start,
                        similarity=SIMILARITY[similarity], group=GROUP[group])


def sel_heads(cfg, n_q_heads, n_kv_heads):
    """Selection lists per (layer, sequence) under the config's group rule."""
    return n_q_heads if cfg.group == GROUP["head"] else n_kv_heads


def _slots(cap, cfg):
    C = -(-cap // cfg.cluster_size)
    return C, -(-C // cfg.fanout)


def mpc_build_clusters(k_cache, cent, scent, cfg, *, Ts=None, layer0=0, stream=None):
    """k_cache [L][B][Hkv][Tcap][d] (rows [0, Ts) used, Ts = Tcap by default) -> cent
    [L][B][Hkv][Ccap][R][d], scent [L][B][Hkv][Scap][R][d] (float32; R = 2 rows r^max, r^min for the
    max-product bound, else 1 and the R axis may be omitted)."""
    _contig(k_cache, cent, scent)
    dims = dims_of(k_cache, k_cache, layer0)
    Ts = k_cache.shape[3] if Ts is None else Ts
    _check_reps(k_cache, cent, scent, cfg)
    _check("mpc_build_clusters", lib().mpc_build_clusters(
        ctypes.byref(dims), Ts, ctypes.byref(cfg), _ptr(k_cache), _ptr(cent), _ptr(scent), _stream(stream)))


def _check_reps(k_cache, cent, scent, cfg):
    L, B, Hkv, cap, d = k_cache.shape
    C, S = _slots(cap, cfg)
    R = 2 if cfg.similarity == SIMILARITY["maxprod"] else 1
    if cent.numel() != L * B * Hkv * C * R * d or scent.numel() != L * B * Hkv * S * R * d:
        raise ValueError(f"cent / scent must hold [L][B][Hkv][C or S][{R}][d] floats")
    if cent.dtype != torch.float32 or scent.dtype != torch.float32:
        raise TypeError("cent / scent must be float32")


def mpc_prefill(q_win, k, v, kept_idx, k_out, v_out, cent, scent, cfg, *, keep, local_keep, sm_scale, causal=True,
                layer0=0, share_period=1, share_start=2, token_score=None, row_lse=None, ws=None, stream=None):
    """mpc_static_evict then mpc_build_clusters over the kept rows (Ts = keep) in one call, with the
    selection owners' rows gathered inside the build; the eviction's sharing rule is
    share_period / share_start, the representatives' that of cfg."""
    _contig(q_win, k, v, kept_idx, k_out, v_out, cent, scent, token_score, row_lse, ws)
    _check_reps(k_out, cent, scent, cfg)
    dims = dims_of(q_win, k, layer0)
    dims.kv_capacity = k_out.shape[3]
    T, W = k.shape[3], q_win.shape[3]
    ecfg = MpcEvictCfg(window=W, keep=keep, local_keep=local_keep, sm_scale=sm_scale, causal=int(causal),
                       share_period=share_period, share_start=share_start)
    if ws is None:
        ws = workspace(workspace_bytes(MPC_OP_STATIC_EVICT, dims, T, ecfg), k.device)
    _check("mpc_prefill", lib().mpc_prefill(
        ctypes.byref(dims), T, ctypes.byref(ecfg), ctypes.byref(cfg), _ptr(q_win), _ptr(k), _ptr(v), _ptr(kept_idx),
        _ptr(k_out), _ptr(v_out), _ptr(cent), _ptr(scent), _ptr(token_score), _ptr(row_lse), _ptr(ws), ws.numel(),
        _stream(stream)))


def mpc_select_clusters(q, cent, scent, sel, cfg, *, Ts, sel_score=None, layer0=0, stream=None):
    """q [L][B][Hq][d], cent / scent with Ccap / Scap slots (the first ceil(Ts / s) used) ->
    sel [L][B][H][k_clusters] (int32, ascending), H = Hq for the "head" group rule, else Hkv."""
    _contig(q, cent, scent, sel, sel_score)
    dims = dims_of(q, cent, layer0)
    dims.head_dim = q.shape[-1]
    dims.dtype = DTYPE_CODE[q.dtype]
    dims.kv_capacity = cent.shape[3] * cfg.cluster_size
    if scent.shape[3] != _slots(dims.kv_capacity, cfg)[1]:
        raise ValueError("scent must have ceil(Ccap / fanout) super-cluster slots")
    if sel.shape[2] != sel_heads(cfg, q.shape[2], cent.shape[2]):
        raise ValueError("sel must have one list per q-head for the head rule, per kv head otherwise")
    _check("mpc_select_clusters", lib().mpc_select_clusters(
        ctypes.byref(dims), Ts, ctypes.byref(cfg), _ptr(q), _ptr(cent), _ptr(scent), _ptr(sel), _ptr(sel_score),
        None, 0, _stream(stream)))


def mpc_sparse_decode_attn(q, k_cache, v_cache, sel, out, *, cluster_size, sm_scale, Ts=None, n_tail=0, lse=None,
                           ws=None, layer0=0, stream=None):
    """q [L][B][Hq][d], k/v [L][B][Hkv][Tcap][d], sel [L][B][H][k] (H = Hkv: one list per kv head;
    H = Hq: one per q-head) -> out [L][B][Hq][d]. Clustered rows [0, Ts) (Ts = Tcap - n_tail by
    default) and tail rows [Ts, Ts + n_tail)."""
    _contig(q, k_cache, v_cache, sel, out, lse, ws)
    dims = dims_of(q, k_cache, layer0)
    Ts = k_cache.shape[3] - n_tail if Ts is None else Ts
    if ws is None:
        ws = workspace(workspace_bytes(MPC_OP_DECODE_ATTN, dims, Ts), q.device)
    _check("mpc_sparse_decode_attn", lib().mpc_sparse_decode_attn(
        ctypes.byref(dims), Ts, n_tail, cluster_size, _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(sel), sel.shape[2],
        sel.shape[-1], sm_scale, _ptr(out), _ptr(lse), _ptr(ws), ws.numel(), _stream(stream)))


def mpc_decode_step(q, cent, scent, k_cache, v_cache, sel, out, cfg, *, sm_scale, Ts=None, n_tail=0, sel_score=None,
                    lse=None, ws=None, layer0=0, stream=None):
    """Selection of every owner head then sparse attention of every head, in one call.

    q [L][B][Hq][d], cent/scent as built, k/v [L][B][Hkv][Tcap][d] (clustered rows [0, Ts), Ts = Tcap - n_tail
    by default, then the tail) -> sel [L][B][H][k] (H as for mpc_select_clusters), out [L][B][Hq][d].
    ws must come from workspace() (zero-filled) and be reused by later calls of the same shape.
    """
    _contig(q, cent, scent, k_cache, v_cache, sel, out, sel_score, lse, ws)
    dims = dims_of(q, k_cache, layer0)
    Ts = k_cache.shape[3] - n_tail if Ts is None else Ts
    if ws is None:
        ws = workspace(workspace_bytes(MPC_OP_DECODE_STEP, dims, Ts, cfg), q.device)
    _check("mpc_decode_step", lib().mpc_decode_step(
        ctypes.byref(dims), Ts, n_tail, ctypes.byref(cfg), _ptr(q), _ptr(cent), _ptr(scent), _ptr(k_cache), _ptr(v_cache),
        sm_scale, _ptr(sel), _ptr(sel_score), _ptr(out), _ptr(lse), _ptr(ws), ws.numel(), _stream(stream)))
    return ws


def mpc_commonality(idx, out, m, stream=None):
    """idx [L][...][k] int32 top-k sets per layer -> out [...] float64: commonality score of m + 1
    adjacent layers (Sec. 3, Observation 3) for every unit of the middle axes."""
    _contig(idx, out)
    if idx.dtype != torch.int32 or out.dtype != torch.float64:
        raise TypeError("idx must be int32 and out float64")
    L, k = idx.shape[0], idx.shape[-1]
    units = idx[0, ..., 0].numel()
    if out.numel() != units:
        raise ValueError("out must hold one value per unit")
    _check("mpc_commonality", lib().mpc_commonality(L, units, k, m, _ptr(idx), _ptr(out), _stream(stream)))


def mpc_append_kv(k_new, v_new, k_cache, v_cache, cent, scent, cfg, *, Ts, n_tail, layer0=0, stream=None):
    """Appends one decoded token: k_new / v_new [L][B][Hkv][d] into k/v [L][B][Hkv][Tcap][d] (sealing a full
    tail into a cluster, whose representatives in cent / scent are rebuilt). Returns the new (Ts, n_tail)."""
    _contig(k_new, v_new, k_cache, v_cache, cent, scent)
    dims = dims_of(k_cache, k_cache, layer0)
    if k_new.shape != k_cache.shape[:3] + k_cache.shape[4:] or v_new.shape != k_new.shape:
        raise ValueError("k_new / v_new must be [L][B][Hkv][d] like the cache")
    if k_new.dtype != k_cache.dtype or v_new.dtype != k_cache.dtype or v_cache.dtype != k_cache.dtype:
        raise TypeError("k_new / v_new / v_cache must have the cache's dtype")
    C, S = _slots(k_cache.shape[3], cfg)
    if cent.shape[3] != C or scent.shape[3] != S:
        raise ValueError(f"cent / scent must have {C} / {S} slots for a capacity of {k_cache.shape[3]} rows")
    ts_out, tail_out = ctypes.c_int32(), ctypes.c_int32()
    _check("mpc_append_kv", lib().mpc_append_kv(
        ctypes.byref(dims), Ts, n_tail, ctypes.byref(cfg), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache),
        _ptr(cent), _ptr(scent), ctypes.byref(ts_out), ctypes.byref(tail_out), _stream(stream)))
    return ts_out.value, tail_out.value


def mpc_decode_step_status(ws, clear=False):
    """Error word of a decode-step workspace (bit 0: a unit gave up waiting for its selection and
    wrote NaN outputs); blocking, call after the steps' stream has completed."""
    _contig(ws)
    flags = ctypes.c_int32()
    _check("mpc_decode_step_status", lib().mpc_decode_step_status(_ptr(ws), ws.numel() * ws.element_size(),
                                                                  int(bool(clear)), ctypes.byref(flags)))
    return flags.value
