"""ctypes binding of the CPU oracle (``liboracle.so``). TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use this
package. Inputs are numpy arrays holding raw element bits (float32 for fp32, uint16 for fp16 and
bf16); results are fp64 numpy arrays or int32 index arrays.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None
DTYPE_CODE = {"fp32": 0, "fp16": 1, "bf16": 2}


def lib():
    global _LIB
    if _LIB is None:
        # MPC_SANITIZE=1: the AddressSanitizer / UBSan build (tests/sanitize.sh)
        san = os.environ.get("MPC_SANITIZE") == "1"
        path = os.path.join(HERE, "liboracle_san.so" if san else "liboracle.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(path)
        I, F, D, V = ctypes.c_int32, ctypes.c_float, ctypes.c_double, ctypes.c_void_p
        sigs = {
            "mpcref_window_rows": ([I], I),
            "mpcref_owner_layer": ([I, I, I], I),
            "mpcref_keep_tokens": ([I, D, I], I),
            "mpcref_level1_keep": ([I, D], I),
            "mpcref_level2_keep": ([I, D, I, I], I),
            "mpcref_level2_keep_of_prompt": ([I, D, I, I], I),
            "mpcref_token_scores": ([I, I, I, I, I, F, I, V, V, V, V], ctypes.c_int),
            "mpcref_row_lse": ([I, I, I, I, F, I, V, I, V, V], ctypes.c_int),
            "mpcref_static_topk": ([I, V, I, I, V], ctypes.c_int),
            "mpcref_cluster_bounds": ([I, I, I, V, I, I, V, V], ctypes.c_int),
            "mpcref_centroid": ([D, D, F], F),
            "mpcref_cluster_scores": ([I, I, I, I, I, V, I, V, V], ctypes.c_int),
            "mpcref_cluster_mean": ([I, I, I, V, I, I, V], ctypes.c_int),
            "mpcref_mp_bound": ([I, V, V, V, V], ctypes.c_int),
            "mpcref_topk": ([I, V, I, V], ctypes.c_int),
            "mpcref_attend": ([I, I, F, V, I, V, V, V, V, V], ctypes.c_int),
            "mpcref_static_evict": ([I] * 11 + [F, I, I, I] + [V] * 7, ctypes.c_int),
            "mpcref_build_clusters": ([I] * 9 + [F, I, I, I] + [V] * 3, ctypes.c_int),
            "mpcref_select_clusters": ([I] * 16 + [V] * 5, ctypes.c_int),
            "mpcref_append_state": ([I, I, I, V, V], ctypes.c_int),
            "mpcref_sparse_decode_attn": ([I] * 9 + [V] * 4 + [I, I, F, V, V], ctypes.c_int),
            "mpcref_commonality": ([I] * 4 + [V, V], ctypes.c_int),
            "mpcref_dense_decode_attn": ([I] * 7 + [V] * 3 + [F, V, V], ctypes.c_int),
            "mpcref_threads": ([], ctypes.c_int),
            "mpcref_set_threads": ([I], None),
        }
        for name, (args, res) in sigs.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _LIB = L
    return _LIB


class OracleError(RuntimeError):
    def __init__(self, what, code):
        super().__init__(f"{what} returned status {code}")
        self.code = code


def _p(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def _c(a, dt=None):
    a = np.ascontiguousarray(a) if dt is None else np.ascontiguousarray(a, dtype=dt)
    return a


def _ok(rc, what):
    if rc != 0:
        raise OracleError(what, rc)


# ------------------------------------------------------------------ rules
def window_rows(T):
    return lib().mpcref_window_rows(T)


def owner_layer(layer, period, start=2):
    return lib().mpcref_owner_layer(layer, period, start)


def keep_tokens(T, ratio, cluster):
    return lib().mpcref_keep_tokens(T, ratio, cluster)


def level1_keep(n_super, final_ratio):
    return lib().mpcref_level1_keep(n_super, final_ratio)


def level2_keep(keep, ratio, cluster, n_cand):
    return lib().mpcref_level2_keep(keep, ratio, cluster, n_cand)


def level2_keep_of_prompt(T, ratio, cluster, n_cand):
    """Level-2 budget with the dynamic ratio read against the prompt length T (Fig. 9 caption)."""
    return lib().mpcref_level2_keep_of_prompt(T, ratio, cluster, n_cand)


def threads():
    return lib().mpcref_threads()


def set_threads(n):
    """Threads of the oracle's parallel loops from now on (timing only)."""
    lib().mpcref_set_threads(int(n))


# ------------------------------------------------------------------ per head
def token_scores(q_win, k, dtype, sm_scale, causal=True, with_lse=False):
    """q_win [G][W][d], k [T][d] -> score [T] (and row log-sum-exp [G][W])."""
    q_win, k = _c(q_win), _c(k)
    G, W, d = q_win.shape
    T = k.shape[0]
    score = np.empty(T, np.float64)
    lse = np.empty((G, W), np.float64) if with_lse else None
    _ok(lib().mpcref_token_scores(G, d, T, W, DTYPE_CODE[dtype], sm_scale, int(causal), _p(q_win),
                                  _p(k), _p(score), _p(lse)), "mpcref_token_scores")
    return (score, lse) if with_lse else score


def row_lse(q_row, t, W, k, dtype, sm_scale, causal=True):
    q_row, k = _c(q_row), _c(k)
    T, d = k.shape
    out = np.empty(1, np.float64)
    _ok(lib().mpcref_row_lse(d, T, W, DTYPE_CODE[dtype], sm_scale, int(causal), _p(q_row), t, _p(k),
                             _p(out)), "mpcref_row_lse")
    return float(out[0])


def static_topk(score, keep, local_keep):
    score = _c(score, np.float64)
    kept = np.empty(keep, np.int32)
    _ok(lib().mpcref_static_topk(score.shape[0], _p(score), keep, local_keep, _p(kept)),
        "mpcref_static_topk")
    return kept


def cluster_bounds(k, dtype, first, count):
    k = _c(k)
    n, d = k.shape
    rmax, rmin = np.empty(d), np.empty(d)
    _ok(lib().mpcref_cluster_bounds(n, d, DTYPE_CODE[dtype], _p(k), first, count, _p(rmax), _p(rmin)),
        "mpcref_cluster_bounds")
    return rmax, rmin


def centroid(rmax, rmin, alpha):
    return lib().mpcref_centroid(float(rmax), float(rmin), float(alpha))


SIMILARITY = {"linear": 0, "maxprod": 1, "mean": 2}
GROUP = {"sum": 0, "max": 1, "head": 2}


def rep_rows(similarity):
    """Rows of d floats per representative: r^max and r^min for the max-product bound."""
    return 2 if SIMILARITY[similarity] == 1 else 1


def cluster_scores(q_group, cent, dtype, similarity="linear", group="sum"):
    """q_group [G][d] (raw bits), cent [n][R][d] (or [n][d] when R = 1) float32 -> fp64 scores [n];
    the G heads' similarities are summed (group="sum") or their maximum taken (group="max")."""
    q_group, cent = _c(q_group), _c(cent, np.float32)
    G, d = q_group.shape
    n = cent.shape[0]
    out = np.empty(n, np.float64)
    _ok(lib().mpcref_cluster_scores(G, d, DTYPE_CODE[dtype], SIMILARITY[similarity], GROUP[group], _p(q_group), n,
                                    _p(cent), _p(out)), "mpcref_cluster_scores")
    return out


def cluster_mean(k, dtype, first, count):
    k = _c(k)
    n_tok, d = k.shape
    out = np.empty(d, np.float64)
    _ok(lib().mpcref_cluster_mean(n_tok, d, DTYPE_CODE[dtype], _p(k), first, count, _p(out)), "mpcref_cluster_mean")
    return out


def mp_bound(q, rmax, rmin):
    q, rmax, rmin = (_c(x, np.float64) for x in (q, rmax, rmin))
    out = np.empty(1, np.float64)
    _ok(lib().mpcref_mp_bound(q.shape[0], _p(q), _p(rmax), _p(rmin), _p(out)), "mpcref_mp_bound")
    return float(out[0])


def topk(score, k):
    score = _c(score, np.float64)
    idx = np.empty(k, np.int32)
    _ok(lib().mpcref_topk(score.shape[0], _p(score), k, _p(idx)), "mpcref_topk")
    return idx


def attend(q, rows, k, v, dtype, sm_scale):
    q, k, v = _c(q), _c(k), _c(v)
    rows = _c(rows, np.int32)
    d = q.shape[-1]
    out = np.empty(d, np.float64)
    lse = np.empty(1, np.float64)
    _ok(lib().mpcref_attend(d, DTYPE_CODE[dtype], sm_scale, _p(q), rows.shape[0], _p(rows), _p(k),
                            _p(v), _p(out), _p(lse)), "mpcref_attend")
    return out, float(lse[0])


# ------------------------------------------------------------------ whole tensors
def static_evict(q_win, k, v, dtype, *, keep, local_keep, sm_scale, causal=True, layer0=0,
                 share_period=1, share_start=2, kept_in=None, with_scores=False):
    """q_win [L][B][Hq][W][d], k/v [L][B][Hkv][T][d] -> (kept [L][B][Hkv][keep], k_out, v_out[, score])."""
    q_win, k, v = _c(q_win), _c(k), _c(v)
    L, B, Hq, W, d = q_win.shape
    Hkv, T = k.shape[2], k.shape[3]
    kept = np.zeros((L, B, Hkv, keep), np.int32) if kept_in is None else _c(kept_in, np.int32).copy()
    k_out = np.empty((L, B, Hkv, keep, d), k.dtype)
    v_out = np.empty_like(k_out)
    score = np.zeros((L, B, Hkv, T), np.float64) if with_scores else None
    _ok(lib().mpcref_static_evict(B, layer0, L, Hq, Hkv, d, DTYPE_CODE[dtype], T, W, keep, local_keep,
                                  sm_scale, int(causal), share_period, share_start, _p(q_win), _p(k),
                                  _p(v), _p(kept), _p(k_out), _p(v_out), _p(score)),
        "mpcref_static_evict")
    return (kept, k_out, v_out, score) if with_scores else (kept, k_out, v_out)


def build_clusters(k_cache, dtype, *, cluster, fanout, alpha=0.6, layer0=0, share_period=1,
                   share_start=2, similarity="linear"):
    """-> cent [L][B][Hkv][C][d], scent [L][B][Hkv][S][d]; with similarity="maxprod" the
    representative is two rows (r^max, r^min): [..][C][2][d], [..][S][2][d]."""
    k_cache = _c(k_cache)
    L, B, Hkv, Ts, d = k_cache.shape
    C = -(-Ts // cluster)
    S = -(-C // fanout)
    R = rep_rows(similarity)
    rows = (R, d) if R > 1 else (d,)
    cent = np.zeros((L, B, Hkv, C) + rows, np.float32)
    scent = np.zeros((L, B, Hkv, S) + rows, np.float32)
    _ok(lib().mpcref_build_clusters(B, layer0, L, Hkv, d, DTYPE_CODE[dtype], Ts, cluster, fanout, alpha,
                                    share_period, share_start, SIMILARITY[similarity], _p(k_cache), _p(cent),
                                    _p(scent)), "mpcref_build_clusters")
    return cent, scent


def select_clusters(q, cent, scent, dtype, *, Ts, cluster, fanout, k_super, k_clusters, layer0=0,
                    share_period=1, share_start=2, sel_in=None, similarity="linear", group="sum"):
    """-> sel [L][B][H][k_clusters] (ascending cluster ids) and their fp64 scores, with H = Hkv
    (group "sum" / "max": one selection per kv head) or H = Hq (group "head")."""
    q, cent, scent = _c(q), _c(cent, np.float32), _c(scent, np.float32)
    L, B, Hq, d = q.shape
    Hkv = cent.shape[2]
    H = Hq if group == "head" else Hkv
    sel = np.zeros((L, B, H, k_clusters), np.int32) if sel_in is None else _c(sel_in, np.int32).copy()
    score = np.zeros((L, B, H, k_clusters), np.float64)
    _ok(lib().mpcref_select_clusters(B, layer0, L, Hq, Hkv, d, DTYPE_CODE[dtype], Ts, cluster, fanout,
                                     k_super, k_clusters, share_period, share_start, SIMILARITY[similarity],
                                     GROUP[group], _p(q), _p(cent), _p(scent), _p(sel), _p(score)),
        "mpcref_select_clusters")
    return sel, score


def append_state(Ts, n_tail, cluster):
    """(Ts, n_tail) after one decode-time append (App. A.3; sealing rule is our reading)."""
    a, b = ctypes.c_int32(), ctypes.c_int32()
    _ok(lib().mpcref_append_state(Ts, n_tail, cluster, ctypes.byref(a), ctypes.byref(b)), "mpcref_append_state")
    return a.value, b.value


def sparse_decode_attn(q, k_cache, v_cache, sel, dtype, *, cluster, sm_scale, n_tail=0):
    """k_cache / v_cache [L][B][Hkv][Ts + n_tail][d]: clustered rows, then n_tail tail rows that every
    head attends. sel [L][B][Hkv][k] (one list per kv head) or [L][B][Hq][k] (one per query head)."""
    q, k_cache, v_cache, sel = _c(q), _c(k_cache), _c(v_cache), _c(sel, np.int32)
    L, B, Hq, d = q.shape
    Hkv, Ts = k_cache.shape[2], k_cache.shape[3] - n_tail
    out = np.empty((L, B, Hq, d), np.float64)
    lse = np.empty((L, B, Hq), np.float64)
    _ok(lib().mpcref_sparse_decode_attn(B, L, Hq, Hkv, d, DTYPE_CODE[dtype], Ts, n_tail, cluster, _p(q),
                                        _p(k_cache), _p(v_cache), _p(sel), sel.shape[2], sel.shape[-1], sm_scale,
                                        _p(out), _p(lse)), "mpcref_sparse_decode_attn")
    return out, lse


def commonality(idx, m):
    """idx [L][...][k] top-k index sets per layer -> commonality score of m + 1 adjacent layers
    (Sec. 3, Observation 3) for every unit of the middle axes (fp64, shape idx.shape[1:-1])."""
    idx = _c(idx, np.int32)
    L, k = idx.shape[0], idx.shape[-1]
    units = int(np.prod(idx.shape[1:-1], dtype=np.int64))
    out = np.empty(units, np.float64)
    _ok(lib().mpcref_commonality(L, units, k, m, _p(idx), _p(out)), "mpcref_commonality")
    return out.reshape(idx.shape[1:-1])


def dense_decode_attn(q, k_cache, v_cache, dtype, *, sm_scale):
    q, k_cache, v_cache = _c(q), _c(k_cache), _c(v_cache)
    L, B, Hq, d = q.shape
    Hkv, Ts = k_cache.shape[2], k_cache.shape[3]
    out = np.empty((L, B, Hq, d), np.float64)
    lse = np.empty((L, B, Hq), np.float64)
    _ok(lib().mpcref_dense_decode_attn(B, L, Hq, Hkv, d, DTYPE_CODE[dtype], Ts, _p(q), _p(k_cache),
                                       _p(v_cache), sm_scale, _p(out), _p(lse)),
        "mpcref_dense_decode_attn")
    return out, lse
