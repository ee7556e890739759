"""Preallocated prefill + decode path over the C-ABI entry points."""
import ctypes
import math

import torch

from . import _lib as L


class MPCachePath:
    """Buffers and calls for one workload: static eviction and cluster build at prefill, then
    selection + sparse attention for every decode step, all layers of the block per call.

    decode() runs them as two calls (mpc_select_clusters, mpc_sparse_decode_attn); decode_fused()
    runs both in one launch (mpc_decode_step) with the same results. With `capacity` rows per
    (layer, sequence, kv head) above `keep`, append() adds each decoded token's k, v to the cache
    (mpc_append_kv) and later steps select over the grown clusters and attend the tail."""

    def __init__(self, *, n_layers, batch, n_q_heads, n_kv_heads, head_dim, dtype, T, window, keep,
                 local_keep, cluster, fanout, k_super, k_clusters, share_period, share_start=2,
                 alpha=0.6, causal=True, layer0=0, device="cuda", keep_scores=False, similarity="linear",
                 group="sum", capacity=None):
        self.L, self.B, self.Hq, self.Hkv, self.d = n_layers, batch, n_q_heads, n_kv_heads, head_dim
        self.dtype, self.T, self.W, self.keep = dtype, T, window, keep
        self.local_keep, self.causal, self.layer0 = local_keep, causal, layer0
        self.cluster, self.k_clusters = cluster, k_clusters
        self.share_period, self.share_start = share_period, share_start
        self.sm_scale = 1.0 / math.sqrt(head_dim)
        self.rows = keep if capacity is None else capacity
        if self.rows < keep:
            raise ValueError("capacity below the kept tokens")
        self.C = -(-keep // cluster)
        self.S = -(-self.C // fanout)
        n_c = -(-self.rows // cluster)
        self.Ts, self.n_tail = keep, 0
        self.cfg = L.select_cfg(cluster, fanout, k_super, k_clusters, alpha, share_period, share_start, similarity,
                                group)
        self.Hsel = L.sel_heads(self.cfg, n_q_heads, n_kv_heads)  # selection lists per (layer, sequence)
        R = L.rep_rows(similarity)
        rep = (R, head_dim) if R > 1 else (head_dim,)
        dev = torch.device(device)
        kv_shape = (n_layers, batch, n_kv_heads)
        self.kept = torch.zeros(*kv_shape, keep, dtype=torch.int32, device=dev)
        self.k_s = torch.empty(*kv_shape, self.rows, head_dim, dtype=dtype, device=dev)
        self.v_s = torch.empty_like(self.k_s)
        self.cent = torch.zeros(*kv_shape, n_c, *rep, dtype=torch.float32, device=dev)
        self.scent = torch.zeros(*kv_shape, -(-n_c // fanout), *rep, dtype=torch.float32, device=dev)
        self.sel = torch.zeros(n_layers, batch, self.Hsel, k_clusters, dtype=torch.int32, device=dev)
        self.sel_score = torch.zeros(n_layers, batch, self.Hsel, k_clusters, dtype=torch.float32, device=dev)
        self.out = torch.empty(n_layers, batch, n_q_heads, head_dim, dtype=dtype, device=dev)
        self.lse = torch.empty(n_layers, batch, n_q_heads, dtype=torch.float32, device=dev)
        self.token_score = (torch.zeros(*kv_shape, T, dtype=torch.float32, device=dev)
                            if keep_scores else None)
        self.row_lse = (torch.zeros(n_layers, batch, n_q_heads, window, dtype=torch.float32, device=dev)
                        if keep_scores else None)
        qd = L.MpcDims(batch=batch, layer0=layer0, n_layers=n_layers, n_q_heads=n_q_heads,
                       n_kv_heads=n_kv_heads, head_dim=head_dim, dtype=L.DTYPE_CODE[dtype])
        ecfg = L.MpcEvictCfg(window=window, keep=keep, local_keep=local_keep, sm_scale=self.sm_scale,
                             causal=int(causal), share_period=share_period, share_start=share_start)
        self.ws_evict = L.workspace(L.workspace_bytes(L.MPC_OP_STATIC_EVICT, qd, T, ecfg), dev)
        self.ws_decode = L.workspace(L.workspace_bytes(L.MPC_OP_DECODE_ATTN, qd, keep), dev)
        self.ws_step = L.workspace(L.workspace_bytes(L.MPC_OP_DECODE_STEP, qd, keep, self.cfg), dev)

        # argument tuples of the per-step calls, built once per cache state (only the query pointer
        # and the stream change between decode steps that do not grow the cache)
        self._qdims = qd
        kvd = L.dims_of(self.out, self.k_s, layer0)
        self._kvdims = kvd
        lib = L.lib()
        self._select_fn = lib.mpc_select_clusters
        self._attend_fn = lib.mpc_sparse_decode_attn
        self._step_fn = lib.mpc_decode_step
        self._prepare()

    def _prepare(self):
        P = lambda t: None if t is None else ctypes.c_void_p(t.data_ptr())
        kvd, Ts, nt = self._kvdims, self.Ts, self.n_tail
        self.C = -(-Ts // self.cluster)  # selectable clusters of the current cache
        self._select_args = (ctypes.byref(kvd), Ts, ctypes.byref(self.cfg))
        self._select_tail = (P(self.cent), P(self.scent), P(self.sel), P(self.sel_score), None, 0)
        self._attend_args = (ctypes.byref(kvd), Ts, nt, self.cluster)
        self._attend_mid = (P(self.k_s), P(self.v_s), P(self.sel), self.Hsel, self.k_clusters, self.sm_scale,
                            P(self.out), P(self.lse), P(self.ws_decode), self.ws_decode.numel())
        self._step_args = (ctypes.byref(kvd), Ts, nt, ctypes.byref(self.cfg))
        self._step_tail = (P(self.cent), P(self.scent), P(self.k_s), P(self.v_s), self.sm_scale, P(self.sel),
                           P(self.sel_score), P(self.out), P(self.lse), P(self.ws_step), self.ws_step.numel())

    def prefill(self, q_win, k, v, stream=None, fused=True):
        """Static eviction into rows [0, keep) of the kept cache and the cluster build; the cache
        state returns to (keep, 0). fused: one call (mpc_prefill), else mpc_static_evict then
        mpc_build_clusters (same results)."""
        kw = dict(keep=self.keep, local_keep=self.local_keep, sm_scale=self.sm_scale, causal=self.causal,
                  layer0=self.layer0, share_period=self.share_period, share_start=self.share_start,
                  token_score=self.token_score, row_lse=self.row_lse, ws=self.ws_evict, stream=stream)
        if fused:
            L.mpc_prefill(q_win, k, v, self.kept, self.k_s, self.v_s, self.cent, self.scent, self.cfg, **kw)
        else:
            L.mpc_static_evict(q_win, k, v, self.kept, self.k_s, self.v_s, **kw)
            L.mpc_build_clusters(self.k_s, self.cent, self.scent, self.cfg, Ts=self.keep, layer0=self.layer0,
                                 stream=stream)
        if (self.Ts, self.n_tail) != (self.keep, 0):
            self.Ts, self.n_tail = self.keep, 0
            self._prepare()

    def append(self, k_new, v_new, stream=None):
        """Adds one decoded token's k, v ([L][B][Hkv][d]) to every layer's cache."""
        self.Ts, self.n_tail = L.mpc_append_kv(k_new, v_new, self.k_s, self.v_s, self.cent, self.scent, self.cfg,
                                               Ts=self.Ts, n_tail=self.n_tail, layer0=self.layer0, stream=stream)
        self._prepare()

    def select(self, q, stream=None):
        """q: [L][B][Hq][d] contiguous CUDA tensor of the path's dtype."""
        st = L._stream(stream)
        L._check("mpc_select_clusters",
                 self._select_fn(*self._select_args, ctypes.c_void_p(q.data_ptr()), *self._select_tail, st))

    def attend(self, q, stream=None):
        st = L._stream(stream)
        L._check("mpc_sparse_decode_attn",
                 self._attend_fn(*self._attend_args, ctypes.c_void_p(q.data_ptr()), *self._attend_mid, st))

    def attend_call(self, sel):
        """A prepared attention call that reads the selection from `sel` (same shape as self.sel)
        instead of self.sel: returns f(q, stream=None)."""
        if sel.shape != self.sel.shape or sel.dtype != torch.int32 or not sel.is_contiguous():
            raise ValueError("sel must be a contiguous int32 tensor shaped like the path's selection")
        mid = (self._attend_mid[0], self._attend_mid[1], ctypes.c_void_p(sel.data_ptr())) + self._attend_mid[3:]

        def call(q, stream=None):
            L._check("mpc_sparse_decode_attn",
                     self._attend_fn(*self._attend_args, ctypes.c_void_p(q.data_ptr()), *mid, L._stream(stream)))
        return call

    def decode(self, q, stream=None):
        self.select(q, stream)
        self.attend(q, stream)
        return self.out

    def capture(self, fn, *args):
        """A HIP graph (torch.cuda.CUDAGraph) of fn(*args), e.g. capture(self.decode, q_buf) or
        capture(self.prefill, q_win, k, v). Replaying it reruns the same kernels on the same buffers,
        so the caller refills the input buffers between replays. The entry points only enqueue kernels
        (no allocation, memset or host wait), so capture needs nothing else from them. A graph keeps
        the cache state (Ts, n_tail) it was captured with: capture again after append()."""
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn(*args)
        return g

    def decode_fused(self, q, stream=None):
        st = L._stream(stream)
        L._check("mpc_decode_step",
                 self._step_fn(*self._step_args, ctypes.c_void_p(q.data_ptr()), *self._step_tail, st))
        return self.out
