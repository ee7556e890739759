"""MI355X (gfx950) implementation of the MPCache decode hot path behind a C ABI.

The entry points mirror include/mpcache.h: mpc_static_evict, mpc_build_clusters, mpc_prefill (the
two in one call, the cluster build gathering its own rows), mpc_select_clusters,
mpc_sparse_decode_attn, mpc_decode_step (selection and attention in one launch) with
mpc_decode_step_status (its workspace's error word), mpc_append_kv (decode-time growth of the kept
cache) and mpc_commonality (agreement of adjacent layers' top-k sets). ``MPCachePath`` strings them together for one prefill and repeated
decode steps, with all buffers preallocated.
"""
from ._lib import (  # noqa: F401
    GROUP, MPC_OP_DECODE_ATTN, MPC_OP_DECODE_STEP, MPC_OP_SELECT, MPC_OP_STATIC_EVICT, MpcDims, MpcError,
    MpcEvictCfg, MpcSelectCfg, SIMILARITY, dims_of, lib, mpc_append_kv, mpc_build_clusters,
    mpc_commonality, mpc_decode_step, mpc_decode_step_status, mpc_prefill, mpc_select_clusters, mpc_sparse_decode_attn, mpc_static_evict,
    mpc_static_evict_noalloc, noalloc_limit, owner_layer, rep_rows, sel_heads, select_cfg, workspace, workspace_bytes)
from .pipeline import MPCachePath  # noqa: F401
