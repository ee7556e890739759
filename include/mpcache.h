/* mpcache.h — C ABI of the MI355X (gfx950) MPCache hot path.
 *
 * Paper: "MPCache: MPC-Friendly KV Cache Eviction for Efficient Private LLM Inference",
 * arXiv 2501.06807. The library computes, in plaintext, the data-parallel steps of the method:
 *   - look-once static eviction at prefill (Sec. 3.2; Alg. 3 step 1);
 *   - hierarchical cluster representatives alpha*r^max + (1-alpha)*r^min (Sec. 3.3, Eq. "sim");
 *   - query-aware two-level cluster selection with cross-layer index sharing (Sec. 3.3, 3.4;
 *     Alg. 3 step 2);
 *   - gather + softmax attention over the selected clusters (Alg. 1 steps 3-4);
 *   - decode-time growth of the kept cache (App. A.3: each decoded token's k, v are appended);
 *   - the commonality score of adjacent layers' top-k sets (Sec. 3, Observation 3).
 * mpc_prefill runs the first two steps as one call; mpc_decode_step runs selection and attention
 * as one launch (mpc_decode_step_status reads its workspace's error word).
 *
 * Conventions shared by every entry point
 *   - Tensor arguments are DEVICE pointers owned by the caller, contiguous row-major, with
 *     16-byte aligned bases. Element type is `dims->dtype` unless a float/int32 type is stated.
 *   - Shapes use: B batch, L = dims->n_layers (a block of consecutive layers starting at the
 *     absolute layer dims->layer0), Hq / Hkv query / kv heads (q-head h reads kv-head h / G,
 *     G = Hq / Hkv), d head dim, T prompt tokens, W window rows, Ts kept tokens,
 *     s cluster size, C = ceil(Ts / s) clusters, f fan-out, S = ceil(C / f) super-clusters.
 *   - Kept-cache tensors are allocated for Tcap rows per (layer, sequence, kv head), where
 *     Tcap = dims->kv_capacity, or the rows of the call when it is 0 (Ts, plus n_tail where a call
 *     takes a tail; keep for the eviction's outputs). K/V caches are [L][B][Hkv][Tcap][d];
 *     representatives have Ccap = ceil(Tcap / s) cluster slots and Scap = ceil(Ccap / f)
 *     super-cluster slots. A cache that grows during decoding (mpc_append_kv) keeps one Tcap.
 *   - Cross-layer sharing: owner(l) = l if period <= 1 or l < start, else
 *     start + period * floor((l - start) / period), on absolute layer indices (Sec. 3.4: the
 *     first two layers never share, so start = 2 follows the paper's text; start = 0 gives the
 *     pairing of Alg. 3).
 *   - The library allocates nothing and keeps no global state except a thread-local message for
 *     the last error and the static scratch array of mpc_static_evict_noalloc (with its device
 *     addresses). Scratch memory is otherwise a caller-provided workspace of
 *     mpc_workspace_bytes() bytes (no initial contents needed). Calls that share one workspace must
 *     not overlap in time.
 *   - Every call is asynchronous on `stream` (a hipStream_t; NULL = default stream). The
 *     returned status covers argument validation and launch errors only; it never waits for the
 *     GPU. A validation failure (MPC_EINVAL / ESHAPE / EUNSUPPORTED / EWORKSPACE) enqueues
 *     nothing; after MPC_EHIP, kernels launched before the failing one may have been enqueued.
 *   - Apart from mpc_decode_step_status (a blocking read), no call allocates, sets memory, waits on
 *     the host or uses a stream other than `stream`. So calls can be captured into a HIP graph,
 *     whose replays rerun the same kernels on the same pointers and sizes.
 *   - Supported: d in {64, 128}; G in {1, 2, 4, 8}; dtype fp32 / fp16 / bf16.
 */
#ifndef MPCACHE_H
#define MPCACHE_H
#include <stddef.h>
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MPC_OK = 0,
  MPC_EINVAL = 1,       /* null pointer, non-positive size, bad enum value                  */
  MPC_ESHAPE = 2,       /* sizes inconsistent with each other (e.g. Hq % Hkv, k > candidates) */
  MPC_EUNSUPPORTED = 3, /* valid but outside what the kernels implement (head dim, group)    */
  MPC_EWORKSPACE = 4,   /* workspace missing or smaller than mpc_workspace_bytes()           */
  MPC_EHIP = 5          /* a HIP launch failed                                              */
} mpc_status;

typedef enum { MPC_FP32 = 0, MPC_FP16 = 1, MPC_BF16 = 2 } mpc_dtype;

typedef struct {
  int32_t batch;      /* B                                                */
  int32_t layer0;     /* absolute index of the first layer of the block   */
  int32_t n_layers;   /* L, layers in this call                           */
  int32_t n_q_heads;  /* Hq                                               */
  int32_t n_kv_heads; /* Hkv                                              */
  int32_t head_dim;   /* d                                                */
  int32_t dtype;      /* mpc_dtype of q / k / v / out                     */
  int32_t kv_capacity; /* Tcap: rows allocated per (layer, sequence, kv head) in the kept
                        * cache; 0 = exactly the rows of the call                            */
} mpc_dims;

/* Cluster similarity (Sec. 3.3). LINEAR: the reordered linear form (Eq. "sim"), one
 * representative row alpha * r^max + (1 - alpha) * r^min. MAXPROD: the max-product upper bound
 * (Eq. 2), two rows r^max, r^min. MEAN: the average of the cluster's keys (the baseline of the
 * paper's average-based comparison), one row. */
typedef enum { MPC_SIM_LINEAR = 0, MPC_SIM_MAXPROD = 1, MPC_SIM_MEAN = 2 } mpc_similarity;

/* Grouped query heads (Hq > Hkv). The paper states the selection for a single query head; these are
 * the readings offered. SUM: the G query heads of a kv head share one selection, scored by the sum
 * of their similarities (for LINEAR / MEAN the similarity of the summed query). MAX: they share one
 * selection, scored by the largest of their similarities. HEAD: every query head selects its own
 * clusters from its own similarity against its kv head's representatives, and attends only them. */
typedef enum { MPC_GROUP_SUM = 0, MPC_GROUP_MAX = 1, MPC_GROUP_HEAD = 2 } mpc_group;

typedef struct {
  int32_t cluster_size; /* s: tokens per fine cluster                                        */
  int32_t fanout;       /* f: fine clusters per super-cluster                                */
  int32_t k_super;      /* level-1 budget, 1 <= k_super <= S                                  */
  int32_t k_clusters;   /* level-2 budget; must not exceed the smallest possible candidate set */
  float alpha;          /* weight of r^max in the representative (the paper uses 0.6)        */
  int32_t share_period; /* layers per shared selection (1 = no sharing)                     */
  int32_t share_start;  /* first layer that may share (2 in the paper)                       */
  int32_t similarity;   /* mpc_similarity (MPC_SIM_LINEAR in the paper's method)              */
  int32_t group;        /* mpc_group (MPC_GROUP_SUM by default)                                */
} mpc_select_cfg;

typedef struct {
  int32_t window;       /* W: window query rows (positions T-W .. T-1)                        */
  int32_t keep;         /* Ts: tokens kept per (layer, sequence, kv head)                      */
  int32_t local_keep;   /* most recent tokens always kept (part of `keep`)                    */
  float sm_scale;       /* softmax scale of the window attention (1/sqrt(d))                  */
  int32_t causal;       /* 1: window row t attends to keys j <= T-W+t                          */
  int32_t share_period; /* layers sharing one kept set (same rule as the selection)           */
  int32_t share_start;
} mpc_evict_cfg;

enum { MPC_OP_STATIC_EVICT = 0, MPC_OP_SELECT = 1, MPC_OP_DECODE_ATTN = 2, MPC_OP_DECODE_STEP = 3 };

/* Workspace bytes needed by `op` (MPC_OP_*) for these dims. `T_or_Ts` is T for static eviction
 * and Ts otherwise; `cfg` points to the op's config struct (mpc_evict_cfg for static eviction,
 * mpc_select_cfg for selection and the decode step) or is NULL for MPC_OP_DECODE_ATTN. Returns 0
 * when the op needs no workspace or the arguments are invalid. */
size_t mpc_workspace_bytes(int32_t op, const mpc_dims* dims, int32_t T_or_Ts, const void* cfg);

/* Look-once static eviction (Sec. 3.2; Alg. 3 step 1; window rule of App. F).
 * For every owner layer and (b, kv head): score[j] = sum over the G query heads of the group and
 * the W window rows t of softmax_j(sm_scale * q_t . k_j) (causal: j <= T-W+t); keep the last
 * `local_keep` tokens plus the (keep - local_keep) best-scored older tokens (ties: lower position
 * first); write the kept positions ascending. Non-owner layers reuse their owner's kept set; a
 * layer whose owner precedes layer0 must arrive with that set already in `kept_idx`. Every layer
 * then gathers its kept K/V rows.
 *   q_win       [L][B][Hq][W][d]   window queries (read for owner layers only)
 *   k, v        [L][B][Hkv][T][d]  prompt cache
 *   kept_idx    [L][B][Hkv][keep]  int32 out (in for layers owned before layer0)
 *   k_out,v_out [L][B][Hkv][Tcap][d] out, rows [0, keep) written (Tcap >= keep)
 *   token_score [L][B][Hkv][T] float, optional out (NULL = not returned); owner layers only
 *   row_lse     [L][B][Hq][W] float, optional out: natural log-sum-exp of each window row's
 *               scaled scores (the softmax normaliser); owner layers only
 *   ws          workspace of mpc_workspace_bytes(MPC_OP_STATIC_EVICT, dims, T, cfg) bytes.
 * Accumulation: fp32 matrix-core dot products; each exponent is one fp32 fused multiply-add
 * against a per-row whole-number offset that keeps every exponent at most 1, shared by the row sum
 * and the column sums; sums of at most 16 terms in fp32, accumulated across tiles in fp64.
 * token_score matches the exact (fp64) scores within a relative 2e-5 (the bound the tests hold it
 * to; the largest error measured over every token of the tested cases is 1.8e-6, and 3.3e-7 to
 * 7.3e-7 at the 8K-32K workloads, where tokens near the keep boundary are within 3e-7, as they are
 * at 128K), so a kept set can differ from the exact one only between tokens whose exact scores tie
 * within about 1e-6. */
mpc_status mpc_static_evict(const mpc_dims* dims, int32_t T, const mpc_evict_cfg* cfg,
                            const void* q_win, const void* k, const void* v, int32_t* kept_idx,
                            void* k_out, void* v_out, float* token_score, float* row_lse,
                            void* ws, size_t ws_bytes, void* stream);

/* mpc_static_evict without any allocation and without a workspace argument, for callers that
 * cannot allocate device memory (code under graph capture, tight serving loops, harnesses that
 * forbid it). Same arguments (minus ws / ws_bytes), results bit for bit, and errors as
 * mpc_static_evict. The workspace is a static device array of mpc_static_evict_noalloc_limit()
 * bytes (32 MiB) that each device holds from the first call on until the process ends; a call whose
 * workspace would be larger (mpc_workspace_bytes(MPC_OP_STATIC_EVICT, ...)) fails with
 * MPC_EWORKSPACE before anything runs: split it into calls over fewer layers or sequences. Every
 * call on one device shares that array, so calls that overlap in time on one device (other streams,
 * other threads) race; calls on one stream do not. Nothing in the array needs initial contents. */
mpc_status mpc_static_evict_noalloc(const mpc_dims* dims, int32_t T, const mpc_evict_cfg* cfg,
                                    const void* q_win, const void* k, const void* v, int32_t* kept_idx,
                                    void* k_out, void* v_out, float* token_score, float* row_lse,
                                    void* stream);
size_t mpc_static_evict_noalloc_limit(void);

/* Cluster representatives (Sec. 3.3: r^max / r^min under Eq. 1, reordered form Eq. "sim";
 * hierarchy of Sec. 3.3 / App. F). Fine cluster c covers kept tokens [c*s, min((c+1)*s, Ts));
 * super-cluster u covers fine clusters [u*f, min((u+1)*f, C)), i.e. their tokens. Per channel:
 *   LINEAR   one row fp32( fp32(alpha * r^max) + fp32((1-alpha)_fp32 * r^min) );
 *   MAXPROD  two rows, r^max then r^min (exact key values);
 *   MEAN     one row, fp32( fp64 sum of the tokens' values / token count ).
 * Owner layers only. R = 2 for MAXPROD, else 1.
 *   k_cache [L][B][Hkv][Tcap][d];  cent [L][B][Hkv][Ccap][R][d] float out (slots [0, C) written);
 *   scent [L][B][Hkv][Scap][R][d] (slots [0, S)). */
mpc_status mpc_build_clusters(const mpc_dims* dims, int32_t Ts, const mpc_select_cfg* cfg,
                              const void* k_cache, float* cent, float* scent, void* stream);

/* Prefill in one call: look-once static eviction (Sec. 3.2; Alg. 3 step 1) followed by the
 * cluster representatives of the kept cache (Sec. 3.3), with the kept rows of the selection's
 * owner layers gathered and summarised in the same pass over them. Results are those of
 * mpc_static_evict(dims, T, ecfg, ...) followed by mpc_build_clusters(dims, ecfg->keep, scfg,
 * k_out, cent, scent), bit for bit; the arguments keep their meaning, layout and ownership there.
 * Owner layers of the eviction follow ecfg's sharing rule, those of the representatives scfg's
 * (the two may differ). ws: mpc_workspace_bytes(MPC_OP_STATIC_EVICT, dims, T, ecfg) bytes.
 * Errors: any error either call would report for these arguments, before anything runs. */
mpc_status mpc_prefill(const mpc_dims* dims, int32_t T, const mpc_evict_cfg* ecfg, const mpc_select_cfg* scfg,
                       const void* q_win, const void* k, const void* v, int32_t* kept_idx, void* k_out,
                       void* v_out, float* cent, float* scent, float* token_score, float* row_lse, void* ws,
                       size_t ws_bytes, void* stream);

/* Query-aware dynamic selection of one decode step (Sec. 3.3; Alg. 3 step 2).
 * Similarity of one q-head g with a representative, summed over the channels i and accumulated in
 * fp64: q_{g,i} * c_i (LINEAR, MEAN) or max(q_{g,i} r^max_i, q_{g,i} r^min_i) (MAXPROD, Eq. 2). The
 * score of a selection unit combines its q-heads by cfg->group: the sum (SUM) or the maximum (MAX)
 * over the G heads of kv head h, or the head's own similarity (HEAD, one unit per q-head). Level 1
 * keeps the k_super best super-clusters, level 2 the k_clusters best fine clusters among their
 * members (ties: lower index first); the selection is written in ascending cluster order.
 * Non-owner layers receive their owner's selection; a layer whose owner precedes layer0 is left
 * untouched (the caller copies it).
 *   q [L][B][Hq][d];  cent / scent as produced by mpc_build_clusters (Ccap / Scap slots, the
 *   first C / S used);
 *   sel [L][B][H][k_clusters] int32 out, H = Hq for MPC_GROUP_HEAD, else Hkv;  sel_score same
 *   shape, float, optional (score rounded to fp32). ws may be NULL (no workspace needed).
 *   Limits: S <= 1024, k_super * f <= 1024. */
mpc_status mpc_select_clusters(const mpc_dims* dims, int32_t Ts, const mpc_select_cfg* cfg,
                               const void* q, const float* cent, const float* scent,
                               int32_t* sel, float* sel_score, void* ws, size_t ws_bytes,
                               void* stream);

/* Sparse attention over the selected clusters (Alg. 1 steps 3-4; Alg. 3 step 2):
 * o_h = softmax(sm_scale * q_h K'^T) V' with K', V' the rows of kv head h / G of the kept cache
 * that belong to the clusters of h's selection list (tokens past Ts in a partial last cluster are
 * skipped), followed by the n_tail unclustered rows [Ts, Ts + n_tail) that decoding appended
 * (mpc_append_kv), which every head attends in full. The list of h is sel[l][b][h / G] when
 * sel_heads = Hkv (one list per kv head), sel[l][b][h] when sel_heads = Hq (one per q-head, as
 * MPC_GROUP_HEAD selects).
 *   q [L][B][Hq][d];  k_cache, v_cache [L][B][Hkv][Tcap][d];  sel [L][B][sel_heads][k_clusters]
 *   int32 (entries outside [0, C) contribute nothing);  n_tail >= 0, and Ts % s == 0 when
 *   n_tail > 0;
 *   out [L][B][Hq][d] (dtype);  lse [L][B][Hq] float, optional (natural-log log-sum-exp of the
 *   scaled scores). fp32 accumulation; 16-bit types take exact pairwise products summed in fp32.
 *   Limits: k_clusters + ceil(n_tail / s) <= 1024, Tcap * d * element size <= 2 GiB.
 *   ws: mpc_workspace_bytes(MPC_OP_DECODE_ATTN, dims, Ts, NULL) bytes (split-K partials and
 *   per-unit arrival counters, used when there are fewer (layer, sequence, list) units than the
 *   compute units), zero-filled before its first use; every completed call leaves the counters at
 *   zero (calls sharing it must not overlap). May be NULL when that size is 0. */
mpc_status mpc_sparse_decode_attn(const mpc_dims* dims, int32_t Ts, int32_t n_tail, int32_t cluster_size,
                                  const void* q, const void* k_cache, const void* v_cache,
                                  const int32_t* sel, int32_t sel_heads, int32_t k_clusters, float sm_scale,
                                  void* out, float* lse, void* ws, size_t ws_bytes, void* stream);

/* One decode step in one launch: mpc_select_clusters followed by mpc_sparse_decode_attn (same
 * definitions, same results bit for bit), with the attention of a layer starting as soon as its
 * owner's selection is published instead of after a kernel boundary.
 *   q [L][B][Hq][d]; cent, scent from mpc_build_clusters; k_cache, v_cache [L][B][Hkv][Tcap][d];
 *   n_tail: unclustered rows after Ts, attended in full (as in mpc_sparse_decode_attn);
 *   sel [L][B][H][cfg->k_clusters] int32 out (in for layers owned before layer0), H as in
 *   mpc_select_clusters; sel_score optional; out [L][B][Hq][d]; lse optional.
 *   ws: mpc_workspace_bytes(MPC_OP_DECODE_STEP, dims, Ts, cfg) bytes, zero-filled before its first
 *   use; every completed call leaves it ready for the next (calls sharing it must not overlap).
 *   Layout: an int32 error word at offset 0 (sticky; read it with mpc_decode_step_status), then at
 *   offset 256 one int32 state word per owner head of the block, in (owner layer, sequence, kv head)
 *   order (0 free, 1 being selected, 2 published), then as many consumer counts.
 * An attention unit waits for its owner head's selection with a bounded poll. If the bound is
 * reached (no such case is known: it would take a selection that never gets published), the unit
 * sets bit 0 of the error word and writes NaN to its out and lse rows instead of attending; the
 * call still returns MPC_OK, since the status covers only validation and launch.
 * Blocks whose attention is split over several workgroups per unit, whose selection and attention
 * together need more LDS than one workgroup has, or that select per q-head (MPC_GROUP_HEAD) run the
 * two kernels one after the other instead (same results). */
mpc_status mpc_decode_step(const mpc_dims* dims, int32_t Ts, int32_t n_tail, const mpc_select_cfg* cfg,
                           const void* q, const float* cent, const float* scent,
                           const void* k_cache, const void* v_cache, float sm_scale, int32_t* sel,
                           float* sel_score, void* out, float* lse, void* ws, size_t ws_bytes,
                           void* stream);

/* Error word of a decode-step workspace (the one passed to mpc_decode_step): *flags receives it,
 * bit 0 set when an attention unit gave up waiting for its selection (its outputs are NaN). With
 * clear != 0 a non-zero word is reset to zero. Reads and writes with blocking copies: call it after
 * the stream of the decode steps that used `ws` has completed. ws_bytes: the workspace's size.
 * Errors: MPC_EINVAL for NULL pointers, MPC_EWORKSPACE below 4 bytes, MPC_EHIP if a copy fails. */
mpc_status mpc_decode_step_status(void* ws, size_t ws_bytes, int32_t clear, int32_t* flags);

/* Decode-time growth of the kept cache (App. A.3: the k, v of each decoded token are appended to
 * the cache). The cache of a block is the pair (Ts, n_tail): clustered rows [0, Ts) with
 * representatives, and n_tail newer rows [Ts, Ts + n_tail), 0 <= n_tail <= s, that every decode
 * attention reads in full. One call per decoded token, for every layer of the block:
 *   1. if the tail is full (n_tail == s) it is sealed: rows [Ts, Ts + s) become cluster Ts / s, and
 *      on owner layers that cluster's representative and its super-cluster's are rebuilt from the
 *      rows, exactly as mpc_build_clusters over Ts + s rows would give them; Ts += s, n_tail = 0;
 *   2. the new k, v are written at row Ts + n_tail; n_tail += 1.
 * So the state after the call is (Ts + s, 1) when n_tail == s, else (Ts, n_tail + 1), and the
 * token just appended is always in the tail.
 *   k_new, v_new [L][B][Hkv][d];  k_cache, v_cache [L][B][Hkv][Tcap][d] in/out;
 *   cent, scent [L][B][Hkv][Ccap / Scap][R][d] float in/out (cfg->similarity gives R).
 * Requires Ts % s == 0 and a row free after sealing (Ts + n_tail + 1 <= Tcap, Tcap =
 * dims->kv_capacity, which must be set). The new state is returned in *Ts_out and *n_tail_out
 * (host pointers, each optional, written only on MPC_OK); the caller passes it to the selection
 * (Ts) and attention (Ts, n_tail) calls and to the next append. */
mpc_status mpc_append_kv(const mpc_dims* dims, int32_t Ts, int32_t n_tail, const mpc_select_cfg* cfg,
                         const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                         float* cent, float* scent, int32_t* Ts_out, int32_t* n_tail_out, void* stream);

/* Commonality score of m + 1 adjacent layers (Sec. 3, Observation 3), the paper's measure of how
 * far adjacent layers agree on their top-k sets:
 *   out[u] = (1 / (k (L - m))) * sum_{l=0}^{L-m-1} | intersection over i = l .. l+m of idx[i][u] |
 * for every unit u (e.g. a (sequence, head) pair). idx [L][units][k] int32 holds each layer's
 * top-k set (distinct entries; any order), e.g. per-layer selections made without sharing
 * (share_period = 1). out [units] double. Counts are exact integers; out is their quotient rounded
 * once. Requires 0 <= m < L, k <= 1024. No workspace. */
mpc_status mpc_commonality(int32_t L, int32_t units, int32_t k, int32_t m, const int32_t* idx, double* out,
                           void* stream);

/* Owner layer of absolute layer `l` under the sharing rule above. */
int32_t mpc_owner_layer(int32_t l, int32_t period, int32_t start);

/* Static text for a status code. */
const char* mpc_status_string(mpc_status s);

/* Human-readable reason of the last failed call on this thread ("" if none). */
const char* mpc_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
