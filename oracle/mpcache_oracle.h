/* CPU oracle for the MPCache decode/prefill hot path. TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, fp64 implementation of what the paper defines, written to be checked against the
 * paper by eye. It shares no code with the GPU library. Only the test-suite, the smoke check and
 * the benchmark's CPU-baseline leg may load it; the product path never calls it.
 *
 * Paper: "MPCache: MPC-Friendly KV Cache Eviction for Efficient Private LLM Inference"
 * (arXiv 2501.06807). Citations name the section / equation / algorithm they follow.
 *
 * Conventions
 *   - dtype codes: 0 = fp32, 1 = fp16, 2 = bf16; tensors are raw element bits, converted exactly
 *     to double on load.
 *   - layouts are row-major and contiguous:
 *       q_win [n_layers][B][Hq][W][d], k/v [n_layers][B][Hkv][T][d], q [n_layers][B][Hq][d],
 *       kept  [n_layers][B][Hkv][keep], cent [n_layers][B][Hkv][C][R][d], scent [...][S][R][d]
 *       (R = 2 rows r^max, r^min for the max-product bound, else 1),
 *       sel   [n_layers][B][Hkv][k_clusters] (or [..][Hq][..] with one selection per query head),
 *       out [n_layers][B][Hq][d].
 *   - q-head h reads kv-head h / (Hq / Hkv).
 *   - layer indices passed to the sharing rule are absolute: layer0 + local index.
 *   - return value: 0 ok, 1 invalid argument, 2 inconsistent shape, 3 unsupported.
 *
 * Functions whose result is pinned only by our reading of a silent or garbled passage say so.
 */
#ifndef MPCACHE_ORACLE_H
#define MPCACHE_ORACLE_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

/* ---- rules (hyper-parameters of the method) ---- */
int32_t mpcref_window_rows(int32_t T);
int32_t mpcref_owner_layer(int32_t layer, int32_t period, int32_t start);
int32_t mpcref_keep_tokens(int32_t T, double static_ratio, int32_t cluster);
int32_t mpcref_level1_keep(int32_t n_super, double final_ratio);
int32_t mpcref_level2_keep(int32_t keep, double dynamic_ratio, int32_t cluster, int32_t n_cand);
/* Same budget with eta read as a fraction of the prompt length T (Fig. 9 caption), not of the
 * post-eviction cache. */
int32_t mpcref_level2_keep_of_prompt(int32_t T, double dynamic_ratio, int32_t cluster, int32_t n_cand);

/* ---- per-head steps ---- */
int mpcref_token_scores(int32_t G, int32_t d, int32_t T, int32_t W, int32_t dtype, float sm_scale,
                        int32_t causal, const void* q_win /*[G][W][d]*/, const void* k /*[T][d]*/,
                        double* score /*[T]*/, double* row_lse /*[G][W] or NULL*/);
int mpcref_row_lse(int32_t d, int32_t T, int32_t W, int32_t dtype, float sm_scale, int32_t causal,
                   const void* q_row /*[d]*/, int32_t t, const void* k, double* lse);
int mpcref_static_topk(int32_t T, const double* score, int32_t keep, int32_t local_keep,
                       int32_t* kept /*[keep], ascending*/);
int mpcref_cluster_bounds(int32_t n_tok, int32_t d, int32_t dtype, const void* k /*[n_tok][d]*/,
                          int32_t first, int32_t count, double* rmax, double* rmin);
int mpcref_cluster_mean(int32_t n_tok, int32_t d, int32_t dtype, const void* k /*[n_tok][d]*/,
                        int32_t first, int32_t count, double* mean);
float mpcref_centroid(double rmax, double rmin, float alpha);
/* similarity: 0 linear alpha r^max + (1 - alpha) r^min, 1 max-product bound (rows r^max, r^min),
 * 2 average; representatives have (similarity == 1 ? 2 : 1) rows of d floats. group: the G heads'
 * similarities are summed (0) or their maximum is taken (1). */
int mpcref_cluster_scores(int32_t G, int32_t d, int32_t dtype, int32_t similarity, int32_t group,
                          const void* q /*[G][d]*/, int32_t n, const float* rep /*[n][R][d]*/,
                          double* score);
int mpcref_mp_bound(int32_t d, const double* q, const double* rmax, const double* rmin,
                    double* bound);
int mpcref_topk(int32_t n, const double* score, int32_t k, int32_t* idx /*[k], rank order*/);
int mpcref_attend(int32_t d, int32_t dtype, float sm_scale, const void* q /*[d]*/, int32_t n_tok,
                  const int32_t* rows, const void* k, const void* v, double* out /*[d]*/,
                  double* lse);

/* ---- whole-tensor mirrors of the library entry points (host pointers) ---- */
int mpcref_static_evict(int32_t B, int32_t layer0, int32_t n_layers, int32_t Hq, int32_t Hkv,
                        int32_t d, int32_t dtype, int32_t T, int32_t W, int32_t keep,
                        int32_t local_keep, float sm_scale, int32_t causal, int32_t share_period,
                        int32_t share_start, const void* q_win, const void* k, const void* v,
                        int32_t* kept, void* k_out, void* v_out, double* token_score);
int mpcref_build_clusters(int32_t B, int32_t layer0, int32_t n_layers, int32_t Hkv, int32_t d,
                          int32_t dtype, int32_t Ts, int32_t cluster, int32_t fanout, float alpha,
                          int32_t share_period, int32_t share_start, int32_t similarity,
                          const void* k_cache, float* cent /*[..][C][R][d]*/, float* scent);
int mpcref_select_clusters(int32_t B, int32_t layer0, int32_t n_layers, int32_t Hq, int32_t Hkv,
                           int32_t d, int32_t dtype, int32_t Ts, int32_t cluster, int32_t fanout,
                           int32_t k_super, int32_t k_clusters, int32_t share_period,
                           int32_t share_start, int32_t similarity, int32_t group, const void* q,
                           const float* cent, const float* scent, int32_t* sel, double* sel_score);
/* Decode-time growth: (Ts, n_tail) after one appended token (a full tail of `cluster` rows is
 * sealed into a cluster first). Our reading; the paper only states the concatenation. */
int mpcref_append_state(int32_t Ts, int32_t n_tail, int32_t cluster, int32_t* Ts_out,
                        int32_t* n_tail_out);
/* k_cache / v_cache hold Ts + n_tail rows per (layer, sequence, kv head): the clustered rows, then
 * the tail rows every head attends. */
int mpcref_sparse_decode_attn(int32_t B, int32_t n_layers, int32_t Hq, int32_t Hkv, int32_t d,
                              int32_t dtype, int32_t Ts, int32_t n_tail, int32_t cluster, const void* q,
                              const void* k_cache, const void* v_cache, const int32_t* sel,
                              int32_t sel_heads, int32_t k_clusters, float sm_scale, double* out,
                              double* lse);
int mpcref_dense_decode_attn(int32_t B, int32_t n_layers, int32_t Hq, int32_t Hkv, int32_t d,
                             int32_t dtype, int32_t Ts, const void* q, const void* k_cache,
                             const void* v_cache, float sm_scale, double* out, double* lse);
/* Commonality score of m + 1 adjacent layers' top-k index sets (Sec. 3, Observation 3), per unit:
 * idx [L][units][k] -> out [units]. */
int mpcref_commonality(int32_t L, int32_t units, int32_t k, int32_t m, const int32_t* idx, double* out);
int mpcref_threads(void);
/* Threads the OpenMP loops use from now on (n >= 1); for timing on a chosen number of cores. */
void mpcref_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
