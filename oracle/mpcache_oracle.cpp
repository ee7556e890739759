// CPU oracle for the MPCache decode/prefill hot path. TEST INFRASTRUCTURE ONLY: it is loaded by
// the tests, the smoke check and the benchmark's CPU-baseline leg, never by the product path.
//
// Plain fp64 loops in the paper's order and notation; std::sort / std::exp / std::log are the
// only library steps. Nothing here is blocked, fused or reordered for speed.
//
// Parity status of each function (what pins it is in tests/test_oracle_pins.py):
//   mpcref_token_scores    pinned (row sums, closed forms for uniform keys, brute force vs torch)
//   mpcref_static_topk     pinned (full-sort ranking vs numpy lexsort, ties, identity budget)
//   mpcref_cluster_bounds  pinned (numpy max/min, member bounds = token bounds)
//   mpcref_centroid        pinned (alpha = 1 / 0 give the bounds, fp32 rounding by numpy float32)
//   mpcref_cluster_scores  pinned (Eq. 2 ordering: linear score <= MP bound >= max dot product;
//                          single-token clusters give the dot product in every mode; with a
//                          non-negative query the bound equals the alpha = 1 linear score)
//   mpcref_cluster_mean    pinned (numpy mean in fp64)
//   mpcref_topk            pinned (numpy lexsort)
//   mpcref_attend          pinned (torch scaled_dot_product_attention, fp64)
//   grouped heads          pinned (max / sum of per-head numpy scores; per-head and max-rule
//                          selections against independent numpy ranking; one-head groups select
//                          alike in every rule; per-head lists against torch attention)
//   mpcref_commonality     pinned (worked cases, python set intersections, exact fractions)
//   the rule functions     pinned by the integers stated for the five workloads
// The readings of silent passages (GQA aggregation, causal mask and 1/sqrt(d) in static scoring,
// a recent-token window, integer rounding of budgets, fp32 storage of centroids) are conventions
// applied identically on both sides; the paper itself does not pin them.
#include "mpcache_oracle.h"

#include <omp.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <numeric>
#include <vector>

namespace {

enum { OK = 0, EINVAL = 1, ESHAPE = 2, EUNSUPPORTED = 3 };

// Exact conversion of one stored element to double.
double load(const void* base, size_t i, int dtype) {
  if (dtype == 0) return (double)((const float*)base)[i];
  const uint16_t h = ((const uint16_t*)base)[i];
  if (dtype == 2) {
    uint32_t bits = (uint32_t)h << 16;
    float f;
    std::memcpy(&f, &bits, 4);
    return (double)f;
  }
  const int e = (h >> 10) & 0x1F, m = h & 0x3FF;
  double v;
  if (e == 0)
    v = std::ldexp((double)m, -24);
  else if (e == 31)
    v = m ? NAN : INFINITY;
  else
    v = std::ldexp((double)(1024 + m), e - 25);
  return (h & 0x8000) ? -v : v;
}

size_t elt_size(int dtype) { return dtype == 0 ? 4 : 2; }

bool valid_dtype(int dtype) { return dtype >= 0 && dtype <= 2; }

// Ranking used by every top-k of the method: larger score first, lower index on ties.
std::vector<int32_t> rank_desc(const double* score, int32_t n) {
  std::vector<int32_t> idx(n);
  std::iota(idx.begin(), idx.end(), 0);
  std::sort(idx.begin(), idx.end(), [&](int32_t a, int32_t b) {
    if (score[a] != score[b]) return score[a] > score[b];
    return a < b;
  });
  return idx;
}

int32_t ceil_div(int32_t a, int32_t b) { return (a + b - 1) / b; }

}  // namespace

// ------------------------------------------------------------------------------------ rules

// Static eviction scores only the last 20% of the prompt's queries, and 10% once the prompt is
// longer than 24k tokens (Sec. 3.2; App. F, static-eviction setting). Reading: 24k = 24 * 1024 tokens,
// the row count is rounded down, and at least one row is used.
int32_t mpcref_window_rows(int32_t T) {
  if (T <= 0) return 0;
  const int64_t w = T > 24 * 1024 ? (int64_t)T / 10 : (int64_t)T * 2 / 10;
  return (int32_t)std::max<int64_t>(1, w);
}

// Cross-layer index sharing (Sec. 3.4): adjacent layers reuse one selection, except the first
// two layers, which always select for themselves. With period P and start s0 the owner of layer
// l >= s0 is the first layer of its block of P. (Alg. 3 writes the pairing as l % 2, which would
// also pair layers 0 and 1; Sec. 3.4 excludes them, and start = 0 reproduces the algorithm.)
int32_t mpcref_owner_layer(int32_t layer, int32_t period, int32_t start) {
  if (period <= 1 || layer < start) return layer;
  return start + period * ((layer - start) / period);
}

// Tokens kept by static eviction: ratio * T, rounded down to whole clusters (reading; the paper
// states only the ratio), and at least one cluster.
int32_t mpcref_keep_tokens(int32_t T, double static_ratio, int32_t cluster) {
  if (T <= 0 || cluster <= 0) return 0;
  const int32_t n = (int32_t)std::floor(static_ratio * T / cluster + 1e-9);
  return std::min(T, std::max(cluster, n * cluster));
}

// Level-1 budget of the two-level hierarchy (App. F): when the final selection ratio is below
// 0.5, half of the coarse clusters are dropped at level 1 (the text writes the ratio as "alpha",
// a clash with the similarity weight; read as the dynamic ratio). Half is rounded up.
int32_t mpcref_level1_keep(int32_t n_super, double final_ratio) {
  if (n_super <= 0) return 0;
  return final_ratio < 0.5 ? ceil_div(n_super, 2) : n_super;
}

// Level-2 budget in clusters: Alg. 3 takes topk with k = |K| * eta over the (post-eviction)
// cache while ranking clusters, so the token budget eta * T_s is converted to clusters of size s,
// rounded down, at least one, and at most the number of candidates.
int32_t mpcref_level2_keep(int32_t keep, double dynamic_ratio, int32_t cluster, int32_t n_cand) {
  if (keep <= 0 || cluster <= 0 || n_cand <= 0) return 0;
  const int32_t n = (int32_t)std::floor(dynamic_ratio * keep / cluster + 1e-9);
  return std::min(n_cand, std::max(1, n));
}

// The other reading of the same budget: the Fig. 9 caption calls the selection ratio the "final
// KV cache budget", i.e. a fraction of the prompt. Then eta * T tokens are selected, converted to
// clusters of size s the same way (rounded down, at least one, at most the candidates). With a
// static ratio r it selects 1 / r times as many clusters as the post-eviction reading (twice as
// many on the GPT-2 workload: 16 instead of 8).
int32_t mpcref_level2_keep_of_prompt(int32_t T, double dynamic_ratio, int32_t cluster, int32_t n_cand) {
  if (T <= 0 || cluster <= 0 || n_cand <= 0) return 0;
  const int32_t n = (int32_t)std::floor(dynamic_ratio * T / cluster + 1e-9);
  return std::min(n_cand, std::max(1, n));
}

// ------------------------------------------------------------------------------- per head

// Accumulated attention of the window queries (Sec. 3.2; Alg. 3 step 1): row t of the window is
// the query at position T-W+t; its attention over keys j is softmax_j(sm_scale * q_t . k_j)
// (the prefill attention of App. A.3, causal: j <= T-W+t); score[j] sums those probabilities over
// all window rows and over the G query heads that read this kv head (reading for grouped heads).
int mpcref_token_scores(int32_t G, int32_t d, int32_t T, int32_t W, int32_t dtype, float sm_scale,
                        int32_t causal, const void* q_win, const void* k, double* score,
                        double* row_lse) {
  if (G <= 0 || d <= 0 || T <= 0 || W <= 0 || W > T || !valid_dtype(dtype) || !q_win || !k ||
      !score)
    return EINVAL;
  for (int32_t j = 0; j < T; ++j) score[j] = 0.0;
  std::vector<double> s(T), q(d);
  for (int32_t g = 0; g < G; ++g) {
    for (int32_t t = 0; t < W; ++t) {
      for (int32_t i = 0; i < d; ++i) q[i] = load(q_win, ((size_t)g * W + t) * d + i, dtype);
      const int32_t n = causal ? T - W + t + 1 : T;
      double m = -INFINITY;
      for (int32_t j = 0; j < n; ++j) {
        double dot = 0.0;
        for (int32_t i = 0; i < d; ++i) dot += q[i] * load(k, (size_t)j * d + i, dtype);
        s[j] = (double)sm_scale * dot;
        m = std::max(m, s[j]);
      }
      double l = 0.0;
      for (int32_t j = 0; j < n; ++j) l += std::exp(s[j] - m);
      for (int32_t j = 0; j < n; ++j) score[j] += std::exp(s[j] - m) / l;
      if (row_lse) row_lse[(size_t)g * W + t] = m + std::log(l);
    }
  }
  return OK;
}

// Log-sum-exp of a single window row t (used to check one row of a large problem).
int mpcref_row_lse(int32_t d, int32_t T, int32_t W, int32_t dtype, float sm_scale, int32_t causal,
                   const void* q_row, int32_t t, const void* k, double* lse) {
  if (d <= 0 || T <= 0 || W <= 0 || W > T || t < 0 || t >= W || !valid_dtype(dtype) || !q_row ||
      !k || !lse)
    return EINVAL;
  const int32_t n = causal ? T - W + t + 1 : T;
  std::vector<double> s(n);
  double m = -INFINITY;
  for (int32_t j = 0; j < n; ++j) {
    double dot = 0.0;
    for (int32_t i = 0; i < d; ++i) dot += load(q_row, i, dtype) * load(k, (size_t)j * d + i, dtype);
    s[j] = (double)sm_scale * dot;
    m = std::max(m, s[j]);
  }
  double l = 0.0;
  for (int32_t j = 0; j < n; ++j) l += std::exp(s[j] - m);
  *lse = m + std::log(l);
  return OK;
}

// Look-once static eviction (Sec. 3.2; Alg. 3 step 1): rank tokens by accumulated attention and
// keep the highest. Reading: the most recent `local_keep` tokens are always kept (they cannot be
// judged by a window they belong to); the rest of the budget goes to the best-scored older tokens.
// Output is ascending original positions, so the kept cache preserves token order.
int mpcref_static_topk(int32_t T, const double* score, int32_t keep, int32_t local_keep,
                       int32_t* kept) {
  if (T <= 0 || keep <= 0 || keep > T || local_keep < 0 || !score || !kept) return EINVAL;
  const int32_t local = std::min(local_keep, keep);
  const int32_t n_old = T - local;
  const std::vector<int32_t> order = rank_desc(score, n_old);
  std::vector<int32_t> out(order.begin(), order.begin() + (keep - local));
  for (int32_t j = n_old; j < T; ++j) out.push_back(j);
  std::sort(out.begin(), out.end());
  std::copy(out.begin(), out.end(), kept);
  return OK;
}

// r^max_i and r^min_i of a cluster (Sec. 3.3, definition under Eq. 1): per-channel maximum and
// minimum of the keys of tokens [first, first + count) of the cache.
int mpcref_cluster_bounds(int32_t n_tok, int32_t d, int32_t dtype, const void* k, int32_t first,
                          int32_t count, double* rmax, double* rmin) {
  if (n_tok <= 0 || d <= 0 || first < 0 || count <= 0 || first >= n_tok || !valid_dtype(dtype) ||
      !k || !rmax || !rmin)
    return EINVAL;
  const int32_t last = std::min(n_tok, first + count);
  for (int32_t i = 0; i < d; ++i) {
    rmax[i] = -INFINITY;
    rmin[i] = INFINITY;
  }
  for (int32_t j = first; j < last; ++j)
    for (int32_t i = 0; i < d; ++i) {
      const double x = load(k, (size_t)j * d + i, dtype);
      rmax[i] = std::max(rmax[i], x);
      rmin[i] = std::min(rmin[i], x);
    }
  return OK;
}

// Average of a cluster's keys, the naive representative the paper compares against (Sec. 3.3
// opening; the appendix that compares it with the paper's similarity): the fp64 sum over the cluster's
// tokens in token order divided by their count. Reading: the score is the dot product with this
// average (like the other representatives), and it is stored rounded to fp32.
int mpcref_cluster_mean(int32_t n_tok, int32_t d, int32_t dtype, const void* k, int32_t first,
                        int32_t count, double* mean) {
  if (n_tok <= 0 || d <= 0 || first < 0 || count <= 0 || first >= n_tok || !valid_dtype(dtype) ||
      !k || !mean)
    return EINVAL;
  const int32_t last = std::min(n_tok, first + count);
  for (int32_t i = 0; i < d; ++i) mean[i] = 0.0;
  for (int32_t j = first; j < last; ++j)
    for (int32_t i = 0; i < d; ++i) mean[i] += load(k, (size_t)j * d + i, dtype);
  for (int32_t i = 0; i < d; ++i) mean[i] /= (double)(last - first);
  return OK;
}

// Reordered linear similarity (Sec. 3.3, Eq. "sim"): the cluster is represented by
// alpha * r^max + (1 - alpha) * r^min, precomputed once. Reading: it is stored in fp32, each
// product rounded to fp32 and then their sum rounded to fp32, with alpha given in fp32 and
// 1 - alpha rounded to fp32. Products of fp32 numbers and sums of two fp32 numbers are exact or
// correctly rounded when done in fp64 and rounded once, so this equals fp32 arithmetic.
float mpcref_centroid(double rmax, double rmin, float alpha) {
  const float a = alpha;
  const float b = (float)(1.0 - (double)a);
  const float pa = (float)((double)a * rmax);
  const float pb = (float)((double)b * rmin);
  return (float)((double)pa + (double)pb);
}

// Similarity of one query head with one cluster representative. Linear (Sec. 3.3, Eq. "sim") and
// average: sum_i q_i * c_i with the stored representative c. Max-product bound (Sec. 3.3, Eq. 2):
// sum_i max(q_i r^max_i, q_i r^min_i) over the stored bounds (rows r^max, r^min).
static double head_similarity(int32_t d, int32_t dtype, int32_t similarity, const void* q, const float* r) {
  double acc = 0.0;
  for (int32_t i = 0; i < d; ++i) {
    const double qi = load(q, i, dtype);
    if (similarity == 1)
      acc += std::max(qi * (double)r[i], qi * (double)r[d + i]);
    else
      acc += qi * (double)r[i];
  }
  return acc;
}

// Similarity of the G query heads of a kv head with each cluster representative. The paper states
// the similarity for one query. Readings for grouped heads (group): 0, the heads share one
// selection scored by the sum of their similarities (for the linear forms, the similarity of the
// summed query); 1, they share one selection scored by the largest of their similarities. `rep`
// holds n representatives of (similarity == 1 ? 2 : 1) rows of d floats.
int mpcref_cluster_scores(int32_t G, int32_t d, int32_t dtype, int32_t similarity, int32_t group, const void* q,
                          int32_t n, const float* rep, double* score) {
  if (G <= 0 || d <= 0 || n < 0 || !valid_dtype(dtype) || similarity < 0 || similarity > 2 || group < 0 ||
      group > 1 || !q || (n && (!rep || !score)))
    return EINVAL;
  const int32_t R = similarity == 1 ? 2 : 1;
  const size_t es = elt_size(dtype);
  for (int32_t c = 0; c < n; ++c) {
    const float* r = rep + (size_t)c * R * d;
    double acc = group == 0 ? 0.0 : -INFINITY;
    for (int32_t g = 0; g < G; ++g) {
      const double sg = head_similarity(d, dtype, similarity, (const char*)q + (size_t)g * d * es, r);
      acc = group == 0 ? acc + sg : std::max(acc, sg);
    }
    score[c] = acc;
  }
  return OK;
}

// Upper bound of the maximum dot product (Sec. 3.3, Eq. 2): sum_i max(q_i r^max_i, q_i r^min_i).
int mpcref_mp_bound(int32_t d, const double* q, const double* rmax, const double* rmin,
                    double* bound) {
  if (d <= 0 || !q || !rmax || !rmin || !bound) return EINVAL;
  double acc = 0.0;
  for (int32_t i = 0; i < d; ++i) acc += std::max(q[i] * rmax[i], q[i] * rmin[i]);
  *bound = acc;
  return OK;
}

// Top-k ranking (Alg. 1 step 2): the k best scores, larger first, lower index on ties.
int mpcref_topk(int32_t n, const double* score, int32_t k, int32_t* idx) {
  if (n < 0 || k < 0 || k > n || (n && !score) || (k && !idx)) return EINVAL;
  const std::vector<int32_t> order = rank_desc(score, n);
  std::copy(order.begin(), order.begin() + k, idx);
  return OK;
}

// Sparse attention over gathered rows (Alg. 1 steps 3-4; Alg. 3 step 2):
// o = softmax(sm_scale * q K'^T) V' with K', V' the rows listed in `rows`.
int mpcref_attend(int32_t d, int32_t dtype, float sm_scale, const void* q, int32_t n_tok,
                  const int32_t* rows, const void* k, const void* v, double* out, double* lse) {
  if (d <= 0 || n_tok <= 0 || !valid_dtype(dtype) || !q || !rows || !k || !v || !out) return EINVAL;
  std::vector<double> z(n_tok);
  double m = -INFINITY;
  for (int32_t j = 0; j < n_tok; ++j) {
    double dot = 0.0;
    for (int32_t i = 0; i < d; ++i)
      dot += load(q, i, dtype) * load(k, (size_t)rows[j] * d + i, dtype);
    z[j] = (double)sm_scale * dot;
    m = std::max(m, z[j]);
  }
  double l = 0.0;
  for (int32_t j = 0; j < n_tok; ++j) l += std::exp(z[j] - m);
  for (int32_t i = 0; i < d; ++i) out[i] = 0.0;
  for (int32_t j = 0; j < n_tok; ++j) {
    const double p = std::exp(z[j] - m) / l;
    for (int32_t i = 0; i < d; ++i) out[i] += p * load(v, (size_t)rows[j] * d + i, dtype);
  }
  if (lse) *lse = m + std::log(l);
  return OK;
}

// ------------------------------------------------------------------------- whole tensors

// Step 1 of Alg. 3 over a block of layers: owner layers score and rank their tokens; layers that
// share (Sec. 3.4) reuse the owner's kept set; every layer gathers its kept K/V rows. A layer whose
// owner precedes layer0 takes `kept` for that layer as input.
int mpcref_static_evict(int32_t B, int32_t layer0, int32_t n_layers, int32_t Hq, int32_t Hkv,
                        int32_t d, int32_t dtype, int32_t T, int32_t W, int32_t keep,
                        int32_t local_keep, float sm_scale, int32_t causal, int32_t share_period,
                        int32_t share_start, const void* q_win, const void* k, const void* v,
                        int32_t* kept, void* k_out, void* v_out, double* token_score) {
  if (B <= 0 || layer0 < 0 || n_layers <= 0 || Hq <= 0 || Hkv <= 0 || d <= 0 || T <= 0 ||
      !valid_dtype(dtype) || !q_win || !k || !v || !kept || !k_out || !v_out)
    return EINVAL;
  if (Hq % Hkv || W <= 0 || W > T || keep <= 0 || keep > T || local_keep < 0) return ESHAPE;
  const int32_t G = Hq / Hkv;
  const size_t es = elt_size(dtype);
  const size_t kv_head = (size_t)T * d, q_head = (size_t)W * d;
  const int64_t units = (int64_t)n_layers * B * Hkv;
  int rc = OK;
#pragma omp parallel for schedule(dynamic) reduction(max : rc)
  for (int64_t u = 0; u < units; ++u) {
    const int32_t l = (int32_t)(u / ((int64_t)B * Hkv));
    if (mpcref_owner_layer(layer0 + l, share_period, share_start) != layer0 + l) continue;
    const int32_t b = (int32_t)((u / Hkv) % B), h = (int32_t)(u % Hkv);
    std::vector<double> score(T);
    const char* qw = (const char*)q_win + (((size_t)l * B + b) * Hq + (size_t)h * G) * q_head * es;
    const char* kh = (const char*)k + (size_t)u * kv_head * es;
    int r = mpcref_token_scores(G, d, T, W, dtype, sm_scale, causal, qw, kh, score.data(), nullptr);
    if (!r) r = mpcref_static_topk(T, score.data(), keep, local_keep, kept + (size_t)u * keep);
    if (token_score) std::copy(score.begin(), score.end(), token_score + (size_t)u * T);
    rc = std::max(rc, r);
  }
  if (rc) return rc;
  for (int32_t l = 0; l < n_layers; ++l) {
    const int32_t o = mpcref_owner_layer(layer0 + l, share_period, share_start) - layer0;
    if (o == l || o < 0) continue;
    std::memcpy(kept + (size_t)l * B * Hkv * keep, kept + (size_t)o * B * Hkv * keep,
                (size_t)B * Hkv * keep * sizeof(int32_t));
  }
  for (int64_t u = 0; u < units; ++u) {
    const int32_t* kp = kept + (size_t)u * keep;
    for (int32_t i = 0; i < keep; ++i) {
      if (kp[i] < 0 || kp[i] >= T) return EINVAL;
      std::memcpy((char*)k_out + ((size_t)u * keep + i) * d * es,
                  (const char*)k + ((size_t)u * kv_head + (size_t)kp[i] * d) * es, d * es);
      std::memcpy((char*)v_out + ((size_t)u * keep + i) * d * es,
                  (const char*)v + ((size_t)u * kv_head + (size_t)kp[i] * d) * es, d * es);
    }
  }
  return OK;
}

// Cluster representatives (Sec. 3.3): fine clusters of `cluster` adjacent tokens of the kept
// cache and coarse clusters of `fanout` adjacent fine clusters (hierarchy, Sec. 3.3 and App. F),
// each summarised by the reordered representative. Coarse bounds are taken over their tokens.
// Only owner layers are written.
int mpcref_build_clusters(int32_t B, int32_t layer0, int32_t n_layers, int32_t Hkv, int32_t d,
                          int32_t dtype, int32_t Ts, int32_t cluster, int32_t fanout, float alpha,
                          int32_t share_period, int32_t share_start, int32_t similarity,
                          const void* k_cache, float* cent, float* scent) {
  if (B <= 0 || layer0 < 0 || n_layers <= 0 || Hkv <= 0 || d <= 0 || Ts <= 0 || cluster <= 0 ||
      fanout <= 0 || !valid_dtype(dtype) || similarity < 0 || similarity > 2 || !k_cache || !cent ||
      !scent)
    return EINVAL;
  const int32_t C = ceil_div(Ts, cluster), S = ceil_div(C, fanout);
  const int32_t R = similarity == 1 ? 2 : 1;
  const size_t es = elt_size(dtype);
  const int64_t units = (int64_t)n_layers * B * Hkv;
#pragma omp parallel for schedule(dynamic)
  for (int64_t u = 0; u < units; ++u) {
    const int32_t l = (int32_t)(u / ((int64_t)B * Hkv));
    if (mpcref_owner_layer(layer0 + l, share_period, share_start) != layer0 + l) continue;
    const char* kh = (const char*)k_cache + (size_t)u * Ts * d * es;
    std::vector<double> rmax(d), rmin(d);
    // one representative of the tokens [first, first + count) into `out` (R rows of d)
    auto represent = [&](int32_t first, int32_t count, float* out) {
      if (similarity == 2) {
        mpcref_cluster_mean(Ts, d, dtype, kh, first, count, rmax.data());
        for (int32_t i = 0; i < d; ++i) out[i] = (float)rmax[i];
        return;
      }
      mpcref_cluster_bounds(Ts, d, dtype, kh, first, count, rmax.data(), rmin.data());
      for (int32_t i = 0; i < d; ++i) {
        if (similarity == 1) {
          out[i] = (float)rmax[i];  // key elements: exact in fp32
          out[d + i] = (float)rmin[i];
        } else {
          out[i] = mpcref_centroid(rmax[i], rmin[i], alpha);
        }
      }
    };
    for (int32_t c = 0; c < C; ++c) represent(c * cluster, cluster, cent + ((size_t)u * C + c) * R * d);
    for (int32_t s2 = 0; s2 < S; ++s2)
      represent(s2 * fanout * cluster, fanout * cluster, scent + ((size_t)u * S + s2) * R * d);
  }
  return OK;
}

// Query-aware dynamic selection at one decode step (Sec. 3.3; Alg. 3 step 2): level 1 ranks the
// coarse clusters and keeps k_super; level 2 ranks the fine clusters inside the kept coarse ones
// and keeps k_clusters, written in ascending order. Non-owner layers copy their owner's selection
// (Sec. 3.4); a layer whose owner precedes layer0 keeps the `sel` the caller passed in.
// group: 0 / 1, one selection per kv head scored by the sum / the maximum of its query heads'
// similarities (sel [n_layers][B][Hkv][k_clusters]); 2, one selection per query head from its own
// similarity against its kv head's representatives (sel [n_layers][B][Hq][k_clusters]). The paper
// states the selection for one query head; the grouped forms are readings.
int mpcref_select_clusters(int32_t B, int32_t layer0, int32_t n_layers, int32_t Hq, int32_t Hkv,
                           int32_t d, int32_t dtype, int32_t Ts, int32_t cluster, int32_t fanout,
                           int32_t k_super, int32_t k_clusters, int32_t share_period,
                           int32_t share_start, int32_t similarity, int32_t group, const void* q,
                           const float* cent, const float* scent, int32_t* sel, double* sel_score) {
  if (B <= 0 || layer0 < 0 || n_layers <= 0 || Hq <= 0 || Hkv <= 0 || d <= 0 || Ts <= 0 ||
      cluster <= 0 || fanout <= 0 || !valid_dtype(dtype) || similarity < 0 || similarity > 2 || group < 0 ||
      group > 2 || !q || !cent || !scent || !sel)
    return EINVAL;
  const int32_t R = similarity == 1 ? 2 : 1;
  const int32_t C = ceil_div(Ts, cluster), S = ceil_div(C, fanout);
  if (Hq % Hkv || k_super <= 0 || k_super > S || k_clusters <= 0) return ESHAPE;
  const int32_t tail = C - (S - 1) * fanout;
  if (k_clusters > k_super * fanout - (fanout - tail)) return ESHAPE;
  const int32_t G = Hq / Hkv;
  const size_t es = elt_size(dtype);
  // selection heads per (layer, sequence); query heads scored together; the kv head of head h
  const int32_t H = group == 2 ? Hq : Hkv, Gs = group == 2 ? 1 : G, rdiv = group == 2 ? G : 1;
  const int64_t units = (int64_t)n_layers * B * H;
#pragma omp parallel for schedule(dynamic)
  for (int64_t u = 0; u < units; ++u) {
    const int32_t l = (int32_t)(u / ((int64_t)B * H));
    if (mpcref_owner_layer(layer0 + l, share_period, share_start) != layer0 + l) continue;
    const int32_t b = (int32_t)((u / H) % B), h = (int32_t)(u % H);
    const char* qg = (const char*)q + (((size_t)l * B + b) * Hq + (size_t)h * Gs) * d * es;
    const size_t ru = ((size_t)l * B + b) * Hkv + h / rdiv;  // representatives of this kv head
    std::vector<double> s1(S);
    mpcref_cluster_scores(Gs, d, dtype, similarity, group == 1, qg, S, scent + ru * S * R * d, s1.data());
    std::vector<int32_t> top1(k_super);
    mpcref_topk(S, s1.data(), k_super, top1.data());
    std::sort(top1.begin(), top1.end());
    std::vector<int32_t> cand;
    for (int32_t s : top1)
      for (int32_t c = s * fanout; c < std::min(C, (s + 1) * fanout); ++c) cand.push_back(c);
    const int32_t n = (int32_t)cand.size();
    std::vector<double> s2(n);
    for (int32_t j = 0; j < n; ++j)
      mpcref_cluster_scores(Gs, d, dtype, similarity, group == 1, qg, 1, cent + (ru * C + cand[j]) * R * d, &s2[j]);
    std::vector<int32_t> top2(k_clusters);
    mpcref_topk(n, s2.data(), k_clusters, top2.data());
    std::sort(top2.begin(), top2.end());  // positions in the ascending candidate list
    for (int32_t j = 0; j < k_clusters; ++j) {
      sel[(size_t)u * k_clusters + j] = cand[top2[j]];
      if (sel_score) sel_score[(size_t)u * k_clusters + j] = s2[top2[j]];
    }
  }
  for (int32_t l = 0; l < n_layers; ++l) {
    const int32_t o = mpcref_owner_layer(layer0 + l, share_period, share_start) - layer0;
    if (o == l || o < 0) continue;
    const size_t n = (size_t)B * H * k_clusters;
    std::memcpy(sel + (size_t)l * n, sel + (size_t)o * n, n * sizeof(int32_t));
    if (sel_score) std::memcpy(sel_score + (size_t)l * n, sel_score + (size_t)o * n, n * sizeof(double));
  }
  return OK;
}

// Decode-time cache growth (App. A.3): every decoded token's k, v are concatenated to the cache.
// The paper does not say how new tokens join clusters. Reading: they collect in an unclustered
// tail that is always attended; when a token arrives and the tail already holds s tokens, those s
// become the next cluster (Ts grows by s) before the new token starts the tail again.
int mpcref_append_state(int32_t Ts, int32_t n_tail, int32_t cluster, int32_t* Ts_out, int32_t* n_tail_out) {
  if (Ts < 0 || cluster <= 0 || n_tail < 0 || n_tail > cluster || !Ts_out || !n_tail_out) return EINVAL;
  if (n_tail == cluster) {
    Ts += cluster;
    n_tail = 0;
  }
  *Ts_out = Ts;
  *n_tail_out = n_tail + 1;
  return OK;
}

// Sparse attention of every query head over the tokens of its selected clusters, then the n_tail
// decode-time tokens that follow the clustered ones (k_cache holds Ts + n_tail rows per head).
// sel_heads = Hkv: one list per kv head, shared by its query heads; sel_heads = Hq: one list per
// query head, over its kv head's rows.
int mpcref_sparse_decode_attn(int32_t B, int32_t n_layers, int32_t Hq, int32_t Hkv, int32_t d,
                              int32_t dtype, int32_t Ts, int32_t n_tail, int32_t cluster, const void* q,
                              const void* k_cache, const void* v_cache, const int32_t* sel, int32_t sel_heads,
                              int32_t k_clusters, float sm_scale, double* out, double* lse) {
  if (B <= 0 || n_layers <= 0 || Hq <= 0 || Hkv <= 0 || d <= 0 || Ts <= 0 || n_tail < 0 || cluster <= 0 ||
      k_clusters <= 0 || !valid_dtype(dtype) || !q || !k_cache || !v_cache || !sel || !out)
    return EINVAL;
  if (Hq % Hkv || (sel_heads != Hkv && sel_heads != Hq)) return ESHAPE;
  const int32_t G = Hq / Hkv, C = ceil_div(Ts, cluster);
  const int32_t rows_per_head = Ts + n_tail;
  const size_t es = elt_size(dtype);
  const int64_t units = (int64_t)n_layers * B * Hq;
  int rc = OK;
#pragma omp parallel for schedule(dynamic) reduction(max : rc)
  for (int64_t u = 0; u < units; ++u) {
    const int64_t lb = u / Hq;
    const int32_t h = (int32_t)(u % Hq);
    const int64_t kvu = lb * Hkv + h / G;
    const int64_t su = sel_heads == Hq ? u : kvu;  // the head's selection list
    std::vector<int32_t> rows;
    for (int32_t j = 0; j < k_clusters; ++j) {
      const int32_t c = sel[su * k_clusters + j];
      if (c < 0 || c >= C) {
        rc = EINVAL;
        rows.clear();
        break;
      }
      for (int32_t t = c * cluster; t < std::min(Ts, (c + 1) * cluster); ++t) rows.push_back(t);
    }
    if (rows.empty()) continue;
    // the tokens appended while decoding (App. A.3), not yet in any cluster: always attended
    for (int32_t t = Ts; t < Ts + n_tail; ++t) rows.push_back(t);
    const size_t head = (size_t)kvu * rows_per_head * d * es;
    mpcref_attend(d, dtype, sm_scale, (const char*)q + (size_t)u * d * es, (int32_t)rows.size(),
                  rows.data(), (const char*)k_cache + head, (const char*)v_cache + head,
                  out + (size_t)u * d, lse ? lse + u : nullptr);
  }
  return rc;
}

// Full decode attention over the whole cache (App. A.3, decode-stage attention): the reference
// the sparse path must reproduce when every cluster is selected.
int mpcref_dense_decode_attn(int32_t B, int32_t n_layers, int32_t Hq, int32_t Hkv, int32_t d,
                             int32_t dtype, int32_t Ts, const void* q, const void* k_cache,
                             const void* v_cache, float sm_scale, double* out, double* lse) {
  if (B <= 0 || n_layers <= 0 || Hq <= 0 || Hkv <= 0 || d <= 0 || Ts <= 0 || !valid_dtype(dtype) ||
      !q || !k_cache || !v_cache || !out)
    return EINVAL;
  if (Hq % Hkv) return ESHAPE;
  const int32_t G = Hq / Hkv;
  const size_t es = elt_size(dtype);
  std::vector<int32_t> rows(Ts);
  std::iota(rows.begin(), rows.end(), 0);
  const int64_t units = (int64_t)n_layers * B * Hq;
#pragma omp parallel for schedule(dynamic)
  for (int64_t u = 0; u < units; ++u) {
    const int64_t kvu = (u / Hq) * Hkv + (u % Hq) / G;
    const size_t head = (size_t)kvu * Ts * d * es;
    mpcref_attend(d, dtype, sm_scale, (const char*)q + (size_t)u * d * es, Ts, rows.data(),
                  (const char*)k_cache + head, (const char*)v_cache + head, out + (size_t)u * d,
                  lse ? lse + u : nullptr);
  }
  return OK;
}

// Commonality score of m + 1 adjacent layers (Sec. 3, Observation 3):
// (1 / (k (L - m))) * sum_{l=0}^{L-m-1} |intersection of idx_i[:k] for i = l .. l+m|, for every
// (sequence, head) unit. idx [L][units][k] holds each layer's top-k index set (any order, distinct
// entries). The paper's sum runs over l = 1 .. L - m with the sets of layers l .. l + m; with
// layers counted from 0 that is l = 0 .. L - m - 1.
int mpcref_commonality(int32_t L, int32_t units, int32_t k, int32_t m, const int32_t* idx, double* out) {
  if (L <= 0 || units <= 0 || k <= 0 || m < 0 || m >= L || !idx || !out) return EINVAL;
  for (int32_t u = 0; u < units; ++u) {
    int64_t total = 0;
    for (int32_t l = 0; l + m < L; ++l) {
      const int32_t* a = idx + ((size_t)l * units + u) * k;
      for (int32_t j = 0; j < k; ++j) {
        bool in_all = true;
        for (int32_t i = l + 1; i <= l + m && in_all; ++i) {
          const int32_t* b = idx + ((size_t)i * units + u) * k;
          in_all = std::find(b, b + k, a[j]) != b + k;
        }
        total += in_all;
      }
    }
    out[u] = (double)total / ((double)k * (double)(L - m));
  }
  return OK;
}

int mpcref_threads(void) { return omp_get_max_threads(); }
void mpcref_set_threads(int n) {
  if (n >= 1) omp_set_num_threads(n);
}
