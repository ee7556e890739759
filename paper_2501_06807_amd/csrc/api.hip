// C ABI of the MPCache hot path: argument validation, workspace layout, kernel dispatch.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <mutex>

#include "append.h"
#include "clusters.h"
#include "commonality.h"
#include "common.h"
#include "decode_attn.h"
#include "evict.h"
#include "fused.h"
#include "select.h"

namespace {

thread_local char g_err[512] = "";

mpc_status fail(mpc_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

mpc_status ok() {
  g_err[0] = '\0';
  return MPC_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

int elt_size(int dtype) { return dtype == MPC_FP32 ? 4 : 2; }

int ceil_div(int a, int b) { return (a + b - 1) / b; }

mpc_status check_dims(const mpc_dims* d) {
  if (!d) return fail(MPC_EINVAL, "dims is NULL");
  if (d->batch <= 0 || d->n_layers <= 0 || d->layer0 < 0 || d->n_q_heads <= 0 ||
      d->n_kv_heads <= 0 || d->head_dim <= 0)
    return fail(MPC_EINVAL, "dims must be positive (layer0 >= 0)");
  if (d->dtype < MPC_FP32 || d->dtype > MPC_BF16) return fail(MPC_EINVAL, "bad dtype %d", d->dtype);
  if (d->n_q_heads % d->n_kv_heads)
    return fail(MPC_ESHAPE, "n_q_heads %d not a multiple of n_kv_heads %d", d->n_q_heads, d->n_kv_heads);
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(MPC_EUNSUPPORTED, "head_dim %d not in {64, 128}", d->head_dim);
  if ((int64_t)d->n_layers * d->batch * d->n_q_heads > (1 << 24))
    return fail(MPC_EUNSUPPORTED, "too many (layer, sequence, head) units");
  if (d->kv_capacity < 0) return fail(MPC_EINVAL, "kv_capacity must be >= 0");
  return MPC_OK;
}

// Allocated kept-cache rows per (layer, sequence, kv head): dims->kv_capacity, or the rows the call
// uses when it is 0. Fails when the capacity is smaller than those rows.
mpc_status cache_rows(const mpc_dims* d, int64_t used, int* rows) {
  const int64_t cap = d->kv_capacity ? d->kv_capacity : used;
  if (cap < used)
    return fail(MPC_ESHAPE, "kv_capacity %d below the %lld rows in use", d->kv_capacity, (long long)used);
  if (cap * d->head_dim * elt_size(d->dtype) > ((int64_t)1 << 31))
    return fail(MPC_EUNSUPPORTED, "a (layer, sequence, kv head) K/V block above 2 GiB");
  *rows = (int)cap;
  return MPC_OK;
}

// Launch errors are read with hipGetLastError(); an error left by an unrelated earlier runtime call
// on this thread is cleared first so that it is not reported as ours.
void clear_stale_error() { (void)hipGetLastError(); }

mpc_status launched(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(MPC_EHIP, "%s launch failed: %s", what, hipGetErrorString(e));
  return MPC_OK;
}

// Static eviction workspace: the (exponent offset, 1 / sum) pair of every window row, then fp32
// token scores.
struct EvictWs {
  size_t rowstat, score, total;
};
EvictWs evict_ws(const mpc_dims* d, int T, int W) {
  EvictWs w;
  w.rowstat = 0;
  w.score = align256((size_t)d->n_layers * d->batch * d->n_q_heads * W * sizeof(double));
  w.total = w.score + align256((size_t)d->n_layers * d->batch * d->n_kv_heads * T * sizeof(float));
  return w;
}

// Decode workspace: split-K partials, sized for the largest split count any token budget gives,
// then one arrival counter per unit (zero between launches). The attention's work units are the
// selection lists: one per kv head, or one per q-head (then each unit serves one q-head).
struct DecodeWs {
  size_t cnt, total;
};
DecodeWs decode_ws(const mpc_dims* d, bool per_q_head) {
  const int heads = per_q_head ? d->n_q_heads : d->n_kv_heads;
  const int units = d->n_layers * d->batch * heads;
  const int G = d->n_q_heads / heads;
  const mpc::DecodePlan p = mpc::decode_plan(units, 1 << 30, d->head_dim, elt_size(d->dtype));
  DecodeWs w{0, 0};
  if (p.splits <= 1) return w;
  w.cnt = align256((size_t)units * p.splits * G * (d->head_dim + 2) * sizeof(float));
  w.total = w.cnt + align256((size_t)units * sizeof(int));
  return w;
}
// enough for either layout, so that one size serves every selection rule
size_t decode_ws_bytes(const mpc_dims* d) { return std::max(decode_ws(d, false).total, decode_ws(d, true).total); }

// Fused decode-step workspace: the error word, per-owner-head state and consumer counts, then the
// split-K partials used when the block is too small for the fused kernel.
struct StepWs {
  size_t state, cons, part, total;
};
StepWs step_ws(const mpc_dims* d, const mpc_select_cfg* cfg) {
  StepWs w;
  const mpc::OwnerTable own = mpc::owner_table(d->layer0, d->n_layers, cfg->share_period, cfg->share_start);
  const size_t heads = align256((size_t)own.n * d->batch * d->n_kv_heads * sizeof(int));
  w.state = align256(sizeof(mpc::FusedSync));
  w.cons = w.state + heads;
  w.part = w.cons + heads;
  w.total = w.part + decode_ws_bytes(d);
  return w;
}

}  // namespace

extern "C" {

const char* mpc_status_string(mpc_status s) {
  switch (s) {
    case MPC_OK: return "ok";
    case MPC_EINVAL: return "invalid argument";
    case MPC_ESHAPE: return "inconsistent shape";
    case MPC_EUNSUPPORTED: return "unsupported configuration";
    case MPC_EWORKSPACE: return "workspace too small";
    case MPC_EHIP: return "HIP error";
  }
  return "unknown status";
}

const char* mpc_last_error(void) { return g_err; }

int32_t mpc_owner_layer(int32_t l, int32_t period, int32_t start) {
  return mpc::owner_layer(l, period, start);
}

size_t mpc_workspace_bytes(int32_t op, const mpc_dims* dims, int32_t T_or_Ts, const void* cfg) {
  if (check_dims(dims) != MPC_OK || T_or_Ts <= 0) return 0;
  if (op == MPC_OP_STATIC_EVICT) {
    const mpc_evict_cfg* c = (const mpc_evict_cfg*)cfg;
    if (!c || c->window <= 0 || c->window > T_or_Ts) return 0;
    return evict_ws(dims, T_or_Ts, c->window).total;
  }
  if (op == MPC_OP_DECODE_ATTN) return decode_ws_bytes(dims);
  if (op == MPC_OP_DECODE_STEP) {
    if (!cfg) return 0;
    return step_ws(dims, (const mpc_select_cfg*)cfg).total;
  }
  return 0;
}

}  // extern "C"

namespace {

mpc_status prepare_evict(const mpc_dims* dims, int32_t T, const mpc_evict_cfg* cfg, const void* q_win,
                         const void* k, const void* v, int32_t* kept_idx, void* k_out, void* v_out,
                         float* token_score, float* row_lse, void* ws, size_t ws_bytes, mpc::EvictArgs* out) {
  mpc_status s = check_dims(dims);
  if (s != MPC_OK) return s;
  if (!cfg) return fail(MPC_EINVAL, "cfg is NULL");
  if (T <= 0) return fail(MPC_EINVAL, "T must be positive");
  if (!q_win || !k || !v || !kept_idx || !k_out || !v_out)
    return fail(MPC_EINVAL, "a required tensor pointer is NULL");
  if (!aligned16(q_win) || !aligned16(k) || !aligned16(v) || !aligned16(k_out) || !aligned16(v_out))
    return fail(MPC_EINVAL, "tensor bases must be 16-byte aligned");
  if (cfg->window <= 0 || cfg->window > T) return fail(MPC_ESHAPE, "window %d not in [1, T]", cfg->window);
  if (cfg->keep <= 0 || cfg->keep > T) return fail(MPC_ESHAPE, "keep %d not in [1, T]", cfg->keep);
  if (cfg->local_keep < 0) return fail(MPC_EINVAL, "local_keep must be >= 0");
  if (!(cfg->sm_scale >= 0.f) || !std::isfinite(cfg->sm_scale)) return fail(MPC_EINVAL, "bad sm_scale");
  if (cfg->causal != 0 && cfg->causal != 1) return fail(MPC_EINVAL, "causal must be 0 or 1");
  if ((int64_t)T * dims->head_dim * elt_size(dims->dtype) >= ((int64_t)1 << 31))
    return fail(MPC_EUNSUPPORTED, "T too large");
  if (dims->n_layers > mpc::kMaxLayers)
    return fail(MPC_EUNSUPPORTED, "static eviction takes at most %d layers per call", mpc::kMaxLayers);
  if ((int64_t)dims->n_layers * dims->batch * dims->n_q_heads * ((cfg->window + mpc::kRowBlock - 1) / mpc::kRowBlock) >=
          ((int64_t)1 << 31) ||
      (int64_t)dims->n_layers * dims->batch * dims->n_kv_heads * ((T + mpc::kColBlockKeys - 1) / mpc::kColBlockKeys) >=
          ((int64_t)1 << 31))
    return fail(MPC_EUNSUPPORTED, "grid too large");
  int out_rows = 0;
  if ((s = cache_rows(dims, cfg->keep, &out_rows)) != MPC_OK) return s;
  const EvictWs lay = evict_ws(dims, T, cfg->window);
  if (!ws || ws_bytes < lay.total)
    return fail(MPC_EWORKSPACE, "static eviction needs %zu workspace bytes", lay.total);

  mpc::EvictArgs a{};
  a.q_win = q_win;
  a.k = k;
  a.v = v;
  a.kept = kept_idx;
  a.k_out = k_out;
  a.v_out = v_out;
  a.rowstat = (float2*)((char*)ws + lay.rowstat);
  a.score = token_score ? token_score : (float*)((char*)ws + lay.score);
  a.row_lse = row_lse;
  a.B = dims->batch;
  a.layer0 = dims->layer0;
  a.n_layers = dims->n_layers;
  a.Hq = dims->n_q_heads;
  a.Hkv = dims->n_kv_heads;
  a.T = T;
  a.W = cfg->window;
  a.keep = cfg->keep;
  a.out_rows = out_rows;
  a.local_keep = cfg->local_keep;
  a.causal = cfg->causal;
  a.period = cfg->share_period;
  a.start = cfg->share_start;
  a.own = mpc::owner_table(dims->layer0, dims->n_layers, cfg->share_period, cfg->share_start);
  a.c32 = (float)((double)cfg->sm_scale * 1.4426950408889634);
  *out = a;
  return MPC_OK;
}

// Scoring passes and top-k for the owner layers, then the gather of every layer not in `skip`.
mpc_status launch_evict(const mpc::EvictArgs& a, int dt, int D, hipStream_t st) {
  mpc_status s;
  if (a.own.n > 0) {
    if ((s = launched(mpc::launch_rowstats(a, dt, D, st), "row statistics")) != MPC_OK) return s;
    if ((s = launched(mpc::launch_colsum(a, dt, D, st), "column sums")) != MPC_OK) return s;
    if ((s = launched(mpc::launch_topk(a, st), "top-k")) != MPC_OK) return s;
  }
  return launched(mpc::launch_gather(a, dt, D, st), "gather");
}

mpc_status prepare_build(const mpc_dims* dims, int32_t Ts, const mpc_select_cfg* cfg, const void* k_cache,
                         float* cent, float* scent, mpc::BuildArgs* out) {
  mpc_status s = check_dims(dims);
  if (s != MPC_OK) return s;
  if (!cfg) return fail(MPC_EINVAL, "cfg is NULL");
  if (Ts <= 0 || cfg->cluster_size <= 0 || cfg->fanout <= 0)
    return fail(MPC_EINVAL, "Ts, cluster_size and fanout must be positive");
  if (!(cfg->alpha >= 0.f && cfg->alpha <= 1.f)) return fail(MPC_EINVAL, "alpha must be in [0, 1]");
  if (cfg->similarity < MPC_SIM_LINEAR || cfg->similarity > MPC_SIM_MEAN)
    return fail(MPC_EINVAL, "unknown similarity %d", cfg->similarity);
  if (!k_cache || !cent || !scent) return fail(MPC_EINVAL, "a required tensor pointer is NULL");
  if (!aligned16(k_cache) || !aligned16(cent) || !aligned16(scent))
    return fail(MPC_EINVAL, "tensor bases must be 16-byte aligned");
  int rows = 0;
  if ((s = cache_rows(dims, Ts, &rows)) != MPC_OK) return s;
  mpc::BuildArgs a{};
  a.k = k_cache;
  a.cent = cent;
  a.scent = scent;
  a.B = dims->batch;
  a.layer0 = dims->layer0;
  a.n_layers = dims->n_layers;
  a.Hkv = dims->n_kv_heads;
  a.Ts = Ts;
  a.s = cfg->cluster_size;
  a.f = cfg->fanout;
  a.C = ceil_div(Ts, a.s);
  a.S = ceil_div(a.C, a.f);
  a.rows = rows;
  a.cs = ceil_div(rows, a.s);
  a.ss = ceil_div(a.cs, a.f);
  a.sup0 = 0;
  a.n_sup = a.S;
  a.period = cfg->share_period;
  a.start = cfg->share_start;
  a.alpha = cfg->alpha;
  a.beta = (float)(1.0 - (double)cfg->alpha);
  a.similarity = cfg->similarity;
  if (a.n_layers > mpc::kMaxLayers) return fail(MPC_EUNSUPPORTED, "at most %d layers per call", mpc::kMaxLayers);
  if ((int64_t)a.n_layers * a.B * a.Hkv * a.S >= ((int64_t)1 << 31))
    return fail(MPC_EUNSUPPORTED, "grid too large");
  a.own = mpc::owner_table(a.layer0, a.n_layers, a.period, a.start);
  *out = a;
  return MPC_OK;
}

}  // namespace

extern "C" {

mpc_status mpc_static_evict(const mpc_dims* dims, int32_t T, const mpc_evict_cfg* cfg,
                            const void* q_win, const void* k, const void* v, int32_t* kept_idx,
                            void* k_out, void* v_out, float* token_score, float* row_lse,
                            void* ws, size_t ws_bytes, void* stream) {
  mpc::EvictArgs a;
  mpc_status s = prepare_evict(dims, T, cfg, q_win, k, v, kept_idx, k_out, v_out, token_score, row_lse, ws,
                               ws_bytes, &a);
  if (s != MPC_OK) return s;
  clear_stale_error();
  if ((s = launch_evict(a, dims->dtype, dims->head_dim, (hipStream_t)stream)) != MPC_OK) return s;
  return ok();
}

mpc_status mpc_build_clusters(const mpc_dims* dims, int32_t Ts, const mpc_select_cfg* cfg,
                              const void* k_cache, float* cent, float* scent, void* stream) {
  mpc::BuildArgs a;
  mpc_status s = prepare_build(dims, Ts, cfg, k_cache, cent, scent, &a);
  if (s != MPC_OK) return s;
  if (a.own.n == 0) return ok();
  clear_stale_error();
  if ((s = launched(mpc::launch_build(a, dims->dtype, dims->head_dim, (hipStream_t)stream), "build")) != MPC_OK)
    return s;
  return ok();
}

mpc_status mpc_prefill(const mpc_dims* dims, int32_t T, const mpc_evict_cfg* ecfg, const mpc_select_cfg* scfg,
                       const void* q_win, const void* k, const void* v, int32_t* kept_idx, void* k_out,
                       void* v_out, float* cent, float* scent, float* token_score, float* row_lse, void* ws,
                       size_t ws_bytes, void* stream) {
  mpc::EvictArgs a;
  mpc_status s = prepare_evict(dims, T, ecfg, q_win, k, v, kept_idx, k_out, v_out, token_score, row_lse, ws,
                               ws_bytes, &a);
  if (s != MPC_OK) return s;
  mpc::BuildArgs b;
  if ((s = prepare_build(dims, ecfg->keep, scfg, k_out, cent, scent, &b)) != MPC_OK) return s;
  // the selection's owner layers gather their rows inside the build; the gather takes the rest
  for (int i = 0; i < b.own.n; ++i) a.skip[b.own.local(i) >> 6] |= 1ull << (b.own.local(i) & 63);
  b.g.kept = kept_idx;
  b.g.k_src = k;
  b.g.v_src = v;
  b.g.k_dst = k_out;
  b.g.v_dst = v_out;
  b.g.T = T;
  b.g.keep = ecfg->keep;
  b.g.period = ecfg->share_period;
  b.g.start = ecfg->share_start;
  hipStream_t st = (hipStream_t)stream;
  clear_stale_error();
  if ((s = launch_evict(a, dims->dtype, dims->head_dim, st)) != MPC_OK) return s;
  if (b.own.n > 0 && (s = launched(mpc::launch_build(b, dims->dtype, dims->head_dim, st), "build")) != MPC_OK)
    return s;
  return ok();
}

}  // extern "C"

namespace {

mpc_status prepare_select(const mpc_dims* dims, int32_t Ts, const mpc_select_cfg* cfg, const void* q,
                          const float* cent, const float* scent, int32_t* sel, float* sel_score,
                          mpc::SelectArgs* out) {
  mpc_status s = check_dims(dims);
  if (s != MPC_OK) return s;
  if (!cfg) return fail(MPC_EINVAL, "cfg is NULL");
  if (Ts <= 0 || cfg->cluster_size <= 0 || cfg->fanout <= 0 || cfg->k_super <= 0 || cfg->k_clusters <= 0)
    return fail(MPC_EINVAL, "Ts, cluster_size, fanout and budgets must be positive");
  if (!q || !cent || !scent || !sel) return fail(MPC_EINVAL, "a required tensor pointer is NULL");
  if (cfg->similarity < MPC_SIM_LINEAR || cfg->similarity > MPC_SIM_MEAN)
    return fail(MPC_EINVAL, "unknown similarity %d", cfg->similarity);
  if (cfg->group < MPC_GROUP_SUM || cfg->group > MPC_GROUP_HEAD) return fail(MPC_EINVAL, "unknown group rule %d", cfg->group);
  const int C = ceil_div(Ts, cfg->cluster_size), S = ceil_div(C, cfg->fanout);
  if (cfg->k_super > S) return fail(MPC_ESHAPE, "k_super %d > super-clusters %d", cfg->k_super, S);
  const int tail = C - (S - 1) * cfg->fanout;
  const int min_cand = cfg->k_super * cfg->fanout - (cfg->fanout - tail);
  if (cfg->k_clusters > min_cand)
    return fail(MPC_ESHAPE, "k_clusters %d exceeds the smallest candidate set %d", cfg->k_clusters, min_cand);
  if (S > mpc::kSelMaxSuper || (int64_t)cfg->k_super * cfg->fanout > mpc::kSelMaxCand)
    return fail(MPC_EUNSUPPORTED, "selection sizes beyond the kernel limits");
  const bool per_q_head = cfg->group == MPC_GROUP_HEAD;
  const int Hsel = per_q_head ? dims->n_q_heads : dims->n_kv_heads;
  if (dims->n_layers > mpc::kMaxLayers) return fail(MPC_EUNSUPPORTED, "at most %d layers per call", mpc::kMaxLayers);
  int rows = 0;
  if ((s = cache_rows(dims, Ts, &rows)) != MPC_OK) return s;
  mpc::SelectArgs a{};
  a.q = q;
  a.cent = cent;
  a.scent = scent;
  a.sel = sel;
  a.sel_score = sel_score;
  a.B = dims->batch;
  a.layer0 = dims->layer0;
  a.n_layers = dims->n_layers;
  a.Hq = dims->n_q_heads;
  a.Hkv = dims->n_kv_heads;
  a.Hsel = Hsel;
  a.rep_div = per_q_head ? dims->n_q_heads / dims->n_kv_heads : 1;
  a.C = C;
  a.S = S;
  a.cs = ceil_div(rows, cfg->cluster_size);
  a.ss = ceil_div(a.cs, cfg->fanout);
  a.f = cfg->fanout;
  a.NC = cfg->k_super * cfg->fanout;
  a.k_super = cfg->k_super;
  a.k_clusters = cfg->k_clusters;
  a.period = cfg->share_period;
  a.start = cfg->share_start;
  a.similarity = cfg->similarity;
  a.group = cfg->group;
  a.own = mpc::owner_table(a.layer0, a.n_layers, a.period, a.start);
  if (mpc::select_smem_bytes(dims->head_dim, S, a.NC, mpc::select_query_rows(a)) > mpc::kMaxLds)
    return fail(MPC_EUNSUPPORTED, "selection sizes need more LDS than a workgroup has");
  *out = a;
  return MPC_OK;
}

// Attention arguments; *units and *G receive the work units (selection lists) of the launch and the
// q-heads each serves.
mpc_status prepare_decode(const mpc_dims* dims, int32_t Ts, int32_t n_tail, int32_t cluster_size, const void* q,
                          const void* k_cache, const void* v_cache, const int32_t* sel, int32_t sel_heads,
                          int32_t k_clusters, float sm_scale, void* out, float* lse, mpc::DecodeArgs* da,
                          mpc::DecodePlan* plan, int* units_out, int* G_out) {
  mpc_status s = check_dims(dims);
  if (s != MPC_OK) return s;
  if (Ts <= 0 || cluster_size <= 0 || k_clusters <= 0)
    return fail(MPC_EINVAL, "Ts, cluster_size and k_clusters must be positive");
  if (!q || !k_cache || !v_cache || !sel || !out) return fail(MPC_EINVAL, "a required tensor pointer is NULL");
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache))
    return fail(MPC_EINVAL, "tensor bases must be 16-byte aligned");
  if (!std::isfinite(sm_scale)) return fail(MPC_EINVAL, "bad sm_scale");
  const int Gkv = dims->n_q_heads / dims->n_kv_heads;
  if (Gkv != 1 && Gkv != 2 && Gkv != 4 && Gkv != 8)
    return fail(MPC_EUNSUPPORTED, "group size %d not in {1,2,4,8}", Gkv);
  if (sel_heads != dims->n_kv_heads && sel_heads != dims->n_q_heads)
    return fail(MPC_ESHAPE, "sel_heads %d is neither n_kv_heads nor n_q_heads", sel_heads);
  const bool per_q_head = sel_heads != dims->n_kv_heads;
  const int G = per_q_head ? 1 : Gkv;  // q-heads per work unit
  const int C = ceil_div(Ts, cluster_size);
  if (k_clusters > C) return fail(MPC_ESHAPE, "k_clusters %d > clusters %d", k_clusters, C);
  if (n_tail < 0) return fail(MPC_EINVAL, "n_tail must be >= 0");
  if (n_tail > 0 && Ts % cluster_size)
    return fail(MPC_ESHAPE, "a tail needs Ts (%d) to be a multiple of the cluster size %d", Ts, cluster_size);
  int rows = 0;
  if ((s = cache_rows(dims, (int64_t)Ts + n_tail, &rows)) != MPC_OK) return s;
  const int n_list = k_clusters + ceil_div(n_tail, cluster_size);
  if (n_list > 1024) return fail(MPC_EUNSUPPORTED, "k_clusters plus tail clusters above 1024");
  if ((int64_t)n_list * cluster_size >= ((int64_t)1 << 30)) return fail(MPC_EUNSUPPORTED, "too many tokens");
  const int units = dims->n_layers * dims->batch * sel_heads;
  *plan = mpc::decode_plan(units, n_list * cluster_size, dims->head_dim, elt_size(dims->dtype));
  mpc::DecodeArgs a{};
  a.q = q;
  a.k = k_cache;
  a.v = v_cache;
  a.sel = sel;
  a.out = out;
  a.lse = lse;
  a.part = nullptr;
  a.cnt = nullptr;
  a.Ts = Ts;
  a.rows = rows;
  a.n_tail = n_tail;
  a.s = cluster_size;
  a.C = C;
  a.k_sel = k_clusters;
  a.Hq = dims->n_q_heads;
  a.Hkv = sel_heads;
  a.cache_heads = dims->n_kv_heads;
  a.cache_div = per_q_head ? Gkv : 1;
  a.splits = plan->splits;
  a.qscale = (float)((double)sm_scale * 1.4426950408889634);
  // K rows stay cacheable while they fit the memory-side cache together with what the next
  // selection reads: the fine-cluster representatives of the call's units (C rows of d floats each)
  const long long k_bytes = 1ll * units * n_list * cluster_size * dims->head_dim * elt_size(dims->dtype);
  const long long rep_bytes = 1ll * units * C * dims->head_dim * 4;
  a.stream_k = k_bytes + rep_bytes > mpc::kStreamKBytes;
  *da = a;
  *units_out = units;
  *G_out = G;
  return MPC_OK;
}

}  // namespace

extern "C" {

mpc_status mpc_select_clusters(const mpc_dims* dims, int32_t Ts, const mpc_select_cfg* cfg,
                               const void* q, const float* cent, const float* scent,
                               int32_t* sel, float* sel_score, void* ws, size_t ws_bytes,
                               void* stream) {
  (void)ws;
  (void)ws_bytes;
  mpc::SelectArgs a{};
  mpc_status s = prepare_select(dims, Ts, cfg, q, cent, scent, sel, sel_score, &a);
  if (s != MPC_OK) return s;
  if (a.own.n == 0) return ok();
  clear_stale_error();
  if ((s = launched(mpc::launch_select(a, dims->dtype, dims->head_dim, (hipStream_t)stream), "select")) != MPC_OK)
    return s;
  return ok();
}

mpc_status mpc_sparse_decode_attn(const mpc_dims* dims, int32_t Ts, int32_t n_tail, int32_t cluster_size,
                                  const void* q, const void* k_cache, const void* v_cache,
                                  const int32_t* sel, int32_t sel_heads, int32_t k_clusters, float sm_scale,
                                  void* out, float* lse, void* ws, size_t ws_bytes, void* stream) {
  mpc::DecodeArgs a{};
  mpc::DecodePlan plan{};
  int units = 0, G = 0;
  mpc_status s = prepare_decode(dims, Ts, n_tail, cluster_size, q, k_cache, v_cache, sel, sel_heads, k_clusters,
                                sm_scale, out, lse, &a, &plan, &units, &G);
  if (s != MPC_OK) return s;
  const size_t need = decode_ws_bytes(dims);
  if (plan.splits > 1 && (!ws || ws_bytes < need))
    return fail(MPC_EWORKSPACE, "sparse decode attention needs %zu workspace bytes", need);
  if (plan.splits > 1) {
    a.part = (float*)ws;
    a.cnt = (int*)((char*)ws + decode_ws(dims, G == 1 && sel_heads != dims->n_kv_heads).cnt);
  }
  clear_stale_error();
  if ((s = launched(mpc::launch_sparse_decode(a, dims->dtype, dims->head_dim, G, units, plan, (hipStream_t)stream),
                    "sparse decode attention")) != MPC_OK)
    return s;
  return ok();
}

mpc_status mpc_decode_step(const mpc_dims* dims, int32_t Ts, int32_t n_tail, const mpc_select_cfg* cfg,
                           const void* q, const float* cent, const float* scent,
                           const void* k_cache, const void* v_cache, float sm_scale, int32_t* sel,
                           float* sel_score, void* out, float* lse, void* ws, size_t ws_bytes,
                           void* stream) {
  mpc::SelectArgs sa{};
  mpc_status s = prepare_select(dims, Ts, cfg, q, cent, scent, sel, sel_score, &sa);
  if (s != MPC_OK) return s;
  mpc::DecodeArgs da{};
  mpc::DecodePlan plan{};
  int units = 0, G = 0;
  s = prepare_decode(dims, Ts, n_tail, cfg->cluster_size, q, k_cache, v_cache, sel, sa.Hsel, cfg->k_clusters,
                     sm_scale, out, lse, &da, &plan, &units, &G);
  if (s != MPC_OK) return s;
  const StepWs lay = step_ws(dims, cfg);
  if (!ws || ws_bytes < lay.total)
    return fail(MPC_EWORKSPACE, "decode step needs %zu workspace bytes", lay.total);
  const bool per_q_head = sa.Hsel != dims->n_kv_heads;
  hipStream_t st = (hipStream_t)stream;
  clear_stale_error();
  const mpc::FusedPlan fp = mpc::fused_plan(sa, dims->head_dim, plan.splits);
  if ((!fp.self && (per_q_head || plan.splits > 1)) || !mpc::fused_fits(fp, dims->head_dim, G)) {
    // two kernels in sequence
    da.part = (float*)((char*)ws + lay.part);
    da.cnt = (int*)((char*)ws + lay.part + decode_ws(dims, per_q_head).cnt);
    if (sa.own.n > 0 &&
        (s = launched(mpc::launch_select(sa, dims->dtype, dims->head_dim, st), "select")) != MPC_OK)
      return s;
    if ((s = launched(mpc::launch_sparse_decode(da, dims->dtype, dims->head_dim, G, units, plan, st),
                      "sparse decode attention")) != MPC_OK)
      return s;
    return ok();
  }
  mpc::FusedArgs f{};
  f.s = sa;
  f.d = da;
  f.sync = (mpc::FusedSync*)ws;
  f.state = (int*)((char*)ws + lay.state);
  f.cons = (int*)((char*)ws + lay.cons);
  if ((s = launched(mpc::launch_decode_step(f, fp, dims->dtype, dims->head_dim, G, st), "decode step")) != MPC_OK)
    return s;
  return ok();
}

mpc_status mpc_commonality(int32_t L, int32_t units, int32_t k, int32_t m, const int32_t* idx, double* out,
                           void* stream) {
  if (L <= 0 || units <= 0 || k <= 0 || m < 0) return fail(MPC_EINVAL, "L, units, k must be positive and m >= 0");
  if (m >= L) return fail(MPC_ESHAPE, "m %d must be below the layer count %d", m, L);
  if (k > mpc::kCommonMaxK) return fail(MPC_EUNSUPPORTED, "k %d above %d", k, mpc::kCommonMaxK);
  if ((int64_t)L * units * k >= ((int64_t)1 << 31)) return fail(MPC_EUNSUPPORTED, "index tensor too large");
  if (!idx || !out) return fail(MPC_EINVAL, "a required tensor pointer is NULL");
  clear_stale_error();
  mpc_status s = launched(mpc::launch_commonality(L, units, k, m, idx, out, (hipStream_t)stream), "commonality");
  if (s != MPC_OK) return s;
  return ok();
}

mpc_status mpc_append_kv(const mpc_dims* dims, int32_t Ts, int32_t n_tail, const mpc_select_cfg* cfg,
                         const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                         float* cent, float* scent, int32_t* Ts_out, int32_t* n_tail_out, void* stream) {
  mpc_status s = check_dims(dims);
  if (s != MPC_OK) return s;
  if (!cfg) return fail(MPC_EINVAL, "cfg is NULL");
  if (cfg->cluster_size <= 0 || cfg->fanout <= 0) return fail(MPC_EINVAL, "cluster_size and fanout must be positive");
  if (!(cfg->alpha >= 0.f && cfg->alpha <= 1.f)) return fail(MPC_EINVAL, "alpha must be in [0, 1]");
  if (cfg->similarity < MPC_SIM_LINEAR || cfg->similarity > MPC_SIM_MEAN)
    return fail(MPC_EINVAL, "unknown similarity %d", cfg->similarity);
  if (!k_new || !v_new || !k_cache || !v_cache || !cent || !scent)
    return fail(MPC_EINVAL, "a required tensor pointer is NULL");
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(cent) ||
      !aligned16(scent))
    return fail(MPC_EINVAL, "tensor bases must be 16-byte aligned");
  const int s_ = cfg->cluster_size;
  if (Ts < 0 || Ts % s_) return fail(MPC_ESHAPE, "Ts %d must be a non-negative multiple of the cluster size %d", Ts, s_);
  if (n_tail < 0 || n_tail > s_) return fail(MPC_ESHAPE, "n_tail %d not in [0, %d]", n_tail, s_);
  if (dims->kv_capacity <= 0) return fail(MPC_EINVAL, "kv_capacity must be set for a growing cache");
  if (dims->n_layers > mpc::kMaxLayers) return fail(MPC_EUNSUPPORTED, "at most %d layers per call", mpc::kMaxLayers);
  const bool seal = n_tail == s_;
  const int Ts_new = seal ? Ts + s_ : Ts;
  const int row = seal ? Ts_new : Ts + n_tail;  // row of the new token
  int rows = 0;
  if ((s = cache_rows(dims, (int64_t)row + 1, &rows)) != MPC_OK) return s;
  const int64_t units = (int64_t)dims->n_layers * dims->batch * dims->n_kv_heads;
  hipStream_t st = (hipStream_t)stream;
  clear_stale_error();
  if (seal) {
    // rebuild the new cluster and its super-cluster on owner layers (the other clusters of that
    // super-cluster are recomputed too, to the same values)
    mpc::BuildArgs a{};
    a.k = k_cache;
    a.cent = cent;
    a.scent = scent;
    a.B = dims->batch;
    a.layer0 = dims->layer0;
    a.n_layers = dims->n_layers;
    a.Hkv = dims->n_kv_heads;
    a.Ts = Ts_new;
    a.s = s_;
    a.f = cfg->fanout;
    a.C = Ts_new / s_;
    a.S = ceil_div(a.C, a.f);
    a.rows = rows;
    a.cs = ceil_div(rows, s_);
    a.ss = ceil_div(a.cs, a.f);
    a.sup0 = (a.C - 1) / a.f;
    a.n_sup = 1;
    a.period = cfg->share_period;
    a.start = cfg->share_start;
    a.alpha = cfg->alpha;
    a.beta = (float)(1.0 - (double)cfg->alpha);
    a.similarity = cfg->similarity;
    a.own = mpc::owner_table(a.layer0, a.n_layers, a.period, a.start);
    if (a.own.n > 0 && (s = launched(mpc::launch_build(a, dims->dtype, dims->head_dim, st), "seal")) != MPC_OK)
      return s;
  }
  mpc::AppendArgs ap{};
  ap.k_new = k_new;
  ap.v_new = v_new;
  ap.k = k_cache;
  ap.v = v_cache;
  ap.units = units;
  ap.rows = rows;
  ap.row = row;
  ap.row_bytes = dims->head_dim * elt_size(dims->dtype);
  if ((s = launched(mpc::launch_append_rows(ap, st), "append")) != MPC_OK) return s;
  if (Ts_out) *Ts_out = Ts_new;
  if (n_tail_out) *n_tail_out = seal ? 1 : n_tail + 1;
  return ok();
}

mpc_status mpc_decode_step_status(void* ws, size_t ws_bytes, int32_t clear, int32_t* flags) {
  if (!ws || !flags) return fail(MPC_EINVAL, "ws and flags must not be NULL");
  if (ws_bytes < sizeof(mpc::FusedSync)) return fail(MPC_EWORKSPACE, "workspace smaller than its error word");
  clear_stale_error();
  mpc::FusedSync sync{};
  if (hipMemcpy(&sync, ws, sizeof(sync), hipMemcpyDeviceToHost) != hipSuccess)
    return fail(MPC_EHIP, "reading the error word: %s", hipGetErrorString(hipGetLastError()));
  *flags = sync.error;
  if (clear && sync.error) {
    const mpc::FusedSync zero{};
    if (hipMemcpy(ws, &zero, sizeof(zero), hipMemcpyHostToDevice) != hipSuccess)
      return fail(MPC_EHIP, "clearing the error word: %s", hipGetErrorString(hipGetLastError()));
  }
  return ok();
}

}  // extern "C"

// ---------------------------------------------------------------------------------------------
// Static eviction without any allocation: the workspace is a file-scope device array. Its name is
// only a host-side stand-in in host code; the array's device address is looked up once per device
// (hipGetSymbolAddress, with that device current) and only that address is handed to kernels.
namespace {

constexpr size_t kScratchBytes = (size_t)32 << 20;
constexpr int kMaxDevices = 64;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// Device address of the scratch array on the device the stream belongs to (the current device for
// the null stream); looked up once per device, with that device current.
mpc_status scratch_address(hipStream_t stream, void** out) {
  int cur = 0, dev = 0;
  if (hipGetDevice(&cur) != hipSuccess) return fail(MPC_EHIP, "no current device: %s", hipGetErrorString(hipGetLastError()));
  dev = cur;
  if (stream && hipStreamGetDevice(stream, &dev) != hipSuccess)
    return fail(MPC_EHIP, "device of the stream: %s", hipGetErrorString(hipGetLastError()));
  if (dev < 0 || dev >= kMaxDevices) return fail(MPC_EUNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    if (dev != cur && hipSetDevice(dev) != hipSuccess)
      return fail(MPC_EHIP, "selecting device %d: %s", dev, hipGetErrorString(hipGetLastError()));
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur) (void)hipSetDevice(cur);
    if (e != hipSuccess || !p) return fail(MPC_EHIP, "scratch address of device %d: %s", dev, hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return MPC_OK;
}

}  // namespace

extern "C" {

size_t mpc_static_evict_noalloc_limit(void) { return kScratchBytes; }

mpc_status mpc_static_evict_noalloc(const mpc_dims* dims, int32_t T, const mpc_evict_cfg* cfg, const void* q_win,
                                    const void* k, const void* v, int32_t* kept_idx, void* k_out, void* v_out,
                                    float* token_score, float* row_lse, void* stream) {
  // every check of the eviction but the workspace's (which is all that is left when it reports
  // the missing workspace), then the scratch size
  mpc::EvictArgs unused{};
  mpc_status s = prepare_evict(dims, T, cfg, q_win, k, v, kept_idx, k_out, v_out, token_score, row_lse, nullptr, 0,
                               &unused);
  if (s != MPC_EWORKSPACE) return s;
  const size_t need = evict_ws(dims, T, cfg->window).total;
  if (need > kScratchBytes)
    return fail(MPC_EWORKSPACE, "static eviction of this block needs %zu scratch bytes, the static array holds %zu "
                "(call it on fewer layers or sequences)", need, kScratchBytes);
  void* ws = nullptr;
  if ((s = scratch_address((hipStream_t)stream, &ws)) != MPC_OK) return s;
  return mpc_static_evict(dims, T, cfg, q_win, k, v, kept_idx, k_out, v_out, token_score, row_lse, ws, kScratchBytes,
                          stream);
}

}  // extern "C"
