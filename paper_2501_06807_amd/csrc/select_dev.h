// Device code of the two-level cluster selection, shared by the standalone kernels and the fused
// decode-step kernel.
#pragma once
#include "select.h"

namespace mpc {
namespace dev {

template <bool COH>
__device__ __forceinline__ void store_sel(int32_t* p, int v) {
  if constexpr (COH)
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    *p = v;
}

// Row scores of the level GEMVs: scores[r] = sum_i qsum[i] * M[idx(r)][i], rows with idx < 0
// score -inf. Four lanes share a row: at load step c the quad reads 64 contiguous bytes (lane k of
// the quad takes floats c*16 + 4k .. +3), so 16 rows per pass are in flight per wave; the quad's
// fp64 partial sums meet through two DPP quad swaps. A tile is loaded first and reduced later, so
// that the first tile's loads can be issued before the query sum exists.
template <int D, int PASS>
struct RowTile {
  float4 x[PASS][D / 16];
  bool valid[PASS];
};

template <int D, int PASS, class RowOf>
__device__ __forceinline__ void tile_load_fn(const float* M, RowOf row_of, int n, int r0, RowTile<D, PASS>& t) {
  constexpr int ROWS = kWave / 4;
  const int lane = threadIdx.x % kWave, rq = lane >> 2, qk = lane & 3;
#pragma unroll
  for (int p = 0; p < PASS; ++p) {
    const int r = r0 + p * ROWS + rq;
    const int row = r < n ? row_of(r) : -1;
    t.valid[p] = row >= 0;
    const float* src = M + (size_t)(t.valid[p] ? row : 0) * D + qk * 4;
#pragma unroll
    for (int c = 0; c < D / 16; ++c) t.x[p][c] = *(const float4*)(src + c * 16);
  }
}

template <int D, int PASS>
__device__ __forceinline__ void tile_load(const float* M, const int* idx, int n, int r0, RowTile<D, PASS>& t) {
  tile_load_fn<D, PASS>(M, [idx](int r) { return idx ? idx[r] : r; }, n, r0, t);
}

__device__ __forceinline__ uint32_t key_hi(double x);
__device__ __forceinline__ unsigned long long rank_key(uint32_t img, int i);

// The lane's share of the summed query, held in registers for every row it reduces: floats
// c*16 + 4k .. +3 (k = lane % 4) of each 16-float step, in fp64.
template <int D>
struct QReg {
  double v[D / 16][4];
};

template <int D>
__device__ __forceinline__ void qreg_load(const double* qsum, QReg<D>& q) {
  const int qk = threadIdx.x & 3;
#pragma unroll
  for (int c = 0; c < D / 16; ++c) {
    const double2 a = *(const double2*)(qsum + c * 16 + qk * 4);
    const double2 b = *(const double2*)(qsum + c * 16 + qk * 4 + 2);
    q.v[c][0] = a.x;
    q.v[c][1] = a.y;
    q.v[c][2] = b.x;
    q.v[c][3] = b.y;
  }
}

// Writes the score of row r (quad lane 0): scores[r], img[r] = key_hi(score), the composite key
// ck[r].
__device__ __forceinline__ void put_score(double acc, bool valid, int r, int n, double* scores, uint32_t* img,
                                          unsigned long long* ck) {
  if ((threadIdx.x & 3) == 0 && r < n) {
    const double sc = valid ? acc : -INFINITY;
    scores[r] = sc;
    img[r] = key_hi(sc);
    ck[r] = rank_key(img[r], r);
  }
}

// Reduces a loaded tile against the summed query held in registers and writes the scores of its
// rows.
template <int D, int PASS>
__device__ __forceinline__ void tile_dot(const RowTile<D, PASS>& t, int n, int r0, const QReg<D>& q,
                                         double* scores, uint32_t* img, unsigned long long* ck) {
  constexpr int ROWS = kWave / 4;
  const int rq = (threadIdx.x % kWave) >> 2;
#pragma unroll
  for (int p = 0; p < PASS; ++p) {
    double acc = 0.0;
#pragma unroll
    for (int c = 0; c < D / 16; ++c)
      acc += q.v[c][0] * (double)t.x[p][c].x + q.v[c][1] * (double)t.x[p][c].y + q.v[c][2] * (double)t.x[p][c].z +
             q.v[c][3] * (double)t.x[p][c].w;
    put_score(group_sum<4>(acc), t.valid[p], r0 + p * ROWS + rq, n, scores, img, ck);
  }
}

// The same with the summed query read from LDS at every row (fewer registers).
template <int D, int PASS>
__device__ __forceinline__ void tile_dot_lds(const RowTile<D, PASS>& t, int n, int r0, const double* qsum,
                                             double* scores, uint32_t* img, unsigned long long* ck) {
  constexpr int ROWS = kWave / 4;
  const int lane = threadIdx.x % kWave, rq = lane >> 2, qk = lane & 3;
#pragma unroll
  for (int p = 0; p < PASS; ++p) {
    double acc = 0.0;
#pragma unroll
    for (int c = 0; c < D / 16; ++c) {
      const double2 q01 = *(const double2*)(qsum + c * 16 + qk * 4);
      const double2 q23 = *(const double2*)(qsum + c * 16 + qk * 4 + 2);
      acc += q01.x * (double)t.x[p][c].x + q01.y * (double)t.x[p][c].y + q23.x * (double)t.x[p][c].z +
             q23.y * (double)t.x[p][c].w;
    }
    put_score(group_sum<4>(acc), t.valid[p], r0 + p * ROWS + rq, n, scores, img, ck);
  }
}

// Max-product bound (Eq. 2) of a loaded tile of two-row representatives (r^max in floats [0, D),
// r^min in [D, 2D) of each row): sum over the G heads and the channels of
// max(q_{g,i} r^max_i, q_{g,i} r^min_i) in fp64 (the products are exact), qh = [G][D] (LDS).
template <int D, int PASS>
__device__ __forceinline__ void tile_dot_mp(const RowTile<2 * D, PASS>& t, int n, int r0, const double* qh, int G,
                                            double* scores, uint32_t* img, unsigned long long* ck) {
  constexpr int ROWS = kWave / 4;
  const int lane = threadIdx.x % kWave, rq = lane >> 2, qk = lane & 3;
#pragma unroll
  for (int p = 0; p < PASS; ++p) {
    double acc = 0.0;
    for (int g = 0; g < G; ++g) {
      const double* qg = qh + g * D;
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const double2 q01 = *(const double2*)(qg + c * 16 + qk * 4);
        const double2 q23 = *(const double2*)(qg + c * 16 + qk * 4 + 2);
        const float4 hi = t.x[p][c], lo = t.x[p][c + D / 16];
        acc += fmax(q01.x * (double)hi.x, q01.x * (double)lo.x) + fmax(q01.y * (double)hi.y, q01.y * (double)lo.y) +
               fmax(q23.x * (double)hi.z, q23.x * (double)lo.z) + fmax(q23.y * (double)hi.w, q23.y * (double)lo.w);
      }
    }
    acc = group_sum<4>(acc);
    const int r = r0 + p * ROWS + rq;
    if (qk == 0 && r < n) {
      const double sc = t.valid[p] ? acc : -INFINITY;
      scores[r] = sc;
      img[r] = key_hi(sc);
      ck[r] = rank_key(img[r], r);
    }
  }
}

// Largest per-head similarity of a loaded tile over the G heads, qh = [G][D] (LDS): the dot
// product (MPB false) or the max-product bound of two-row representatives (MPB true). Each head's
// sum is complete (quad-reduced) before the maximum is taken.
template <int D, int PASS, bool MPB>
__device__ __forceinline__ void tile_dot_gmax(const RowTile<MPB ? 2 * D : D, PASS>& t, int n, int r0,
                                              const double* qh, int G, double* scores, uint32_t* img,
                                              unsigned long long* ck) {
  constexpr int ROWS = kWave / 4;
  const int lane = threadIdx.x % kWave, rq = lane >> 2, qk = lane & 3;
#pragma unroll
  for (int p = 0; p < PASS; ++p) {
    double best = -INFINITY;
    for (int g = 0; g < G; ++g) {
      const double* qg = qh + g * D;
      double acc = 0.0;
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const double2 q01 = *(const double2*)(qg + c * 16 + qk * 4);
        const double2 q23 = *(const double2*)(qg + c * 16 + qk * 4 + 2);
        const float4 x = t.x[p][c];
        if constexpr (MPB) {
          const float4 lo = t.x[p][c + D / 16];
          acc += fmax(q01.x * (double)x.x, q01.x * (double)lo.x) + fmax(q01.y * (double)x.y, q01.y * (double)lo.y) +
                 fmax(q23.x * (double)x.z, q23.x * (double)lo.z) + fmax(q23.y * (double)x.w, q23.y * (double)lo.w);
        } else {
          acc += q01.x * (double)x.x + q01.y * (double)x.y + q23.x * (double)x.z + q23.y * (double)x.w;
        }
      }
      best = fmax(best, group_sum<4>(acc));
    }
    put_score(best, t.valid[p], r0 + p * ROWS + rq, n, scores, img, ck);
  }
}

// Scoring of one mode: dot-product modes (linear, average) take the group's summed query (from
// registers if QREG, else from LDS), the max-product bound the G separate queries (LDS) and
// two-row representatives (one row pass in flight). GMAX: the maximum over the G heads' own
// similarities instead of their sum (separate queries in LDS).
template <int D, int PASS, bool MP, bool QREG = true, bool GMAX = false>
struct Scoring {
  static constexpr int RW = MP ? 2 * D : D;  // floats per representative
  static constexpr int P = MP ? 1 : PASS;    // row passes per wave
  static constexpr bool kSep = MP || GMAX;   // one query row per head
  static constexpr bool kReg = QREG && !kSep;
  using Tile = RowTile<RW, P>;
  struct Empty {};
  struct Query {
    std::conditional_t<kReg, QReg<D>, Empty> reg;
    const double* lds;  // summed query [D], or the bound's [G][D]
    int G;
  };
  // after the query rows are in LDS (and visible to the calling thread)
  __device__ static void prepare(Query& q, const double* lds, int G) {
    q.lds = lds;
    q.G = G;
    if constexpr (kReg) qreg_load<D>(lds, q.reg);
  }
  __device__ static void dot(const Tile& t, int n, int r0, const Query& q, double* scores, uint32_t* img,
                             unsigned long long* ck) {
    if constexpr (GMAX)
      tile_dot_gmax<D, P, MP>(t, n, r0, q.lds, q.G, scores, img, ck);
    else if constexpr (MP)
      tile_dot_mp<D, P>(t, n, r0, q.lds, q.G, scores, img, ck);
    else if constexpr (kReg)
      tile_dot<D, P>(t, n, r0, q.reg, scores, img, ck);
    else
      tile_dot_lds<D, P>(t, n, r0, q.lds, scores, img, ck);
  }
};

// Query rows kept in LDS: the group sum (SEP false) or each of the G heads (SEP true), fp64.
template <class DT, int D, bool SEP>
__device__ __forceinline__ void load_query(const void* q, size_t q0, int G, double* dst, int t0, int nt) {
  if constexpr (SEP) {
    for (int i = t0; i < G * D; i += nt) dst[i] = (double)load_elt<DT>(q, q0 + (size_t)i);
  } else {
    for (int i = t0; i < D; i += nt) {
      double acc = 0.0;
      for (int g = 0; g < G; ++g) acc += (double)load_elt<DT>(q, q0 + (size_t)g * D + i);
      dst[i] = acc;
    }
  }
}

// High 32 bits of an order-preserving integer image of a score (-0 is folded into +0 first).
__device__ __forceinline__ uint32_t key_hi(double x) {
  const unsigned long long b = (unsigned long long)__double_as_longlong(x + 0.0);
  const unsigned long long u = (b >> 63) ? ~b : (b | 0x8000000000000000ull);
  return (uint32_t)(u >> 32);
}

// Unique 64-bit ranking key: the 32-bit image of the score, then the complemented index, so that
// integer order is (image desc, index asc). It orders exactly like (score desc, index asc) except
// inside a group of entries whose images tie; repair_top() re-ranks such a group when it straddles
// the top-k boundary.
__device__ __forceinline__ unsigned long long rank_key(uint32_t img, int i) {
  return ((unsigned long long)img << 32) | (uint32_t)~(uint32_t)i;
}

// Number of keys in key[j0, j1) greater than ki; keys are LDS broadcasts, 16 loads in flight.
__device__ __forceinline__ int count_above(const unsigned long long* key, int j0, int j1,
                                           unsigned long long ki) {
  int c = 0, j = j0;
  for (; j + 16 <= j1; j += 16) {
    unsigned long long v[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) v[u] = key[j + u];
#pragma unroll
    for (int u = 0; u < 16; ++u) c += v[u] > ki;
  }
  for (; j < j1; ++j) c += key[j] > ki;
  return c;
}

// Top k of n entries by composite key, by one workgroup: top[r] = entry of rank r < k, bnd[0] /
// bnd[1] = entries of rank k-1 / k (or -1). Small sets: every entry counts the keys above it.
// Larger sets (a tournament): each slice of 32 entries keeps its local top k+1 in a list, then
// the list entries count the list keys above them. An entry of global rank r <= k is in the list
// (fewer than k+1 keys of its slice beat it) and so is every key above it, so its count is its
// rank; an entry of rank > k finds at least k+1 list keys above it (a slice holding a key above
// it that is not in the list contributes its whole top k+1). list_k / list_i hold
// ceil(n / 32) * (k + 1) entries; ends with a barrier.
constexpr int kSlice = 32;

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// Synchronisation of the threads that rank one set: a whole workgroup, or one wave.
struct BlockSync {
  __device__ static void sync() { __syncthreads(); }
};
struct WaveSync {
  __device__ static void sync() { wave_sync(); }
};

__host__ __device__ inline bool use_tournament(int n, int k) {
  return n > 2 * kSlice && ((n + kSlice - 1) / kSlice) * (k + 1) * 2 <= n;
}

// NT threads rank the set (a workgroup with SY = BlockSync, or one wave with NT = 64 and
// SY = WaveSync); bnd[] must hold -1 on entry.
template <int NT, class SY = BlockSync>
__device__ void block_topk(const unsigned long long* ck, int n, int k, unsigned long long* list_k, int* list_i,
                           int* top, int* bnd) {
  const int tid = threadIdx.x % NT;
  if (!use_tournament(n, k)) {
    for (int i = tid; i < n; i += NT) {
      const int r = count_above(ck, 0, n, ck[i]);
      if (r < k) top[r] = i;
      if (r == k - 1) bnd[0] = i;
      if (r == k) bnd[1] = i;
    }
    SY::sync();
    return;
  }
  const int m = (n + kSlice - 1) / kSlice * (k + 1);
  for (int c = tid; c < m; c += NT) {  // slots a short slice leaves empty: key 0 beats nothing
    list_k[c] = 0ull;
    list_i[c] = -1;
  }
  SY::sync();
  for (int i = tid; i < n; i += NT) {
    const int s0 = i / kSlice * kSlice;
    const int r = count_above(ck, s0, min(n, s0 + kSlice), ck[i]);
    if (r <= k) {
      list_k[i / kSlice * (k + 1) + r] = ck[i];
      list_i[i / kSlice * (k + 1) + r] = i;
    }
  }
  SY::sync();
  for (int c = tid; c < m; c += NT) {
    const int i = list_i[c];
    if (i < 0) continue;
    const int r = count_above(list_k, 0, m, list_k[c]);
    if (r < k) top[r] = i;
    if (r == k - 1) bnd[0] = i;
    if (r == k) bnd[1] = i;
  }
  SY::sync();
}

// When the images of the entries at composite ranks k-1 and k tie, the composite order inside that
// image group (index only) may differ from the exact (score desc, index asc) order: the group's
// members re-rank themselves exactly and take the top slots from the group's first rank on.
// Uniform across the workgroup (reads LDS only); ends with a barrier when it does anything.
template <int NT, class SY = BlockSync>
__device__ void repair_top(const double* sc, const uint32_t* img, int n, int k, const int* bnd, int* top) {
  const int a = bnd[0], b = bnd[1];
  if (a < 0 || b < 0 || img[a] != img[b]) return;
  const uint32_t t = img[a];
  for (int i = threadIdx.x % NT; i < n; i += NT) {
    if (img[i] != t) continue;
    int first = 0, r = 0;
    for (int j = 0; j < n; ++j) {
      first += img[j] > t;
      if (j != i && img[j] == t) r += (sc[j] > sc[i]) | ((sc[j] == sc[i]) & (j < i));
    }
    if (first + r < k) top[first + r] = i;
  }
  SY::sync();
}

// Position of top[j] among top[0, k) in ascending entry order (entries are distinct).
__device__ __forceinline__ int ascending_pos(const int* top, int k, int j) {
  const int v = top[j];
  int p = 0, u = 0;
  for (; u + 4 <= k; u += 4) {
    const int t0 = top[u], t1 = top[u + 1], t2 = top[u + 2], t3 = top[u + 3];
    p += (t0 < v) + (t1 < v) + (t2 < v) + (t3 < v);
  }
  for (; u < k; ++u) p += top[u] < v;
  return p;
}

// Writes the level-2 result: entry top[j] (j < k_clusters) goes to its ascending position, in
// layer l and the following layers of the call that share its selection. Threads t0, t0 + nt, ...
template <bool COH>
__device__ __forceinline__ void emit_selection(const SelectArgs& a, const int* top, const int* cand,
                                               const double* s2, int l, int b, int h, int t0, int nt) {
  const int abs_l = a.layer0 + l;
  int l_end = l + 1;  // layers [l, l_end) of the call use this selection
  while (l_end < a.n_layers && owner_layer(a.layer0 + l_end, a.period, a.start) == abs_l) ++l_end;
  const size_t stride = (size_t)a.B * a.Hsel * a.k_clusters;
  const size_t o0 = (((size_t)l * a.B + b) * a.Hsel + h) * a.k_clusters;
  for (int j = t0; j < a.k_clusters; j += nt) {
    const int i = top[j], p = ascending_pos(top, a.k_clusters, j);
    const int c = cand[i];
    const float sc = (float)s2[i];
    for (int l2 = l; l2 < l_end; ++l2) {
      const size_t o = o0 + (size_t)(l2 - l) * stride + p;
      store_sel<COH>(a.sel + o, c);
      if (a.sel_score) a.sel_score[o] = sc;
    }
  }
}

// Writes the level-2 result of a workgroup that attends one layer itself: entry top[j] (j <
// k_clusters) goes to its ascending position of `pick` (LDS, read by the same workgroup's attention)
// and of layer l's row of the selection output (layer l uses the selection of its owner head, which
// the workgroup computed). Threads t0, t0 + nt, ...
__device__ __forceinline__ void emit_pick(const SelectArgs& a, const int* top, const int* cand, const double* s2,
                                          int l, int b, int h, int32_t* pick, int t0, int nt) {
  const size_t o0 = (((size_t)l * a.B + b) * a.Hsel + h) * a.k_clusters;
  for (int j = t0; j < a.k_clusters; j += nt) {
    const int i = top[j], p = ascending_pos(top, a.k_clusters, j);
    const int c = cand[i];
    pick[p] = c;
    a.sel[o0 + p] = c;
    if (a.sel_score) a.sel_score[o0 + p] = (float)s2[i];
  }
}

// ---------------------------------------------------------------------------------------------
// Register ranking of the workgroup-per-head selection, for up to 64 super-clusters and up to 512
// candidates (fewer than 64 kept when there are more than 64): one entry per lane, ranks counted
// against LDS broadcasts of the keys, selected sets as wave ballots, ascending output positions as
// bit counts of a ballot below the lane. No per-thread list walks and, at level 1, no barrier: every
// wave ranks the super-clusters itself and derives its own candidate rows from the ballot.
__host__ __device__ inline bool register_ranking(int S, int NC, int k_clusters) {
  return S <= kWave && (NC <= kWave || (NC <= 8 * kWave && k_clusters < kWave));
}

// Exact rank (score desc, index asc) of entry i among sc[0, n) (LDS): the boundary fallback when the
// composite keys of ranks k-1 and k share their 32-bit score image.
__device__ __forceinline__ int exact_rank(const double* sc, int n, int i) {
  const double si = sc[i];
  int c = 0;
  for (int j = 0; j < n; ++j) {
    const double x = sc[j];
    c += (x > si) | ((x == si) & (j < i));
  }
  return c;
}

// Position of the n-th (from 0) set bit of m (n below its bit count).
__device__ __forceinline__ int nth_set_bit(unsigned long long m, int n) {
  int pos = 0;
  uint32_t x = (uint32_t)m;
  int c = __popc(x);
  if (n >= c) {
    n -= c;
    pos = 32;
    x = (uint32_t)(m >> 32);
  }
#pragma unroll
  for (int w = 16; w >= 1; w >>= 1) {
    c = __popc(x & ((1u << w) - 1u));
    if (n >= c) {
      n -= c;
      pos += w;
      x >>= w;
    }
  }
  return pos;
}

// Output of one selected entry: cluster c with score sc at ascending position p, to the LDS pick
// list and layer pick_layer's row (pick set), or to every layer of [l, l_end) of the call.
template <bool COH>
__device__ __forceinline__ void emit_entry(const SelectArgs& a, int c, float sc, int p, int l, int l_end, int b,
                                           int h, int32_t* pick, int pick_layer) {
  if (pick) {
    pick[p] = c;
    const size_t o = (((size_t)pick_layer * a.B + b) * a.Hsel + h) * a.k_clusters + p;
    a.sel[o] = c;
    if (a.sel_score) a.sel_score[o] = sc;
    return;
  }
  const size_t stride = (size_t)a.B * a.Hsel * a.k_clusters;
  const size_t o0 = (((size_t)l * a.B + b) * a.Hsel + h) * a.k_clusters + p;
  for (int l2 = l; l2 < l_end; ++l2) {
    store_sel<COH>(a.sel + o0 + (size_t)(l2 - l) * stride, c);
    if (a.sel_score) a.sel_score[o0 + (size_t)(l2 - l) * stride] = sc;
  }
}

// LDS carve-up of the one-workgroup-per-head selection (host and device). The key array is padded
// to whole 64-entry slices and the tournament list to whole 16-key batches.
struct BlockLds {
  size_t qsum, s1, s2, ck, img1, img2, list_k, list_i, top, cand, part, total;
};
__host__ __device__ inline BlockLds block_lds(int D, int S, int NC, int qrows) {
  auto al = [](size_t x) { return (x + 15) & ~(size_t)15; };
  const int m = S > NC ? S : NC;
  const int m64 = (m + 63) / 64 * 64;
  BlockLds o;
  o.qsum = 0;
  o.s1 = al(o.qsum + (size_t)qrows * D * 8);
  o.s2 = al(o.s1 + (size_t)S * 8);
  o.ck = al(o.s2 + (size_t)NC * 8);
  o.img1 = al(o.ck + (size_t)(kWave + m64) * 8);  // level 1 (register ranking: 64 keys), then level 2
  o.img2 = al(o.img1 + (size_t)S * 4);
  o.list_k = al(o.img2 + (size_t)NC * 4);
  o.list_i = al(o.list_k + (size_t)(m64 + 16) * 8);
  o.top = al(o.list_i + (size_t)(m64 + 16) * 4);
  o.cand = al(o.top + (size_t)(m > kWave ? m : kWave) * 4);
  o.part = al(o.cand + (size_t)NC * 4);  // partial counts: level 1, then level 2 (8 x 64 each)
  o.total = al(o.part + (size_t)2 * 8 * kWave * 4);
  return o;
}

// Keys of keys[base, base + KPC) above `mine`, all read before the compares.
template <int KPC>
__device__ __forceinline__ int count_chunk(const unsigned long long* keys, int base, unsigned long long mine) {
  unsigned long long v[KPC];
#pragma unroll
  for (int u = 0; u < KPC; ++u) v[u] = keys[base + u];
  int c = 0;
#pragma unroll
  for (int u = 0; u < KPC; ++u) c += v[u] > mine;
  return c;
}

// Partial ranks of the entries of n_slice 64-entry slices of `keys` (padded to whole slices): the
// workgroup's waves take the items (slice, chunk) of cps chunks per slice (NW for one slice, else 1),
// and item t writes, for the entry of its slice in each lane, the number of its chunk's keys above
// that entry to part[t * 64 + lane]. Returns cps. The rank of entry `lane` of slice sl within its
// slice is then the sum of part[(sl * cps + c) * 64 + lane] over c < cps (after a barrier).
template <int NW>
__device__ __forceinline__ int slice_partials(const unsigned long long* keys, int n_slice, int* part) {
  const int w = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  // chunks only for a single slice: with several slices the extra barrier and partial reads cost
  // more than the compares they save (measured)
  const int cps = n_slice > 1 ? 1 : NW >= 8 ? 8 : NW >= 4 ? 4 : NW >= 2 ? 2 : 1;
  const int kpc = kWave / cps;
  for (int t = w; t < n_slice * cps; t += NW) {
    const int sl = t / cps, base = sl * kWave + (t % cps) * kpc;
    const unsigned long long mine = keys[sl * kWave + lane];
    int c;
    if (kpc == 8)
      c = count_chunk<8>(keys, base, mine);
    else if (kpc == 16)
      c = count_chunk<16>(keys, base, mine);
    else if (kpc == 32)
      c = count_chunk<32>(keys, base, mine);
    else
      c = count_chunk<64>(keys, base, mine);
    part[t * kWave + lane] = c;
  }
  return cps;
}

// Sum of the cps partial ranks of entry `lane` of slice sl.
__device__ __forceinline__ int slice_rank(const int* part, int sl, int cps) {
  const int lane = threadIdx.x % kWave;
  int r = 0;
  for (int c = 0; c < cps; ++c) r += part[(sl * cps + c) * kWave + lane];
  return r;
}

// The rank of every lane's entry of a 64-entry slice is exact in (score desc, index asc) unless the
// entries of ranks k-1 and k share a score image: then every lane takes its exact rank.
__device__ __forceinline__ int exact_at_boundary(int r, const double* sc, const uint32_t* img, int n, int k) {
  const int lane = threadIdx.x % kWave;
  const unsigned long long ba = __ballot(r == k - 1), bb = __ballot(r == k);
  if (ba && bb) {
    const int la = __ffsll((long long)ba) - 1, lb = __ffsll((long long)bb) - 1;
    if (la < n && lb < n && img[la] == img[lb]) r = lane < n ? exact_rank(sc, n, lane) : kWave;
  }
  return r;
}

// Continuation of select_block once the level-1 scores are written (register ranking): level-1
// top-k_super as a ballot in every wave, level-2 rows derived from it, level-2 ranking by 64-entry
// slices (each keeps its local top k_clusters + 1) and a count over the survivors, output by wave 0.
// The ranks of a single 64-entry set are counted by all waves together (partial counts over key
// chunks).
template <class SC, int NW, bool COH>
__device__ void select_block_reg(const SelectArgs& a, typename SC::Tile& tile, const typename SC::Query& qr,
                                 const float* cent, const double* s1, double* s2, unsigned long long* ck,
                                 const uint32_t* img1, uint32_t* img2, unsigned long long* list_k, int* list_i,
                                 int* top, int* part, int* bnd2, int l, int b, int h, int32_t* pick,
                                 int pick_layer) {
  constexpr int NT = NW * kWave;
  constexpr int TILE = NW * (kWave / 4) * SC::P;
  const int tid = threadIdx.x, w = tid / kWave, lane = tid % kWave;
  for (int j = a.S + tid; j < kWave; j += NT) ck[j] = rank_key(0u, j);  // padding below every score
  __syncthreads();
  const int cps1 = slice_partials<NW>(ck, 1, part);
  __syncthreads();
  const unsigned long long sup =
      __ballot(exact_at_boundary(slice_rank(part, 0, cps1), s1, img1, a.S, a.k_super) < a.k_super);

  // level 2: the member clusters of the selected super-clusters, in ascending order; their keys
  // follow the level-1 keys and their partial counts the level-1 ones, which slower waves may still
  // be reading
  ck += kWave;
  part += NW * kWave;
  const int f = a.f, C = a.C, NC = a.NC, k = a.k_clusters;
  const int fs = (f & (f - 1)) == 0 ? __builtin_ctz(f) : -1;  // shift when f is a power of two
  auto cand = [=](int r) {
    const int q = fs >= 0 ? r >> fs : r / f;
    const int c = nth_set_bit(sup, q) * f + (r - q * f);
    return c < C ? c : -1;
  };
  for (int r0 = w * (TILE / NW); r0 < NC; r0 += TILE) {
    tile_load_fn<SC::RW, SC::P>(cent, cand, NC, r0, tile);
    SC::dot(tile, NC, r0, qr, s2, img2, ck);
  }
  const int n64 = (NC + kWave - 1) / kWave * kWave, n_slice = n64 / kWave;
  for (int j = NC + tid; j < n64; j += NT) ck[j] = rank_key(0u, j);
  if (tid < 2) bnd2[tid] = -1;
  const int l_end = a.own.end(a.own.index_of(l));  // layers [l, l_end) of the call use this selection
  __syncthreads();

  if (n_slice == 1) {  // one slice: its ranks are final; wave 0 writes the result
    const int cps = slice_partials<NW>(ck, 1, part);
    __syncthreads();
    if (w == 0) {
      const int r = exact_at_boundary(slice_rank(part, 0, cps), s2, img2, NC, k);
      const unsigned long long chosen = __ballot(r < k);
      if (r < k) {
        const int p = __popcll(chosen & ((1ull << lane) - 1ull));
        emit_entry<COH>(a, cand(lane), (float)s2[lane], p, l, l_end, b, h, pick, pick_layer);
      }
    }
    return;
  }
  // each slice keeps its entries of local rank <= k
  const int per = k + 1, m = n_slice * per, m16 = (m + 15) / 16 * 16;
  for (int sl = w; sl < n_slice; sl += NW) {
    const int e = sl * kWave + lane;
    const int r = count_above(ck, sl * kWave, sl * kWave + kWave, ck[e]);
    if (r <= k) {
      list_k[sl * per + r] = ck[e];
      list_i[sl * per + r] = e < NC ? e : -1;
    }
  }
  for (int j = m + tid; j < m16; j += NT) list_k[j] = 0ull;  // batch padding: above nothing
  __syncthreads();
  // a survivor's count of the survivors above it is its rank when below k + 1
  for (int x = tid; x < m; x += NT) {
    const int r = count_above(list_k, 0, m16, list_k[x]);
    const int i = list_i[x];
    if (r < k) top[r] = i;
    if (r == k - 1) bnd2[0] = i;
    if (r == k) bnd2[1] = i;
  }
  __syncthreads();
  repair_top<NT>(s2, img2, NC, k, bnd2, top);
  if (w == 0 && lane < k) {
    const int i = top[lane];
    emit_entry<COH>(a, cand(i), (float)s2[i], ascending_pos(top, k, lane), l, l_end, b, h, pick, pick_layer);
  }
}

// Selection of owner head `ou` by one workgroup of NW waves (`smem`: block_lds().total bytes).
// COH: write the selection with device-coherent stores (read by another workgroup of the launch).
// PASS: row passes per wave in flight (registers against memory parallelism). MP: max-product
// bound scores (two-row representatives), else dot-product scores. QREG: keep the summed query in
// registers (faster) rather than reading it from LDS at every row (fewer registers). GMAX: the
// unit's score is the maximum of its q-heads' similarities, not their sum. pick: if not null, the
// selection goes to this LDS array and to layer pick_layer's output row only (emit_pick), instead
// of every layer of the call that shares it.
template <class DT, int D, int NW, bool COH, int PASS = 2, bool MP = false, bool QREG = true, bool GMAX = false>
__device__ void select_block(const SelectArgs& a, int ou, unsigned char* smem, int32_t* pick = nullptr,
                             int pick_layer = -1) {
  using SC = Scoring<D, PASS, MP, QREG, GMAX>;
  constexpr int NT = NW * kWave;
  constexpr int TILE = NW * (kWave / 4) * SC::P;  // rows per workgroup pass
  const int G = a.Hq / a.Hsel;  // q-heads of the unit
  const BlockLds lay = block_lds(D, a.S, a.NC, SC::kSep ? G : 1);
  double* qsum = (double*)(smem + lay.qsum);
  double* s1 = (double*)(smem + lay.s1);
  double* s2 = (double*)(smem + lay.s2);
  unsigned long long* ck = (unsigned long long*)(smem + lay.ck);  // composite keys, level 1 then 2
  uint32_t* img1 = (uint32_t*)(smem + lay.img1);
  uint32_t* img2 = (uint32_t*)(smem + lay.img2);
  unsigned long long* list_k = (unsigned long long*)(smem + lay.list_k);
  int* list_i = (int*)(smem + lay.list_i);
  int* top = (int*)(smem + lay.top);
  int* cand = (int*)(smem + lay.cand);
  __shared__ int bnd1[2], bnd2[2];

  const int BH = a.B * a.Hsel;
  const int l = a.own.local(ou / BH), b = (ou / a.Hsel) % a.B, h = ou % a.Hsel;
  const size_t unit = ((size_t)l * a.B + b) * a.Hkv + h / a.rep_div;  // representatives' kv head
  const int tid = threadIdx.x, w = tid / kWave;
  const float* scent = a.scent + unit * a.ss * SC::RW;
  const float* cent = a.cent + unit * a.cs * SC::RW;

  // the first level-1 tile is in flight while the query rows are loaded
  typename SC::Tile tile;
  const int r1 = w * (TILE / NW);
  if (r1 < a.S) tile_load<SC::RW, SC::P>(scent, nullptr, a.S, r1, tile);
  const size_t q0 = (((size_t)l * a.B + b) * a.Hq + (size_t)h * G) * D;
  load_query<DT, D, SC::kSep>(a.q, q0, G, qsum, tid, NT);
  if (tid < 2) {
    bnd1[tid] = -1;
    bnd2[tid] = -1;
  }
  __syncthreads();
  typename SC::Query qr;
  SC::prepare(qr, qsum, G);

  // level 1: super-cluster scores, top-k_super, their member clusters in ascending order
  if (r1 < a.S) SC::dot(tile, a.S, r1, qr, s1, img1, ck);
  for (int r0 = r1 + TILE; r0 < a.S; r0 += TILE) {
    tile_load<SC::RW, SC::P>(scent, nullptr, a.S, r0, tile);
    SC::dot(tile, a.S, r0, qr, s1, img1, ck);
  }
  if (register_ranking(a.S, a.NC, a.k_clusters)) {
    select_block_reg<SC, NW, COH>(a, tile, qr, cent, s1, s2, ck, img1, img2, list_k, list_i, top,
                                  (int*)(smem + lay.part), bnd2, l, b, h, pick, pick_layer);
    return;
  }
  __syncthreads();
  block_topk<NT>(ck, a.S, a.k_super, list_k, list_i, top, bnd1);
  repair_top<NT>(s1, img1, a.S, a.k_super, bnd1, top);
  for (int j = tid; j < a.k_super; j += NT) {
    const int sup = top[j], p = ascending_pos(top, a.k_super, j);
    for (int m = 0; m < a.f; ++m) {
      const int c = sup * a.f + m;
      cand[p * a.f + m] = c < a.C ? c : -1;
    }
  }
  __syncthreads();

  // level 2: candidate scores, top-k_clusters, written in ascending cluster order
  for (int r0 = w * (TILE / NW); r0 < a.NC; r0 += TILE) {
    tile_load<SC::RW, SC::P>(cent, cand, a.NC, r0, tile);
    SC::dot(tile, a.NC, r0, qr, s2, img2, ck);
  }
  __syncthreads();
  block_topk<NT>(ck, a.NC, a.k_clusters, list_k, list_i, top, bnd2);
  repair_top<NT>(s2, img2, a.NC, a.k_clusters, bnd2, top);
  if (pick)
    emit_pick(a, top, cand, s2, pick_layer, b, h, pick, tid, NT);
  else
    emit_selection<COH>(a, top, cand, s2, l, b, h, tid, NT);
}

// ---------------------------------------------------------------------------------------------
// One wave per owner head (many heads): the same two levels with wave-local synchronisation only,
// so thousands of heads progress independently. Each wave owns a private LDS region.
constexpr int kWaveMaxSuper = 256;        // limits of the wave variant's LDS region
constexpr int kWaveMaxCand = 256;

// LDS region of one wave of the wave-per-head selection (host and device).
struct WaveLds {
  size_t qsum, s1, s2, ck, img, list_k, list_i, top, cand, bnd, total;
};
__host__ __device__ inline WaveLds wave_lds(int D, int S, int NC, int qrows) {
  auto al = [](size_t x) { return (x + 15) & ~(size_t)15; };
  const int m = S > NC ? S : NC;
  WaveLds o;
  o.qsum = 0;
  o.s1 = al((size_t)qrows * D * 8);
  o.s2 = al(o.s1 + (size_t)S * 8);
  o.ck = al(o.s2 + (size_t)NC * 8);
  o.img = al(o.ck + (size_t)m * 8);
  o.list_k = al(o.img + (size_t)m * 4);  // a tournament list is at most half its set
  o.list_i = al(o.list_k + (size_t)m * 4);
  o.top = al(o.list_i + (size_t)m * 2);
  o.cand = al(o.top + (size_t)m * 4);
  o.bnd = al(o.cand + (size_t)NC * 4);
  o.total = al(o.bnd + 4 * sizeof(int));
  return o;
}
__host__ __device__ inline size_t wave_region_bytes(int D, int S, int NC, int qrows) {
  return wave_lds(D, S, NC, qrows).total;
}

// Selection of owner heads ou0 + w, one per wave w (`smem`: waves x wave_region_bytes()).
template <class DT, int D, bool COH, bool MP = false, bool GMAX = false>
__device__ void select_waves(const SelectArgs& a, int ou0, unsigned char* smem) {
  using SC = Scoring<D, 2, MP, true, GMAX>;
  constexpr int TILE = (kWave / 4) * SC::P;  // rows per wave pass
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  const int BH = a.B * a.Hsel;
  const int ou = ou0 + w;  // (owner index * B + b) * Hsel + h
  if (ou >= a.own.n * BH) return;
  const int G = a.Hq / a.Hsel;  // q-heads of the unit
  const WaveLds lay = wave_lds(D, a.S, a.NC, SC::kSep ? G : 1);
  unsigned char* base = smem + (size_t)w * lay.total;
  double* qsum = (double*)(base + lay.qsum);
  double* s1 = (double*)(base + lay.s1);
  double* s2 = (double*)(base + lay.s2);
  unsigned long long* ck = (unsigned long long*)(base + lay.ck);
  uint32_t* img = (uint32_t*)(base + lay.img);
  unsigned long long* list_k = (unsigned long long*)(base + lay.list_k);
  int* list_i = (int*)(base + lay.list_i);
  int* top = (int*)(base + lay.top);
  int* cand = (int*)(base + lay.cand);
  int* bnd = (int*)(base + lay.bnd);  // boundary entries of level 1 ([0], [1]) and level 2 ([2], [3])

  const int l = a.own.local(ou / BH), b = (ou / a.Hsel) % a.B, h = ou % a.Hsel;
  const size_t unit = ((size_t)l * a.B + b) * a.Hkv + h / a.rep_div;  // representatives' kv head
  const float* scent = a.scent + unit * a.ss * SC::RW;
  const float* cent = a.cent + unit * a.cs * SC::RW;

  // the first level-1 tile is in flight while the query rows are loaded
  typename SC::Tile tile;
  tile_load<SC::RW, SC::P>(scent, nullptr, a.S, 0, tile);
  const size_t q0 = (((size_t)l * a.B + b) * a.Hq + (size_t)h * G) * D;
  load_query<DT, D, SC::kSep>(a.q, q0, G, qsum, lane, kWave);
  if (lane < 4) bnd[lane] = -1;
  wave_sync();
  typename SC::Query qr;
  SC::prepare(qr, qsum, G);

  // level 1
  SC::dot(tile, a.S, 0, qr, s1, img, ck);
  for (int r0 = TILE; r0 < a.S; r0 += TILE) {
    tile_load<SC::RW, SC::P>(scent, nullptr, a.S, r0, tile);
    SC::dot(tile, a.S, r0, qr, s1, img, ck);
  }
  wave_sync();
  block_topk<kWave, WaveSync>(ck, a.S, a.k_super, list_k, list_i, top, bnd);
  repair_top<kWave, WaveSync>(s1, img, a.S, a.k_super, bnd, top);
  for (int j = lane; j < a.k_super; j += kWave) {
    const int sup = top[j], p = ascending_pos(top, a.k_super, j);
    for (int m = 0; m < a.f; ++m) {
      const int c = sup * a.f + m;
      cand[p * a.f + m] = c < a.C ? c : -1;
    }
  }
  wave_sync();

  // level 2
  for (int r0 = 0; r0 < a.NC; r0 += TILE) {
    tile_load<SC::RW, SC::P>(cent, cand, a.NC, r0, tile);
    SC::dot(tile, a.NC, r0, qr, s2, img, ck);
  }
  wave_sync();
  block_topk<kWave, WaveSync>(ck, a.NC, a.k_clusters, list_k, list_i, top, bnd + 2);
  repair_top<kWave, WaveSync>(s2, img, a.NC, a.k_clusters, bnd + 2, top);
  emit_selection<COH>(a, top, cand, s2, l, b, h, lane, kWave);
}

inline size_t select_smem_bytes_dev(int D, int S, int NC, int qrows) { return block_lds(D, S, NC, qrows).total; }

}  // namespace dev
}  // namespace mpc
