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

template <int D, int PASS>
__device__ __forceinline__ void tile_load(const float* M, const int* idx, int n, int r0, RowTile<D, PASS>& t) {
  constexpr int ROWS = kWave / 4;
  const int lane = threadIdx.x % kWave, rq = lane >> 2, qk = lane & 3;
#pragma unroll
  for (int p = 0; p < PASS; ++p) {
    const int r = r0 + p * ROWS + rq;
    const int row = r < n ? (idx ? idx[r] : r) : -1;
    t.valid[p] = row >= 0;
    const float* src = M + (size_t)(t.valid[p] ? row : 0) * D + qk * 4;
#pragma unroll
    for (int c = 0; c < D / 16; ++c) t.x[p][c] = *(const float4*)(src + c * 16);
  }
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

// LDS carve-up of the one-workgroup-per-head selection (host and device).
struct BlockLds {
  size_t qsum, s1, s2, ck, img1, img2, list_k, list_i, top, cand, total;
};
__host__ __device__ inline BlockLds block_lds(int D, int S, int NC, int qrows) {
  auto al = [](size_t x) { return (x + 15) & ~(size_t)15; };
  const int m = S > NC ? S : NC;
  BlockLds o;
  o.qsum = 0;
  o.s1 = al(o.qsum + (size_t)qrows * D * 8);
  o.s2 = al(o.s1 + (size_t)S * 8);
  o.ck = al(o.s2 + (size_t)NC * 8);
  o.img1 = al(o.ck + (size_t)m * 8);
  o.img2 = al(o.img1 + (size_t)S * 4);
  o.list_k = al(o.img2 + (size_t)NC * 4);  // a tournament list is at most half its set
  o.list_i = al(o.list_k + (size_t)m * 8);
  o.top = al(o.list_i + (size_t)m * 4);
  o.cand = al(o.top + (size_t)m * 4);
  o.total = al(o.cand + (size_t)NC * 4);
  return o;
}

// Selection of owner head `ou` by one workgroup of NW waves (`smem`: block_lds().total bytes).
// COH: write the selection with device-coherent stores (read by another workgroup of the launch).
// PASS: row passes per wave in flight (registers against memory parallelism). MP: max-product
// bound scores (two-row representatives), else dot-product scores. QREG: keep the summed query in
// registers (faster) rather than reading it from LDS at every row (fewer registers). GMAX: the
// unit's score is the maximum of its q-heads' similarities, not their sum.
template <class DT, int D, int NW, bool COH, int PASS = 2, bool MP = false, bool QREG = true, bool GMAX = false>
__device__ void select_block(const SelectArgs& a, int ou, unsigned char* smem) {
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
  const int l = a.own.l[ou / BH], b = (ou / a.Hsel) % a.B, h = ou % a.Hsel;
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

  const int l = a.own.l[ou / BH], b = (ou / a.Hsel) % a.B, h = ou % a.Hsel;
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
