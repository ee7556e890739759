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

// scores[r] = sum_i qsum[i] * M[idx(r)][i] for r < n; rows with idx < 0 score -inf.
// Four lanes share a row: at load step c the quad reads 64 contiguous bytes (lane k of the quad
// takes floats c*16 + 4k .. +3), so 16 rows are in flight per wave per step; the quad's fp64
// partial sums meet through two DPP quad swaps.
template <int D, int NW>
__device__ void gemv_rows(const float* M, const int* idx, int n, const double* qsum, double* scores) {
  constexpr int STEPS = D / 16;      // 16-byte loads per lane per row
  constexpr int ROWS = kWave / 4;    // rows per wave per pass
  constexpr int PASS = 2;            // passes in flight
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  const int rq = lane >> 2, qk = lane & 3;
  double qv[STEPS][4];
#pragma unroll
  for (int c = 0; c < STEPS; ++c)
#pragma unroll
    for (int e = 0; e < 4; ++e) qv[c][e] = qsum[c * 16 + qk * 4 + e];
  for (int r0 = w * ROWS * PASS; r0 < n; r0 += NW * ROWS * PASS) {
    float4 x[PASS][STEPS];
    bool valid[PASS];
#pragma unroll
    for (int p = 0; p < PASS; ++p) {
      const int r = r0 + p * ROWS + rq;
      const int row = r < n ? (idx ? idx[r] : r) : -1;
      valid[p] = row >= 0;
      const float* src = M + (size_t)(valid[p] ? row : 0) * D + qk * 4;
#pragma unroll
      for (int c = 0; c < STEPS; ++c) x[p][c] = *(const float4*)(src + c * 16);
    }
#pragma unroll
    for (int p = 0; p < PASS; ++p) {
      double acc = 0.0;
#pragma unroll
      for (int c = 0; c < STEPS; ++c)
        acc += qv[c][0] * (double)x[p][c].x + qv[c][1] * (double)x[p][c].y + qv[c][2] * (double)x[p][c].z +
               qv[c][3] * (double)x[p][c].w;
      acc = group_sum<4>(acc);
      const int r = r0 + p * ROWS + rq;
      if (qk == 0 && r < n) scores[r] = valid[p] ? acc : -INFINITY;
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
// inside a group of entries whose images tie; select_exact() repairs such a group when it straddles
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

// Entries of rank < k by composite key are flagged. bnd[0] / bnd[1] hold the entries of rank
// k-1 / k (published by their lanes, -1 if absent). If their images tie, the tied group is
// re-ranked by exact (score desc, index asc) and only its flags change. Run by one lane; the
// serial part is reached only on an image tie at the boundary.
__device__ void select_exact(const double* sc, const uint32_t* img, const int* rank, int n, int k,
                             const int* bnd, int* flag) {
  const int a = bnd[0], b = bnd[1];
  if (a < 0 || b < 0 || img[a] != img[b]) return;
  const uint32_t t = img[a];
  int first = n;  // lowest composite rank inside the tied group
  for (int i = 0; i < n; ++i)
    if (img[i] == t && rank[i] < first) first = rank[i];
  const int take = k - first;
  for (int i = 0; i < n; ++i) {
    if (img[i] != t) continue;
    int r = 0;
    for (int j = 0; j < n; ++j)
      if (j != i && img[j] == t) r += (sc[j] > sc[i]) | ((sc[j] == sc[i]) & (j < i));
    flag[i] = r < take;
  }
}

// rank[i] for all entries: every thread of the workgroup takes an (entry, slice) pair so that small
// sets still use all lanes; slice counts meet in LDS.
template <int NT>
__device__ void rank_all(const unsigned long long* key, int n, int* rank) {
  const int parts = n < NT ? NT / n : 1;
  for (int t = threadIdx.x; t < n * parts; t += NT) {
    const int i = t % n, part = t / n;
    atomicAdd(&rank[i], count_above(key, part * n / parts, (part + 1) * n / parts, key[i]));
  }
}

// pos[i] = number of set flags before entry i (wave ballots, then wave totals through LDS).
template <int NW>
__device__ void flag_prefix(const int* flag, int n, int* pos, int* wtot) {
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  int carry = 0;
  for (int base = 0; base < n; base += NW * kWave) {
    const int i = base + threadIdx.x;
    const bool f = i < n && flag[i];
    const unsigned long long m = __ballot(f);
    const int before = __popcll(m & ((1ull << lane) - 1ull));
    if (lane == 0) wtot[w] = __popcll(m);
    __syncthreads();
    int wbase = carry, total = 0;
#pragma unroll
    for (int k = 0; k < NW; ++k) {
      wbase += k < w ? wtot[k] : 0;
      total += wtot[k];
    }
    if (i < n) pos[i] = wbase + before;
    carry += total;
    __syncthreads();
  }
}

// Selection of owner head `ou` by one workgroup of NW waves (`smem`: select_smem_bytes()).
// COH: write the selection with device-coherent stores (read by another workgroup of the launch).
template <class DT, int D, int NW, bool COH>
__device__ void select_block(const SelectArgs& a, int ou, unsigned char* smem) {
  constexpr int NT = NW * kWave;
  double* qsum = (double*)smem;            // [D]
  double* s1 = qsum + D;                   // [S]
  double* s2 = s1 + a.S;                   // [NC]
  unsigned long long* ck = (unsigned long long*)(s2 + a.NC);  // [max(S, NC)] composite keys
  uint32_t* key1 = (uint32_t*)(ck + max(a.S, a.NC));          // [S]
  uint32_t* key2 = key1 + a.S;             // [NC]
  int* rank1 = (int*)(key2 + a.NC);        // [S]
  int* rank2 = rank1 + a.S;                // [NC]
  int* cand = rank2 + a.NC;                // [NC]
  int* flag = cand + a.NC;                 // [max(S, NC)]
  int* pos = flag + max(a.S, a.NC);        // [max(S, NC)]
  __shared__ int wtot[NW];
  __shared__ int bnd[2];

  const int BH = a.B * a.Hkv;
  const int l = a.own.l[ou / BH], b = (ou / a.Hkv) % a.B, h = ou % a.Hkv;
  const size_t unit = (size_t)l * BH + ou % BH;
  const int abs_l = a.layer0 + l;
  const int G = a.Hq / a.Hkv;
  const int tid = threadIdx.x;

  const size_t q0 = (((size_t)l * a.B + b) * a.Hq + (size_t)h * G) * D;
  for (int i = tid; i < D; i += NT) {
    double acc = 0.0;
    for (int g = 0; g < G; ++g) acc += (double)load_elt<DT>(a.q, q0 + (size_t)g * D + i);
    qsum[i] = acc;
  }
  for (int i = tid; i < a.S; i += NT) rank1[i] = 0;
  for (int i = tid; i < a.NC; i += NT) rank2[i] = 0;
  __syncthreads();

  // level 1: super-cluster scores and top-k_super
  gemv_rows<D, NW>(a.scent + unit * a.S * D, nullptr, a.S, qsum, s1);
  __syncthreads();
  for (int i = tid; i < a.S; i += NT) {
    key1[i] = key_hi(s1[i]);
    ck[i] = rank_key(key1[i], i);
  }
  __syncthreads();
  rank_all<NT>(ck, a.S, rank1);
  __syncthreads();
  if (tid < 2) bnd[tid] = -1;
  __syncthreads();
  for (int i = tid; i < a.S; i += NT) {
    flag[i] = rank1[i] < a.k_super;
    if (rank1[i] == a.k_super - 1) bnd[0] = i;
    if (rank1[i] == a.k_super) bnd[1] = i;
  }
  __syncthreads();
  if (tid == 0) select_exact(s1, key1, rank1, a.S, a.k_super, bnd, flag);
  __syncthreads();
  // members of the kept super-clusters, ascending cluster id (invalid tail slots = -1)
  flag_prefix<NW>(flag, a.S, pos, wtot);
  for (int i = tid; i < a.S; i += NT) {
    if (!flag[i]) continue;
    const int p = pos[i];
    for (int m = 0; m < a.f; ++m) {
      const int c = i * a.f + m;
      cand[p * a.f + m] = c < a.C ? c : -1;
    }
  }
  __syncthreads();

  // level 2: scores of the candidates and top-k_clusters
  gemv_rows<D, NW>(a.cent + unit * a.C * D, cand, a.NC, qsum, s2);
  __syncthreads();
  for (int i = tid; i < a.NC; i += NT) {
    key2[i] = key_hi(s2[i]);
    ck[i] = rank_key(key2[i], i);
  }
  __syncthreads();
  rank_all<NT>(ck, a.NC, rank2);
  __syncthreads();
  if (tid < 2) bnd[tid] = -1;
  __syncthreads();
  for (int i = tid; i < a.NC; i += NT) {
    flag[i] = rank2[i] < a.k_clusters;
    if (rank2[i] == a.k_clusters - 1) bnd[0] = i;
    if (rank2[i] == a.k_clusters) bnd[1] = i;
  }
  __syncthreads();
  if (tid == 0) select_exact(s2, key2, rank2, a.NC, a.k_clusters, bnd, flag);
  __syncthreads();
  flag_prefix<NW>(flag, a.NC, pos, wtot);
  for (int i = tid; i < a.NC; i += NT) {
    if (!flag[i]) continue;
    const int p = pos[i];
    const float sc = (float)s2[i];
    // this layer and the following layers that share its selection
    for (int l2 = l; l2 < a.n_layers && owner_layer(a.layer0 + l2, a.period, a.start) == abs_l; ++l2) {
      const size_t o = (((size_t)l2 * a.B + b) * a.Hkv + h) * a.k_clusters + p;
      store_sel<COH>(a.sel + o, cand[i]);
      if (a.sel_score) a.sel_score[o] = sc;
    }
  }
}

// ---------------------------------------------------------------------------------------------
// One wave per owner head (many heads): the same two levels with wave-local synchronisation only,
// so thousands of heads progress independently. Each wave owns a private LDS region.
constexpr int kWaveMaxSuper = 256;        // limits of the wave variant's LDS region
constexpr int kWaveMaxCand = 256;

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

// scores[r] for r < n with one wave (rows of 4 lanes, as in gemv_rows).
template <int D>
__device__ void wave_gemv(const float* M, const int* idx, int n, const double (&qv)[D / 16][4], double* scores) {
  constexpr int STEPS = D / 16;
  constexpr int ROWS = kWave / 4;
  constexpr int PASS = 2;
  const int lane = threadIdx.x % kWave, rq = lane >> 2, qk = lane & 3;
  for (int r0 = 0; r0 < n; r0 += ROWS * PASS) {
    float4 x[PASS][STEPS];
    bool valid[PASS];
#pragma unroll
    for (int p = 0; p < PASS; ++p) {
      const int r = r0 + p * ROWS + rq;
      const int row = r < n ? (idx ? idx[r] : r) : -1;
      valid[p] = row >= 0;
      const float* src = M + (size_t)(valid[p] ? row : 0) * D + qk * 4;
#pragma unroll
      for (int c = 0; c < STEPS; ++c) x[p][c] = *(const float4*)(src + c * 16);
    }
#pragma unroll
    for (int p = 0; p < PASS; ++p) {
      double acc = 0.0;
#pragma unroll
      for (int c = 0; c < STEPS; ++c)
        acc += qv[c][0] * (double)x[p][c].x + qv[c][1] * (double)x[p][c].y + qv[c][2] * (double)x[p][c].z +
               qv[c][3] * (double)x[p][c].w;
      acc = group_sum<4>(acc);
      const int r = r0 + p * ROWS + rq;
      if (qk == 0 && r < n) scores[r] = valid[p] ? acc : -INFINITY;
    }
  }
  wave_sync();
}

// flag[i] = (rank of i < k) with composite keys and the exact boundary repair, one wave.
__device__ void wave_topk_flags(const double* sc, uint32_t* img, unsigned long long* ck, int* rank, int n, int k,
                                int* flag) {
  const int lane = threadIdx.x % kWave;
  for (int i = lane; i < n; i += kWave) {
    img[i] = key_hi(sc[i]);
    ck[i] = rank_key(img[i], i);
  }
  wave_sync();
  int bnd[2] = {-1, -1};
  for (int i = lane; i < n; i += kWave) {
    rank[i] = count_above(ck, 0, n, ck[i]);
    flag[i] = rank[i] < k;
    if (rank[i] == k - 1) bnd[0] = i;
    if (rank[i] == k) bnd[1] = i;
  }
  // each boundary entry is held by exactly one lane: a max-reduction publishes it to all lanes
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    bnd[0] = max(bnd[0], __shfl_xor(bnd[0], o));
    bnd[1] = max(bnd[1], __shfl_xor(bnd[1], o));
  }
  wave_sync();
  if (lane == 0) select_exact(sc, img, rank, n, k, bnd, flag);
  wave_sync();
}

// pos[i] = number of set flags before i, one wave.
__device__ void wave_prefix(const int* flag, int n, int* pos) {
  const int lane = threadIdx.x % kWave;
  int carry = 0;
  for (int base = 0; base < n; base += kWave) {
    const int i = base + lane;
    const unsigned long long m = __ballot(i < n && flag[i]);
    if (i < n) pos[i] = carry + __popcll(m & ((1ull << lane) - 1ull));
    carry += __popcll(m);
  }
  wave_sync();
}

__host__ __device__ inline size_t wave_region_bytes(int S, int NC) {
  const int m = S > NC ? S : NC;
  const size_t region = (size_t)(S + NC + m) * sizeof(double) + (size_t)(NC + 4 * m) * sizeof(int);
  return (region + 15) & ~(size_t)15;
}

// Selection of owner heads ou0 + w, one per wave w (`smem`: waves x wave_region_bytes()).
template <class DT, int D, bool COH>
__device__ void select_waves(const SelectArgs& a, int ou0, unsigned char* smem) {
  constexpr int STEPS = D / 16;
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  const int BH = a.B * a.Hkv;
  const int ou = ou0 + w;  // (owner index * B + b) * Hkv + h
  if (ou >= a.own.n * BH) return;
  // wave-private LDS region
  const int m = a.S > a.NC ? a.S : a.NC;
  unsigned char* base = smem + (size_t)w * wave_region_bytes(a.S, a.NC);
  double* s1 = (double*)base;
  double* s2 = s1 + a.S;
  unsigned long long* ck = (unsigned long long*)(s2 + a.NC);
  int* cand = (int*)(ck + m);
  uint32_t* img = (uint32_t*)(cand + a.NC);
  int* rank = (int*)(img + m);
  int* flag = rank + m;
  int* pos = flag + m;

  const int l = a.own.l[ou / BH], b = (ou / a.Hkv) % a.B, h = ou % a.Hkv;
  const size_t unit = (size_t)l * BH + ou % BH;
  const int abs_l = a.layer0 + l;
  const int G = a.Hq / a.Hkv;
  const int qk = lane & 3;
  const size_t q0 = (((size_t)l * a.B + b) * a.Hq + (size_t)h * G) * D;
  double qv[STEPS][4];
#pragma unroll
  for (int c = 0; c < STEPS; ++c)
#pragma unroll
    for (int e = 0; e < 4; ++e) qv[c][e] = 0.0;
  for (int g = 0; g < G; ++g) {
    float x[STEPS][4];
#pragma unroll
    for (int c = 0; c < STEPS; ++c) load4<DT>(a.q, q0 + (size_t)g * D + c * 16 + qk * 4, x[c]);
#pragma unroll
    for (int c = 0; c < STEPS; ++c)
#pragma unroll
      for (int e = 0; e < 4; ++e) qv[c][e] += (double)x[c][e];
  }

  wave_gemv<D>(a.scent + unit * a.S * D, nullptr, a.S, qv, s1);
  wave_topk_flags(s1, img, ck, rank, a.S, a.k_super, flag);
  wave_prefix(flag, a.S, pos);
  for (int i = lane; i < a.S; i += kWave) {
    if (!flag[i]) continue;
    for (int mm = 0; mm < a.f; ++mm) {
      const int c = i * a.f + mm;
      cand[pos[i] * a.f + mm] = c < a.C ? c : -1;
    }
  }
  wave_sync();
  wave_gemv<D>(a.cent + unit * a.C * D, cand, a.NC, qv, s2);
  wave_topk_flags(s2, img, ck, rank, a.NC, a.k_clusters, flag);
  wave_prefix(flag, a.NC, pos);
  for (int i = lane; i < a.NC; i += kWave) {
    if (!flag[i]) continue;
    const float sc = (float)s2[i];
    for (int l2 = l; l2 < a.n_layers && owner_layer(a.layer0 + l2, a.period, a.start) == abs_l; ++l2) {
      const size_t o = (((size_t)l2 * a.B + b) * a.Hkv + h) * a.k_clusters + pos[i];
      store_sel<COH>(a.sel + o, cand[i]);
      if (a.sel_score) a.sel_score[o] = sc;
    }
  }
}

inline size_t select_smem_bytes_dev(int D, int S, int NC) {
  const int m = S > NC ? S : NC;
  return (size_t)(D + S + NC + m) * sizeof(double) + (size_t)(2 * S + 3 * NC + 2 * m) * sizeof(int);
}

}  // namespace dev
}  // namespace mpc
