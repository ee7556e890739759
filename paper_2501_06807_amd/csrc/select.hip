// Query-aware two-level cluster selection with cross-layer index sharing, gfx950.
//
// One workgroup per owner (layer, sequence, kv head). Scores are GEMVs of the summed group query
// against fp32 representatives, accumulated in fp64 (every product of a 16-bit or fp32 input with
// an fp32 representative is exact in fp64, so only the summation order differs from a sequential
// sum). Ranking is by (score desc, index asc): each candidate counts the candidates that beat it,
// on 32-bit key images with an exact fp64 recount for key ties; output slots come from wave-ballot
// prefix counts. Only owner heads get a workgroup.
#include "select.h"

namespace mpc {
namespace {

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

// rank[i] = number of entries that beat entry i (larger score, or equal score and lower index).
// All threads cooperate: for n below the thread count each entry's comparisons are split over
// several threads and the counts meet in LDS. The hot loop compares the 32-bit key images; only
// an entry whose key ties another's repeats the comparisons in fp64 for those entries.
template <int NT>
__device__ void rank_all(const double* sc, const uint32_t* key, int n, int* rank) {
  const int parts = n < NT ? NT / n : 1;
  for (int t = threadIdx.x; t < n * parts; t += NT) {
    const int i = t % n, part = t / n;
    const int j0 = part * n / parts, j1 = (part + 1) * n / parts;
    const uint32_t ki = key[i];
    int gt = 0, eq = 0, j = j0;
    for (; j + 16 <= j1; j += 16) {
      uint32_t v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = key[j + u];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        gt += v[u] > ki;
        eq += v[u] == ki;
      }
    }
    for (; j < j1; ++j) {
      gt += key[j] > ki;
      eq += key[j] == ki;
    }
    if (eq > (i >= j0 && i < j1 ? 1 : 0)) {
      const double si = sc[i];
      for (j = j0; j < j1; ++j)
        if (j != i && key[j] == ki) gt += (sc[j] > si) | ((sc[j] == si) & (j < i));
    }
    atomicAdd(&rank[i], gt);
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

template <class DT, int D, int NW>
__global__ __launch_bounds__(NW* kWave) void k_select(SelectArgs a) {
  constexpr int NT = NW * kWave;
  extern __shared__ __align__(16) unsigned char smem[];
  double* qsum = (double*)smem;            // [D]
  double* s1 = qsum + D;                   // [S]
  double* s2 = s1 + a.S;                   // [NC]
  uint32_t* key1 = (uint32_t*)(s2 + a.NC); // [S]
  uint32_t* key2 = key1 + a.S;             // [NC]
  int* rank1 = (int*)(key2 + a.NC);        // [S]
  int* rank2 = rank1 + a.S;                // [NC]
  int* cand = rank2 + a.NC;                // [NC]
  int* flag = cand + a.NC;                 // [max(S, NC)]
  int* pos = flag + max(a.S, a.NC);        // [max(S, NC)]
  __shared__ int wtot[NW];

  const int BH = a.B * a.Hkv;
  const int ou = blockIdx.x;  // (owner index * B + b) * Hkv + h
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
  for (int i = tid; i < a.S; i += NT) key1[i] = key_hi(s1[i]);
  __syncthreads();
  rank_all<NT>(s1, key1, a.S, rank1);
  __syncthreads();
  for (int i = tid; i < a.S; i += NT) flag[i] = rank1[i] < a.k_super;
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
  for (int i = tid; i < a.NC; i += NT) key2[i] = key_hi(s2[i]);
  __syncthreads();
  rank_all<NT>(s2, key2, a.NC, rank2);
  __syncthreads();
  for (int i = tid; i < a.NC; i += NT) flag[i] = cand[i] >= 0 && rank2[i] < a.k_clusters;
  __syncthreads();
  flag_prefix<NW>(flag, a.NC, pos, wtot);
  for (int i = tid; i < a.NC; i += NT) {
    if (!flag[i]) continue;
    const int p = pos[i];
    const float sc = (float)s2[i];
    // this layer and the following layers that share its selection
    for (int l2 = l; l2 < a.n_layers && owner_layer(a.layer0 + l2, a.period, a.start) == abs_l; ++l2) {
      const size_t o = (((size_t)l2 * a.B + b) * a.Hkv + h) * a.k_clusters + p;
      a.sel[o] = cand[i];
      if (a.sel_score) a.sel_score[o] = sc;
    }
  }
}

// ---------------------------------------------------------------------------------------------
// One wave per owner head (many heads): the same two levels with wave-local synchronisation only,
// so thousands of heads progress independently. Each wave owns a private LDS region.
constexpr int kWaveHeads = 4;             // heads (waves) per workgroup
constexpr int kWaveMaxSuper = 256;        // limits of the wave variant's LDS region
constexpr int kWaveMaxCand = 512;

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

// flag[i] = (entry i valid) && (rank of i < k); ranks on key images with exact fp64 tie repair.
__device__ void wave_topk_flags(const double* sc, uint32_t* key, const int* valid_idx, int n, int k, int* flag) {
  const int lane = threadIdx.x % kWave;
  for (int i = lane; i < n; i += kWave) key[i] = key_hi(sc[i]);
  wave_sync();
  for (int i = lane; i < n; i += kWave) {
    const uint32_t ki = key[i];
    int gt = 0, eq = 0, j = 0;
    for (; j + 16 <= n; j += 16) {
      uint32_t v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = key[j + u];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        gt += v[u] > ki;
        eq += v[u] == ki;
      }
    }
    for (; j < n; ++j) {
      gt += key[j] > ki;
      eq += key[j] == ki;
    }
    if (eq > 1) {
      const double si = sc[i];
      for (j = 0; j < n; ++j)
        if (j != i && key[j] == ki) gt += (sc[j] > si) | ((sc[j] == si) & (j < i));
    }
    flag[i] = (!valid_idx || valid_idx[i] >= 0) && gt < k;
  }
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

template <class DT, int D>
__global__ __launch_bounds__(kWaveHeads* kWave) void k_select_wave(SelectArgs a) {
  constexpr int STEPS = D / 16;
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  const int BH = a.B * a.Hkv;
  const int ou = blockIdx.x * kWaveHeads + w;  // (owner index * B + b) * Hkv + h
  if (ou >= a.own.n * BH) return;
  // wave-private LDS region
  const int m = a.S > a.NC ? a.S : a.NC;
  const size_t region = (size_t)(a.S + a.NC) * sizeof(double) + (size_t)(a.NC + 3 * m) * sizeof(int);
  unsigned char* base = smem + (size_t)w * ((region + 15) & ~(size_t)15);
  double* s1 = (double*)base;
  double* s2 = s1 + a.S;
  int* cand = (int*)(s2 + a.NC);
  uint32_t* key = (uint32_t*)(cand + a.NC);
  int* flag = (int*)(key + m);
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
    for (int e = 0; e < 4; ++e) {
      double acc = 0.0;
      for (int g = 0; g < G; ++g) acc += (double)load_elt<DT>(a.q, q0 + (size_t)g * D + c * 16 + qk * 4 + e);
      qv[c][e] = acc;
    }

  wave_gemv<D>(a.scent + unit * a.S * D, nullptr, a.S, qv, s1);
  wave_topk_flags(s1, key, nullptr, a.S, a.k_super, flag);
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
  wave_topk_flags(s2, key, cand, a.NC, a.k_clusters, flag);
  wave_prefix(flag, a.NC, pos);
  for (int i = lane; i < a.NC; i += kWave) {
    if (!flag[i]) continue;
    const float sc = (float)s2[i];
    for (int l2 = l; l2 < a.n_layers && owner_layer(a.layer0 + l2, a.period, a.start) == abs_l; ++l2) {
      const size_t o = (((size_t)l2 * a.B + b) * a.Hkv + h) * a.k_clusters + pos[i];
      a.sel[o] = cand[i];
      if (a.sel_score) a.sel_score[o] = sc;
    }
  }
}

size_t wave_region_bytes(int S, int NC) {
  const int m = S > NC ? S : NC;
  const size_t region = (size_t)(S + NC) * sizeof(double) + (size_t)(NC + 3 * m) * sizeof(int);
  return (region + 15) & ~(size_t)15;
}

template <class DT>
hipError_t launch_wave(const SelectArgs& a, int D, hipStream_t st) {
  const int units = a.own.n * a.B * a.Hkv;
  const dim3 grid((units + kWaveHeads - 1) / kWaveHeads);
  const size_t smem = kWaveHeads * wave_region_bytes(a.S, a.NC);
  if (D == 64)
    hipLaunchKernelGGL((k_select_wave<DT, 64>), grid, dim3(kWaveHeads * kWave), smem, st, a);
  else
    hipLaunchKernelGGL((k_select_wave<DT, 128>), grid, dim3(kWaveHeads * kWave), smem, st, a);
  return hipGetLastError();
}

template <class DT, int NW>
hipError_t launch_dt_nw(const SelectArgs& a, int D, int units, size_t smem, hipStream_t st) {
  if (D == 64) {
    hipLaunchKernelGGL((k_select<DT, 64, NW>), dim3(units), dim3(NW * kWave), smem, st, a);
  } else if (D == 128) {
    hipLaunchKernelGGL((k_select<DT, 128, NW>), dim3(units), dim3(NW * kWave), smem, st, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// Few owner heads: one 8-wave workgroup per head shortens each head's chain. Many heads (at least
// two per CU): one wave per head, so every head is in flight at once.
template <class DT>
hipError_t launch_dt(const SelectArgs& a, int D, size_t smem, hipStream_t st) {
  const int units = a.own.n * a.B * a.Hkv;
  if (units >= 512 && a.S <= kWaveMaxSuper && a.NC <= kWaveMaxCand && (D == 64 || D == 128))
    return launch_wave<DT>(a, D, st);
  if (units < 512) return launch_dt_nw<DT, 8>(a, D, units, smem, st);
  return launch_dt_nw<DT, 4>(a, D, units, smem, st);
}

}  // namespace

size_t select_smem_bytes(int D, int S, int NC) {
  const int m = S > NC ? S : NC;
  return (size_t)(D + S + NC) * sizeof(double) + (size_t)(2 * S + 3 * NC + 2 * m) * sizeof(int);
}

hipError_t launch_select(const SelectArgs& a, int dtype, int D, hipStream_t st) {
  const size_t smem = select_smem_bytes(D, a.S, a.NC);
  switch (dtype) {
    case MPC_FP32: return launch_dt<F32>(a, D, smem, st);
    case MPC_FP16: return launch_dt<F16>(a, D, smem, st);
    case MPC_BF16: return launch_dt<BF16>(a, D, smem, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace mpc
