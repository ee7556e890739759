// Query-aware two-level cluster selection with cross-layer index sharing, gfx950.
//
// One workgroup per owner (layer, sequence, kv head). Scores are GEMVs of the summed group query
// against fp32 representatives, accumulated in fp64 (every product of a 16-bit or fp32 input with
// an fp32 representative is exact in fp64, so only the summation order differs from a sequential
// sum). Ranking is by (score desc, index asc): each candidate counts the candidates that beat it,
// which for the few hundred candidates of a head is one LDS pass per lane.
#include "select.h"

namespace mpc {
namespace {

constexpr int kSelThreads = 256;
constexpr int kSelWaves = kSelThreads / kWave;

// scores[r] = sum_i qsum[i] * M[idx(r)][i] for r < n; rows with idx < 0 score -inf.
template <int D>
__device__ void gemv_rows(const float* M, const int* idx, int n, const double* qsum, double* scores) {
  constexpr int PER = D / kWave;  // 1 or 2 floats per lane
  const int lane = threadIdx.x % kWave, w = threadIdx.x / kWave;
  double qv[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) qv[e] = qsum[lane * PER + e];
  constexpr int UN = 4;
  for (int r0 = w * UN; r0 < n; r0 += kSelWaves * UN) {
    float x[UN][PER];
    bool valid[UN];
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      const int r = r0 + u;
      const int row = r < n ? (idx ? idx[r] : r) : -1;
      valid[u] = row >= 0;
      const float* p = M + (size_t)(valid[u] ? row : 0) * D + lane * PER;
#pragma unroll
      for (int e = 0; e < PER; ++e) x[u][e] = p[e];
    }
#pragma unroll
    for (int u = 0; u < UN; ++u) {
      double acc = 0.0;
#pragma unroll
      for (int e = 0; e < PER; ++e) acc += qv[e] * (double)x[u][e];
      acc = wave_sum(acc);
      if (lane == 0 && r0 + u < n) scores[r0 + u] = valid[u] ? acc : -INFINITY;
    }
  }
}

// beats(j over i): score larger, or equal with lower index.
__device__ __forceinline__ bool beats(double sj, int j, double si, int i) {
  return sj > si || (sj == si && j < i);
}

template <class DT, int D>
__global__ __launch_bounds__(kSelThreads) void k_select(SelectArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  double* qsum = (double*)smem;                  // [D]
  double* s1 = qsum + D;                         // [S]
  double* s2 = s1 + a.S;                         // [NC]
  int* cand = (int*)(s2 + a.NC);                 // [NC]
  int* flag1 = cand + a.NC;                      // [S]
  int* flag2 = flag1 + a.S;                      // [NC]

  const int unit = blockIdx.x;
  const int BH = a.B * a.Hkv;
  const int l = unit / BH, b = (unit / a.Hkv) % a.B, h = unit % a.Hkv;
  const int abs_l = a.layer0 + l;
  if (owner_layer(abs_l, a.period, a.start) != abs_l) return;
  const int G = a.Hq / a.Hkv;
  const int tid = threadIdx.x;

  const size_t q0 = (((size_t)l * a.B + b) * a.Hq + (size_t)h * G) * D;
  for (int i = tid; i < D; i += kSelThreads) {
    double acc = 0.0;
    for (int g = 0; g < G; ++g) acc += (double)load_elt<DT>(a.q, q0 + (size_t)g * D + i);
    qsum[i] = acc;
  }
  __syncthreads();

  // level 1: super-cluster scores and top-k_super
  gemv_rows<D>(a.scent + (size_t)unit * a.S * D, nullptr, a.S, qsum, s1);
  __syncthreads();
  for (int i = tid; i < a.S; i += kSelThreads) {
    const double si = s1[i];
    int r = 0;
    for (int j = 0; j < a.S; ++j) r += beats(s1[j], j, si, i);
    flag1[i] = r < a.k_super;
  }
  __syncthreads();
  // members of the kept super-clusters, ascending cluster id (invalid tail slots = -1)
  for (int i = tid; i < a.S; i += kSelThreads) {
    if (!flag1[i]) continue;
    int p = 0;
    for (int j = 0; j < i; ++j) p += flag1[j];
    for (int m = 0; m < a.f; ++m) {
      const int c = i * a.f + m;
      cand[p * a.f + m] = c < a.C ? c : -1;
    }
  }
  __syncthreads();

  // level 2: scores of the candidates and top-k_clusters
  gemv_rows<D>(a.cent + (size_t)unit * a.C * D, cand, a.NC, qsum, s2);
  __syncthreads();
  for (int i = tid; i < a.NC; i += kSelThreads) {
    int r = a.k_clusters;
    if (cand[i] >= 0) {
      const double si = s2[i];
      r = 0;
      for (int j = 0; j < a.NC; ++j) r += beats(s2[j], j, si, i);
    }
    flag2[i] = r < a.k_clusters;
  }
  __syncthreads();
  for (int i = tid; i < a.NC; i += kSelThreads) {
    if (!flag2[i]) continue;
    int p = 0;
    for (int j = 0; j < i; ++j) p += flag2[j];
    const float sc = (float)s2[i];
    // this layer and the following layers that share its selection
    for (int l2 = l; l2 < a.n_layers && owner_layer(a.layer0 + l2, a.period, a.start) == abs_l; ++l2) {
      const size_t o = (((size_t)l2 * a.B + b) * a.Hkv + h) * a.k_clusters + p;
      a.sel[o] = cand[i];
      if (a.sel_score) a.sel_score[o] = sc;
    }
  }
}

template <class DT>
hipError_t launch_dt(const SelectArgs& a, int D, int units, size_t smem, hipStream_t st) {
  if (D == 64) {
    hipLaunchKernelGGL((k_select<DT, 64>), dim3(units), dim3(kSelThreads), smem, st, a);
  } else if (D == 128) {
    hipLaunchKernelGGL((k_select<DT, 128>), dim3(units), dim3(kSelThreads), smem, st, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

size_t select_smem_bytes(int D, int S, int NC) {
  return (size_t)(D + S + NC) * sizeof(double) + (size_t)(NC + S + NC) * sizeof(int);
}

hipError_t launch_select(const SelectArgs& a, int dtype, int D, hipStream_t st) {
  const int units = a.n_layers * a.B * a.Hkv;
  const size_t smem = select_smem_bytes(D, a.S, a.NC);
  switch (dtype) {
    case MPC_FP32: return launch_dt<F32>(a, D, units, smem, st);
    case MPC_FP16: return launch_dt<F16>(a, D, units, smem, st);
    case MPC_BF16: return launch_dt<BF16>(a, D, units, smem, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace mpc
