// Sparse decode attention over the selected clusters (gather + online softmax), gfx950.
//
// One work unit = (layer, sequence, kv head). Its token list is the concatenation of the
// selected clusters' rows of the kept cache. A unit may be split over several workgroups
// (split-K); each writes an (m, l, acc) partial and a second launch merges them.
//
// Lane layout: a K/V row of d elements is read as 16-byte vectors by LPR consecutive lanes, so a
// wave reads RPW = 64 / LPR rows per load instruction, fully coalesced. The G query heads of the
// group are served from the same loaded rows. Scores are kept in log2 units (q is pre-scaled by
// sm_scale * log2 e) so the softmax uses the hardware exp2.
#include "decode_dev.h"

namespace mpc {
namespace {

template <class DT, int D, int G, int NW, int U>
__global__ __launch_bounds__(NW* kWave) void k_sparse_decode(DecodeArgs a) {
  dev::attend_unit<DT, D, G, NW, U, false>(a, blockIdx.x / a.splits, blockIdx.x % a.splits);
}

// Split-K merge: one workgroup per (unit, q-head of the group) combines the splits' partials.
// Runs as its own launch, so the partials are visible without any cross-workgroup fence.
template <class DT, int D, int G>
__global__ __launch_bounds__(D) void k_merge(DecodeArgs a) {
  const int unit = blockIdx.x / G, g = blockIdx.x % G, dim = threadIdx.x;
  const size_t q_row = (size_t)(unit / a.Hkv) * a.Hq + (size_t)(unit % a.Hkv) * G + g;
  const float* p0 = a.part + ((size_t)unit * a.splits * G + g) * (D + 2);
  const size_t stride = (size_t)G * (D + 2);
  float M = -1e30f;
  for (int i = 0; i < a.splits; ++i) M = fmaxf(M, p0[i * stride + D]);
  float L = 0.f, O = 0.f;
  for (int i = 0; i < a.splits; ++i) {
    const float* p = p0 + i * stride;
    const float r = fast_exp2(p[D] - M);
    L += p[D + 1] * r;
    O += p[dim] * r;
  }
  store_elt<DT>(a.out, q_row * D + dim, O / L);
  if (dim == 0 && a.lse) a.lse[q_row] = (M + __log2f(L)) * 0.69314718055994531f;
}

template <class DT, int D, int G>
hipError_t launch_dt_d_g(const DecodeArgs& a, int units, int waves, hipStream_t st) {
  if (waves == 16)
    hipLaunchKernelGGL((k_sparse_decode<DT, D, G, 16, 4>), dim3(units * a.splits), dim3(16 * kWave), 0, st, a);
  else
    hipLaunchKernelGGL((k_sparse_decode<DT, D, G, 8, 4>), dim3(units * a.splits), dim3(8 * kWave), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  hipLaunchKernelGGL((k_merge<DT, D, G>), dim3(units * G), dim3(D), 0, st, a);
  return hipGetLastError();
}

template <class DT, int D>
hipError_t launch_dt_d(const DecodeArgs& a, int G, int units, int waves, hipStream_t st) {
  switch (G) {
    case 1: return launch_dt_d_g<DT, D, 1>(a, units, waves, st);
    case 2: return launch_dt_d_g<DT, D, 2>(a, units, waves, st);
    case 4: return launch_dt_d_g<DT, D, 4>(a, units, waves, st);
    case 8: return launch_dt_d_g<DT, D, 8>(a, units, waves, st);
  }
  return hipErrorInvalidValue;
}

template <class DT>
hipError_t launch_dt(const DecodeArgs& a, int D, int G, int units, int waves, hipStream_t st) {
  if (D == 64) return launch_dt_d<DT, 64>(a, G, units, waves, st);
  if (D == 128) return launch_dt_d<DT, 128>(a, G, units, waves, st);
  return hipErrorInvalidValue;
}

}  // namespace

DecodePlan decode_plan(int units, int n_slot, int D, int elt) {
  // One 8-wave workgroup per unit when there are at least as many units as CUs; otherwise the
  // token list of each unit is split over several workgroups.
  DecodePlan p;
  p.waves = 8;
  p.splits = 1;
  if (units < kNumCU) {
    const int lpr = D * elt / 16;
    const int rows_per_pass = p.waves * (kWave / lpr);
    int max_splits = n_slot / rows_per_pass;
    if (max_splits < 1) max_splits = 1;
    p.splits = (2 * kNumCU + units - 1) / units;
    if (p.splits > max_splits) p.splits = max_splits;
    if (p.splits > kMaxSplits) p.splits = kMaxSplits;
  }
  return p;
}

hipError_t launch_sparse_decode(const DecodeArgs& a, int dtype, int D, int G, int units, int waves,
                                hipStream_t st) {
  switch (dtype) {
    case MPC_FP32: return launch_dt<F32>(a, D, G, units, waves, st);
    case MPC_FP16: return launch_dt<F16>(a, D, G, units, waves, st);
    case MPC_BF16: return launch_dt<BF16>(a, D, G, units, waves, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace mpc
