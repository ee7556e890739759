// Sparse decode attention over the selected clusters (gather + online softmax), gfx950.
//
// One work unit = (layer, sequence, kv head). Its token list is the concatenation of the
// selected clusters' rows of the kept cache. A unit may be split over several workgroups
// (split-K); each writes an (m, l, acc) partial and the last one to finish merges them.
//
// Lane layout: a K/V row of d elements is read as 16-byte vectors by LPR consecutive lanes, so a
// wave reads RPW = 64 / LPR rows per load instruction, fully coalesced. The G query heads of the
// group are served from the same loaded rows. Scores are kept in log2 units (q is pre-scaled by
// sm_scale * log2 e) so the softmax uses the hardware exp2. V rows are loaded with the
// non-temporal hint; K rows too when the decode step's working set passes the memory-side cache
// (DecodeArgs::stream_k, a template variant).
#include "decode_dev.h"

namespace mpc {
namespace {

template <class DT, int D, int G, int NW, int U, bool STREAM_K>
__global__ __launch_bounds__(NW* kWave) void k_sparse_decode(DecodeArgs a) {
  dev::attend<DT, D, G, NW, U, false, STREAM_K>(a, blockIdx.x / a.splits, blockIdx.x % a.splits);
}

template <class DT, int D, int G>
hipError_t launch_dt_d_g(const DecodeArgs& a, int units, const DecodePlan& p, hipStream_t st) {
  (void)p;
  if (a.stream_k)
    hipLaunchKernelGGL((k_sparse_decode<DT, D, G, 8, 4, true>), dim3(units * a.splits), dim3(8 * kWave), 0, st, a);
  else
    hipLaunchKernelGGL((k_sparse_decode<DT, D, G, 8, 4, false>), dim3(units * a.splits), dim3(8 * kWave), 0, st, a);
  return hipGetLastError();
}

template <class DT, int D>
hipError_t launch_dt_d(const DecodeArgs& a, int G, int units, const DecodePlan& p, hipStream_t st) {
  switch (G) {
    case 1: return launch_dt_d_g<DT, D, 1>(a, units, p, st);
    case 2: return launch_dt_d_g<DT, D, 2>(a, units, p, st);
    case 4: return launch_dt_d_g<DT, D, 4>(a, units, p, st);
    case 8: return launch_dt_d_g<DT, D, 8>(a, units, p, st);
  }
  return hipErrorInvalidValue;
}

template <class DT>
hipError_t launch_dt(const DecodeArgs& a, int D, int G, int units, const DecodePlan& p, hipStream_t st) {
  if (D == 64) return launch_dt_d<DT, 64>(a, G, units, p, st);
  if (D == 128) return launch_dt_d<DT, 128>(a, G, units, p, st);
  return hipErrorInvalidValue;
}

}  // namespace

DecodePlan decode_plan(int units, int n_slot, int D, int elt) {
  // One 8-wave workgroup per unit when there are at least as many units as CUs; otherwise the
  // token list of each unit is split over several workgroups (about two per CU).
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

hipError_t launch_sparse_decode(const DecodeArgs& a, int dtype, int D, int G, int units, const DecodePlan& p,
                                hipStream_t st) {
  switch (dtype) {
    case MPC_FP32: return launch_dt<F32>(a, D, G, units, p, st);
    case MPC_FP16: return launch_dt<F16>(a, D, G, units, p, st);
    case MPC_BF16: return launch_dt<BF16>(a, D, G, units, p, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace mpc
