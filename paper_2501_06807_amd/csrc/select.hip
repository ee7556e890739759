// Query-aware two-level cluster selection with cross-layer index sharing, gfx950.
//
// One workgroup per owner (layer, sequence, kv head). Scores are GEMVs of the summed group query
// against fp32 representatives, accumulated in fp64 (every product of a 16-bit or fp32 input with
// an fp32 representative is exact in fp64, so only the summation order differs from a sequential
// sum). Ranking is by (score desc, index asc): each candidate counts the candidates that beat it,
// on 32-bit key images with an exact fp64 recount for key ties; output slots come from wave-ballot
// prefix counts. Only owner heads get a workgroup.
#include "select_dev.h"

namespace mpc {
namespace {

constexpr int kWaveHeads = 4;  // heads (waves) per workgroup of the standalone wave variant

template <class DT, int D, int NW>
__global__ __launch_bounds__(NW* kWave) void k_select(SelectArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  dev::select_block<DT, D, NW, false>(a, blockIdx.x, smem);
}

template <class DT, int D>
__global__ __launch_bounds__(kWaveHeads* kWave) void k_select_wave(SelectArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  dev::select_waves<DT, D, false>(a, blockIdx.x * kWaveHeads, smem);
}

template <class DT>
hipError_t launch_wave(const SelectArgs& a, int D, hipStream_t st) {
  const int units = a.own.n * a.B * a.Hkv;
  const dim3 grid((units + kWaveHeads - 1) / kWaveHeads);
  const size_t smem = kWaveHeads * dev::wave_region_bytes(D, a.S, a.NC);
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

// At most one owner head per CU: one 8-wave workgroup per head shortens each head's chain. More
// heads: 4-wave workgroups, so that all of them are resident at once. Many heads (at least two
// per CU): one wave per head.
template <class DT>
hipError_t launch_dt(const SelectArgs& a, int D, size_t smem, hipStream_t st) {
  const int units = a.own.n * a.B * a.Hkv;
  if (units >= 512 && a.S <= dev::kWaveMaxSuper && a.NC <= dev::kWaveMaxCand && (D == 64 || D == 128))
    return launch_wave<DT>(a, D, st);
  if (units <= kNumCU) return launch_dt_nw<DT, 8>(a, D, units, smem, st);
  return launch_dt_nw<DT, 4>(a, D, units, smem, st);
}

}  // namespace

size_t select_smem_bytes(int D, int S, int NC) { return dev::select_smem_bytes_dev(D, S, NC); }

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
