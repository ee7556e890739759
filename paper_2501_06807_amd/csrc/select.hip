// Query-aware two-level cluster selection with cross-layer index sharing, gfx950.
//
// One workgroup (or one wave) per owner (layer, sequence, selection unit), a unit being a kv head
// (its q-heads share one selection) or a single q-head. Scores are GEMVs against fp32
// representatives accumulated in fp64: the summed group query against one row (linear form,
// average), the G queries against the r^max / r^min rows (max-product bound), or, for the maximum
// over the group, each query on its own followed by the maximum. Every product of
// a 16-bit or fp32 input with an fp32 representative is exact in fp64, so only the summation order
// differs from a sequential sum. Ranking is by (score desc, index asc) on unique composite integer
// keys with an exact fp64 re-rank of a tied boundary group; output positions are counts over the
// selected ids. Only owner heads get work.
#include "select_dev.h"

namespace mpc {
namespace {

constexpr int kWaveHeads = 4;     // heads (waves) per workgroup of the wave variant, by default
constexpr int kWaveHeadsMax = 8;  // and at most (when that spreads the heads evenly over the CUs)

template <class DT, int D, int NW, bool MP, bool GMAX>
__global__ __launch_bounds__(NW* kWave) void k_select(SelectArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  dev::select_block<DT, D, NW, false, 2, MP, true, GMAX>(a, blockIdx.x, smem);
}

template <class DT, int D, bool MP, bool GMAX>
__global__ __launch_bounds__(kWaveHeadsMax* kWave) void k_select_wave(SelectArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  dev::select_waves<DT, D, false, MP, GMAX>(a, blockIdx.x * (blockDim.x / kWave), smem);
}

// Heads per workgroup: one workgroup per CU when the heads fit at most kWaveHeadsMax per CU (every
// CU then runs the same number of heads; with a fixed 4 per workgroup, 1280 heads made 320
// workgroups and a quarter of the CUs ran two), else 4.
int wave_heads(int units) {
  const int per_cu = (units + kNumCU - 1) / kNumCU;
  return per_cu > kWaveHeads && per_cu <= kWaveHeadsMax ? per_cu : kWaveHeads;
}

template <class DT, int D, bool MP, bool GMAX>
void launch_wave(const SelectArgs& a, int hpw, hipStream_t st) {
  const int units = a.own.n * a.B * a.Hsel;
  const dim3 grid((units + hpw - 1) / hpw);
  const size_t smem = hpw * dev::wave_region_bytes(D, a.S, a.NC, select_query_rows(a));
  hipLaunchKernelGGL((k_select_wave<DT, D, MP, GMAX>), grid, dim3(hpw * kWave), smem, st, a);
}

template <class DT, int D, bool MP, bool GMAX>
void launch_block(const SelectArgs& a, int units, int nw, hipStream_t st) {
  const size_t smem = select_smem_bytes(D, a.S, a.NC, select_query_rows(a));
  if (nw == 8)
    hipLaunchKernelGGL((k_select<DT, D, 8, MP, GMAX>), dim3(units), dim3(8 * kWave), smem, st, a);
  else
    hipLaunchKernelGGL((k_select<DT, D, 4, MP, GMAX>), dim3(units), dim3(4 * kWave), smem, st, a);
}

// At most one owner head per CU: one 8-wave workgroup per head shortens each head's chain. More
// heads: 4-wave workgroups, so that all of them are resident at once. Many heads (at least two
// per CU): one wave per head.
template <class DT, int D, bool MP, bool GMAX>
void launch_plan(const SelectArgs& a, hipStream_t st) {
  const int units = a.own.n * a.B * a.Hsel;
  const int hpw = wave_heads(units);
  if (units >= 512 && a.S <= dev::kWaveMaxSuper && a.NC <= dev::kWaveMaxCand &&
      hpw * dev::wave_region_bytes(D, a.S, a.NC, select_query_rows(a)) <= kMaxLds)
    launch_wave<DT, D, MP, GMAX>(a, hpw, st);
  else
    launch_block<DT, D, MP, GMAX>(a, units, units <= kNumCU ? 8 : 4, st);
}

template <class DT, int D>
void launch_mode(const SelectArgs& a, hipStream_t st) {
  const bool mp = a.similarity == MPC_SIM_MAXPROD;
  const bool gmax = a.group == MPC_GROUP_MAX && a.Hq > a.Hsel;  // one-head units: max = sum
  if (gmax)
    mp ? launch_plan<DT, D, true, true>(a, st) : launch_plan<DT, D, false, true>(a, st);
  else
    mp ? launch_plan<DT, D, true, false>(a, st) : launch_plan<DT, D, false, false>(a, st);
}

template <class DT>
hipError_t launch_dt(const SelectArgs& a, int D, hipStream_t st) {
  if (D == 64)
    launch_mode<DT, 64>(a, st);
  else if (D == 128)
    launch_mode<DT, 128>(a, st);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

size_t select_smem_bytes(int D, int S, int NC, int qrows) { return dev::select_smem_bytes_dev(D, S, NC, qrows); }

int select_query_rows(const SelectArgs& a) {
  const bool sep = a.similarity == MPC_SIM_MAXPROD || (a.group == MPC_GROUP_MAX && a.Hq > a.Hsel);
  return sep ? a.Hq / a.Hsel : 1;
}

hipError_t launch_select(const SelectArgs& a, int dtype, int D, hipStream_t st) {
  switch (dtype) {
    case MPC_FP32: return launch_dt<F32>(a, D, st);
    case MPC_FP16: return launch_dt<F16>(a, D, st);
    case MPC_BF16: return launch_dt<BF16>(a, D, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace mpc
