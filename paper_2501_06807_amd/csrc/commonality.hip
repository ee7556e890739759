// Commonality score of m + 1 adjacent layers (Sec. 3, Observation 3), gfx950.
//
// One wave per unit (e.g. a (sequence, head) pair). Each lane takes entries idx[l][u][j] of the
// layers l = 0 .. L-m-1 and counts those present in the sets of all of layers l+1 .. l+m (a scan
// of each set; sets hold distinct entries in any order). The wave's integer count, divided once
// in fp64 by k (L - m), is the score, so it is exact up to that one rounding.
#include "commonality.h"

namespace mpc {
namespace {

constexpr int kWavesPerGroup = 4;

__global__ __launch_bounds__(kWavesPerGroup* kWave) void k_commonality(int L, int units, int k, int m,
                                                                       const int32_t* idx, double* out) {
  const int lane = threadIdx.x % kWave;
  const int u = blockIdx.x * kWavesPerGroup + threadIdx.x / kWave;
  if (u >= units) return;
  const size_t layer_stride = (size_t)units * k;
  const int32_t* base = idx + (size_t)u * k;
  int count = 0;
  for (int p = lane; p < (L - m) * k; p += kWave) {
    const int l = p / k, j = p % k;
    const int32_t v = base[(size_t)l * layer_stride + j];
    bool in_all = true;
    for (int i = l + 1; i <= l + m && in_all; ++i) {
      const int32_t* set = base + (size_t)i * layer_stride;
      bool found = false;
      for (int t = 0; t < k && !found; ++t) found = set[t] == v;
      in_all = found;
    }
    count += in_all;
  }
  count = wave_sum(count);
  if (lane == 0) out[u] = (double)count / ((double)k * (double)(L - m));
}

}  // namespace

hipError_t launch_commonality(int L, int units, int k, int m, const int32_t* idx, double* out, hipStream_t st) {
  const dim3 grid((units + kWavesPerGroup - 1) / kWavesPerGroup);
  hipLaunchKernelGGL(k_commonality, grid, dim3(kWavesPerGroup * kWave), 0, st, L, units, k, m, idx, out);
  return hipGetLastError();
}

}  // namespace mpc
