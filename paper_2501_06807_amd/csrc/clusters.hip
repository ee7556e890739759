// Cluster representatives: per-channel max / min of each fine cluster and super-cluster of the
// kept cache, folded into alpha * r^max + (1 - alpha) * r^min, gfx950.
//
// One workgroup per (owner layer, sequence, kv head, super-cluster). Each wave streams the rows of
// one fine cluster at a time with coalesced 16-byte loads (LPR lanes per row), reduces max / min
// over its row groups with cross-lane shuffles, writes the fine representative and folds the
// bounds into its super-cluster bounds; the waves' super bounds meet in LDS. Max / min are exact,
// and the representative is two fp32 products and one fp32 sum with no contraction.
#include "clusters.h"

namespace mpc {
namespace {

template <class DT, int D, int NW>
__global__ __launch_bounds__(NW* kWave) void k_build(BuildArgs a) {
#pragma clang fp contract(off)
  constexpr int EPL = DT::kVec;
  constexpr int LPR = D / EPL;
  constexpr int RPW = kWave / LPR;
  __shared__ float s_max[NW][D], s_min[NW][D];

  const int sup = blockIdx.x % a.S;
  const int ou = blockIdx.x / a.S;  // (owner index * B + b) * Hkv + h
  const int l = a.own.l[ou / (a.B * a.Hkv)];
  const size_t unit = (size_t)l * a.B * a.Hkv + ou % (a.B * a.Hkv);
  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  const int rg = lane / LPR, li = lane % LPR;
  const char* kh = (const char*)a.k + (size_t)unit * a.Ts * D * DT::kElt;

  float smax[EPL], smin[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    smax[e] = -INFINITY;
    smin[e] = INFINITY;
  }
  const int c_end = min(a.C, (sup + 1) * a.f);
  for (int c = sup * a.f + w; c < c_end; c += NW) {
    float cmax[EPL], cmin[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      cmax[e] = -INFINITY;
      cmin[e] = INFINITY;
    }
    const int r_end = min(a.Ts, (c + 1) * a.s);
    for (int r = c * a.s + rg; r < r_end; r += RPW) {
      float x[EPL];
      unpack<DT>(ldg16(kh + ((size_t)r * D + li * EPL) * DT::kElt), x);
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        cmax[e] = fmaxf(cmax[e], x[e]);
        cmin[e] = fminf(cmin[e], x[e]);
      }
    }
#pragma unroll
    for (int o = LPR; o < kWave; o <<= 1) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        cmax[e] = fmaxf(cmax[e], __shfl_xor(cmax[e], o));
        cmin[e] = fminf(cmin[e], __shfl_xor(cmin[e], o));
      }
    }
    if (rg == 0) {
      float* out = a.cent + ((size_t)unit * a.C + c) * D + li * EPL;
#pragma unroll
      for (int e = 0; e < EPL; ++e) out[e] = a.alpha * cmax[e] + a.beta * cmin[e];
    }
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      smax[e] = fmaxf(smax[e], cmax[e]);
      smin[e] = fminf(smin[e], cmin[e]);
    }
  }
  if (rg == 0) {
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      s_max[w][li * EPL + e] = smax[e];
      s_min[w][li * EPL + e] = smin[e];
    }
  }
  __syncthreads();
  for (int i = tid; i < D; i += NW * kWave) {
    float mx = -INFINITY, mn = INFINITY;
#pragma unroll
    for (int j = 0; j < NW; ++j) {
      mx = fmaxf(mx, s_max[j][i]);
      mn = fminf(mn, s_min[j][i]);
    }
    a.scent[((size_t)unit * a.S + sup) * D + i] = a.alpha * mx + a.beta * mn;
  }
}

template <class DT>
hipError_t launch_dt(const BuildArgs& a, int D, int blocks, hipStream_t st) {
  constexpr int NW = 4;
  if (D == 64) {
    hipLaunchKernelGGL((k_build<DT, 64, NW>), dim3(blocks), dim3(NW * kWave), 0, st, a);
  } else if (D == 128) {
    hipLaunchKernelGGL((k_build<DT, 128, NW>), dim3(blocks), dim3(NW * kWave), 0, st, a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_build(const BuildArgs& a, int dtype, int D, hipStream_t st) {
  const int blocks = a.own.n * a.B * a.Hkv * a.S;
  switch (dtype) {
    case MPC_FP32: return launch_dt<F32>(a, D, blocks, st);
    case MPC_FP16: return launch_dt<F16>(a, D, blocks, st);
    case MPC_BF16: return launch_dt<BF16>(a, D, blocks, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace mpc
