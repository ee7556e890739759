// Cluster representatives of each fine cluster and super-cluster of the kept cache, gfx950:
// per-channel max / min folded into alpha * r^max + (1 - alpha) * r^min (linear form), or the
// two bound rows (max-product bound), or the average (fp64 sums, one rounding to fp32).
//
// One workgroup per (owner layer, sequence, kv head, super-cluster), over all super-clusters or,
// when a decode-time tail is sealed into a new cluster, over the one super-cluster that holds it.
// Each wave streams the rows of one fine cluster at a time with coalesced 16-byte loads (LPR
// lanes per row), reduces max / min over its row groups with cross-lane shuffles, writes the fine
// representative and folds the bounds into its super-cluster bounds; the waves' super bounds meet
// in LDS. In prefill mode a wave first reads the kept positions of up to 64 rows of its cluster
// (one coalesced load) and takes each row's position from its lane; every row it reads from the
// prompt cache is also written, with its value row, to the kept cache. Max / min are exact,
// the linear representative is two fp32 products and one fp32 sum with no contraction, and the
// average's fp64 sums of 16-bit keys are exact, so their order does not matter.
#include "clusters.h"

namespace mpc {
namespace {

template <class DT, int D, int NW, int SIM, bool GATHER>
__global__ __launch_bounds__(NW* kWave) void k_build(BuildArgs a) {
#pragma clang fp contract(off)
  constexpr int EPL = DT::kVec;
  constexpr int LPR = D / EPL;
  constexpr int RPW = kWave / LPR;
  constexpr int R = SIM == MPC_SIM_MAXPROD ? 2 : 1;  // representative rows
  constexpr bool MEAN = SIM == MPC_SIM_MEAN;
  __shared__ float s_max[NW][D], s_min[NW][D];
  __shared__ double s_sum[MEAN ? NW : 1][MEAN ? D : 1];

  const int sup = a.sup0 + blockIdx.x % a.n_sup;
  const int ou = blockIdx.x / a.n_sup;  // (owner index * B + b) * Hkv + h
  const int l = a.own.local(ou / (a.B * a.Hkv));
  const size_t unit = (size_t)l * a.B * a.Hkv + ou % (a.B * a.Hkv);
  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  const int rg = lane / LPR, li = lane % LPR;
  constexpr int RB = D * DT::kElt;  // bytes per row
  const char* kh = (const char*)a.k + (size_t)unit * a.rows * RB;
  // prefill mode: the unit's kept set, prompt rows and kept-cache rows
  size_t src_set = 0, dst_set = 0, src_rows = 0, dst_rows = 0;
  if constexpr (GATHER) {
    const int o = owner_layer(a.layer0 + l, a.g.period, a.g.start) - a.layer0;
    const int src_l = o >= 0 ? o : l;  // an owner before the block: the set is already in place
    src_set = (unit - (size_t)(l - src_l) * a.B * a.Hkv) * a.g.keep;
    dst_set = unit * a.g.keep;
    src_rows = unit * a.g.T;
    dst_rows = unit * a.rows;
  }

  float smax[EPL], smin[EPL];
  double ssum[EPL];
#pragma unroll
  for (int e = 0; e < EPL; ++e) {
    smax[e] = -INFINITY;
    smin[e] = INFINITY;
    ssum[e] = 0.0;
  }
  const int c_end = min(a.C, (sup + 1) * a.f);
  for (int c = sup * a.f + w; c < c_end; c += NW) {
    float cmax[EPL], cmin[EPL];
    double csum[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      cmax[e] = -INFINITY;
      cmin[e] = INFINITY;
      csum[e] = 0.0;
    }
    const int r_end = min(a.Ts, (c + 1) * a.s);
    auto fold = [&](const uint4 raw) {
      float x[EPL];
      unpack<DT>(raw, x);
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        if constexpr (MEAN) {
          csum[e] += (double)x[e];
        } else {
          cmax[e] = fmaxf(cmax[e], x[e]);
          cmin[e] = fminf(cmin[e], x[e]);
        }
      }
    };
    if constexpr (GATHER) {
      for (int r0 = c * a.s; r0 < r_end; r0 += kWave) {
        const int n = min(kWave, r_end - r0);
        int pos = 0;
        if (lane < n) {
          pos = a.g.kept[src_set + r0 + lane];
          if (src_set != dst_set) a.g.kept[dst_set + r0 + lane] = pos;
          pos = min(max(pos, 0), a.g.T - 1);  // positions supplied by the caller are clamped
        }
        for (int j0 = 0; j0 < n; j0 += RPW) {  // wave-uniform trip count: every lane shuffles
          const int j = j0 + rg;
          const int p = __shfl(pos, min(j, n - 1));
          if (j < n) {
            const size_t so = (src_rows + p) * RB + li * 16, dof = (dst_rows + r0 + j) * RB + li * 16;
            const uint4 kr = ldg16((const char*)a.g.k_src + so);
            const uint4 vr = ldg16((const char*)a.g.v_src + so);
            *(uint4*)((char*)a.g.k_dst + dof) = kr;
            *(uint4*)((char*)a.g.v_dst + dof) = vr;
            fold(kr);
          }
        }
      }
    } else {
      for (int r = c * a.s + rg; r < r_end; r += RPW) fold(ldg16(kh + (size_t)r * RB + li * 16));
    }
#pragma unroll
    for (int o = LPR; o < kWave; o <<= 1) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        if constexpr (MEAN) {
          csum[e] += __shfl_xor(csum[e], o);
        } else {
          cmax[e] = fmaxf(cmax[e], __shfl_xor(cmax[e], o));
          cmin[e] = fminf(cmin[e], __shfl_xor(cmin[e], o));
        }
      }
    }
    if (rg == 0) {
      float* out = a.cent + ((size_t)unit * a.cs + c) * R * D + li * EPL;
#pragma unroll
      for (int e = 0; e < EPL; ++e) {
        if constexpr (SIM == MPC_SIM_LINEAR) {
          out[e] = a.alpha * cmax[e] + a.beta * cmin[e];
        } else if constexpr (SIM == MPC_SIM_MAXPROD) {
          out[e] = cmax[e];
          out[D + e] = cmin[e];
        } else {
          out[e] = (float)(csum[e] / (double)(r_end - c * a.s));
        }
      }
    }
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      if constexpr (MEAN) {
        ssum[e] += csum[e];
      } else {
        smax[e] = fmaxf(smax[e], cmax[e]);
        smin[e] = fminf(smin[e], cmin[e]);
      }
    }
  }
  if (rg == 0) {
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
      if constexpr (MEAN) {
        s_sum[w][li * EPL + e] = ssum[e];
      } else {
        s_max[w][li * EPL + e] = smax[e];
        s_min[w][li * EPL + e] = smin[e];
      }
    }
  }
  __syncthreads();
  const int n_tok = min(a.Ts, c_end * a.s) - sup * a.f * a.s;  // tokens of the super-cluster
  float* sout = a.scent + ((size_t)unit * a.ss + sup) * R * D;
  for (int i = tid; i < D; i += NW * kWave) {
    if constexpr (MEAN) {
      double sum = 0.0;
#pragma unroll
      for (int j = 0; j < NW; ++j) sum += s_sum[j][i];
      sout[i] = (float)(sum / (double)n_tok);
    } else {
      float mx = -INFINITY, mn = INFINITY;
#pragma unroll
      for (int j = 0; j < NW; ++j) {
        mx = fmaxf(mx, s_max[j][i]);
        mn = fminf(mn, s_min[j][i]);
      }
      if constexpr (SIM == MPC_SIM_LINEAR) {
        sout[i] = a.alpha * mx + a.beta * mn;
      } else {
        sout[i] = mx;
        sout[D + i] = mn;
      }
    }
  }
}

template <class DT, int D, bool GATHER>
void launch_sim(const BuildArgs& a, int blocks, hipStream_t st) {
  constexpr int NW = 4;
  if (a.similarity == MPC_SIM_MAXPROD)
    hipLaunchKernelGGL((k_build<DT, D, NW, MPC_SIM_MAXPROD, GATHER>), dim3(blocks), dim3(NW * kWave), 0, st, a);
  else if (a.similarity == MPC_SIM_MEAN)
    hipLaunchKernelGGL((k_build<DT, D, NW, MPC_SIM_MEAN, GATHER>), dim3(blocks), dim3(NW * kWave), 0, st, a);
  else
    hipLaunchKernelGGL((k_build<DT, D, NW, MPC_SIM_LINEAR, GATHER>), dim3(blocks), dim3(NW * kWave), 0, st, a);
}

template <class DT, int D>
void launch_mode(const BuildArgs& a, int blocks, hipStream_t st) {
  if (a.g.kept)
    launch_sim<DT, D, true>(a, blocks, st);
  else
    launch_sim<DT, D, false>(a, blocks, st);
}

template <class DT>
hipError_t launch_dt(const BuildArgs& a, int D, int blocks, hipStream_t st) {
  if (D == 64)
    launch_mode<DT, 64>(a, blocks, st);
  else if (D == 128)
    launch_mode<DT, 128>(a, blocks, st);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace

hipError_t launch_build(const BuildArgs& a, int dtype, int D, hipStream_t st) {
  const int blocks = a.own.n * a.B * a.Hkv * a.n_sup;
  switch (dtype) {
    case MPC_FP32: return launch_dt<F32>(a, D, blocks, st);
    case MPC_FP16: return launch_dt<F16>(a, D, blocks, st);
    case MPC_BF16: return launch_dt<BF16>(a, D, blocks, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace mpc
