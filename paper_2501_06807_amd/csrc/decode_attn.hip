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
#include "decode_attn.h"

namespace mpc {
namespace {

constexpr int kMaxSel = 1024;

template <class DT, int D, int G, int NW, int U>
__global__ __launch_bounds__(NW* kWave) void k_sparse_decode(DecodeArgs a) {
  constexpr int EPL = DT::kVec;
  constexpr int LPR = D / EPL;
  constexpr int RPW = kWave / LPR;
  static_assert(LPR <= kWave && kWave % LPR == 0, "row must fit a wave");

  __shared__ int32_t s_sel[kMaxSel];
  __shared__ float s_m[NW][G], s_l[NW][G];
  __shared__ float s_acc[NW][G][D];

  const int unit = blockIdx.x / a.splits;
  const int split = blockIdx.x % a.splits;
  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  const int rg = lane / LPR, li = lane % LPR;

  for (int i = tid; i < a.k_sel; i += NW * kWave) s_sel[i] = a.sel[(size_t)unit * a.k_sel + i];

  // unit = (l * B + b) * Hkv + h ; q-heads h*G .. h*G+G-1 of the same (l, b)
  const size_t q_row0 = (size_t)(unit / a.Hkv) * a.Hq + (size_t)(unit % a.Hkv) * G;
  float qf[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    float t[EPL];
    unpack<DT>(ldg16((const char*)a.q + ((q_row0 + g) * D + li * EPL) * DT::kElt), t);
#pragma unroll
    for (int e = 0; e < EPL; ++e) qf[g][e] = t[e] * a.qscale;
  }
  __syncthreads();

  const int n_slot = a.k_sel * a.s;
  const int chunk = (n_slot + a.splits - 1) / a.splits;
  const int lo = split * chunk, hi = min(n_slot, lo + chunk);
  const char* kbase = (const char*)a.k + (size_t)unit * a.Ts * D * DT::kElt;
  const char* vbase = (const char*)a.v + (size_t)unit * a.Ts * D * DT::kElt;

  float m[G], l[G], acc[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -1e30f;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[g][e] = 0.f;
  }

  for (int base = lo; base < hi; base += NW * RPW * U) {
    uint4 kr[U], vr[U];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      // slot -> (selected cluster, row in cluster); ids come from the caller, so anything outside
      // [0, C) or past the kept length contributes nothing (and loads row 0 harmlessly)
      const int sl = base + (u * NW + w) * RPW + rg;
      const int slc = min(sl, hi - 1);
      const int c = s_sel[slc / a.s];
      const int r = c * a.s + slc % a.s;
      ok[u] = (sl < hi) & ((unsigned)c < (unsigned)a.C) & (r < a.Ts);
      const size_t off = ((size_t)(ok[u] ? r : 0) * D + li * EPL) * DT::kElt;
      kr[u] = ldg16(kbase + off);
      vr[u] = ldg16(vbase + off);
    }
    float sc[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float kf[EPL];
      unpack<DT>(kr[u], kf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float p = 0.f;
#pragma unroll
        for (int e = 0; e < EPL; ++e) p += qf[g][e] * kf[e];
        p = group_sum<LPR>(p);
        sc[u][g] = ok[u] ? p : -INFINITY;
      }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      float mx = m[g];
#pragma unroll
      for (int u = 0; u < U; ++u) mx = fmaxf(mx, sc[u][g]);
      const float r = fast_exp2(m[g] - mx);
      l[g] *= r;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[g][e] *= r;
      m[g] = mx;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float vf[EPL];
      unpack<DT>(vr[u], vf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float p = fast_exp2(sc[u][g] - m[g]);
        l[g] += p;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[g][e] += p * vf[e];
      }
    }
  }

  // merge the RPW row groups of the wave
#pragma unroll
  for (int o = LPR; o < kWave; o <<= 1) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float mo = __shfl_xor(m[g], o), lo2 = __shfl_xor(l[g], o);
      const float mx = fmaxf(m[g], mo);
      const float ra = fast_exp2(m[g] - mx), rb = fast_exp2(mo - mx);
      l[g] = l[g] * ra + lo2 * rb;
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[g][e] = acc[g][e] * ra + __shfl_xor(acc[g][e], o) * rb;
      m[g] = mx;
    }
  }
  if (rg == 0) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) s_acc[w][g][li * EPL + e] = acc[g][e];
      if (li == 0) {
        s_m[w][g] = m[g];
        s_l[w][g] = l[g];
      }
    }
  }
  __syncthreads();

  // merge the NW waves
  for (int t = tid; t < G * D; t += NW * kWave) {
    const int g = t / D, dim = t % D;
    float M = -1e30f;
#pragma unroll
    for (int i = 0; i < NW; ++i) M = fmaxf(M, s_m[i][g]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const float r = fast_exp2(s_m[i][g] - M);
      L += s_l[i][g] * r;
      O += s_acc[i][g][dim] * r;
    }
    if (a.splits == 1) {
      store_elt<DT>(a.out, (q_row0 + g) * D + dim, O / L);
      if (dim == 0 && a.lse) a.lse[q_row0 + g] = (M + __log2f(L)) * 0.69314718055994531f;
    } else {
      float* p = a.part + (((size_t)unit * a.splits + split) * G + g) * (D + 2);
      p[dim] = O;
      if (dim == 0) {
        p[D] = M;
        p[D + 1] = L;
      }
    }
  }
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
