// Device code of the sparse decode attention, shared by the standalone kernel and the fused
// decode-step kernel.
#pragma once
#include "decode_attn.h"

namespace mpc {
namespace dev {

constexpr int kMaxSel = 1024;

// Attention of one work unit (or one split of it). COH_SEL: read the selection with
// device-coherent loads (it was written by another workgroup of the same launch).
template <class DT, int D, int G, int NW, int U, bool COH_SEL>
__device__ __forceinline__ void attend_unit(const DecodeArgs& a, int unit, int split) {
  constexpr int EPL = DT::kVec;
  constexpr int LPR = D / EPL;
  constexpr int RPW = kWave / LPR;
  static_assert(LPR <= kWave && kWave % LPR == 0, "row must fit a wave");

  __shared__ int32_t s_sel[kMaxSel];
  __shared__ float s_m[NW][G], s_l[NW][G];
  __shared__ float s_acc[NW][G][D];

  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  const int rg = lane / LPR, li = lane % LPR;

  for (int i = tid; i < a.k_sel; i += NW * kWave) {
    const int32_t* src = a.sel + (size_t)unit * a.k_sel + i;
    if constexpr (COH_SEL)
      s_sel[i] = __hip_atomic_load(src, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      s_sel[i] = *src;
  }

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

}  // namespace dev
}  // namespace mpc
