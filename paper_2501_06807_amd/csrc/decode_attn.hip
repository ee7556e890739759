// Sparse decode attention over the selected clusters (gather + online softmax), gfx950.
//
// One work unit = (layer, sequence, kv head). Its token list is the concatenation of the
// selected clusters' rows of the kept cache. A unit may be split over several workgroups
// (split-K); each writes an (m, l, acc) partial and the last one to finish merges them.
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
  __shared__ int s_last;

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
      const int sl = base + (u * NW + w) * RPW + rg;
      int row = 0;
      ok[u] = sl < hi;
      if (ok[u]) {
        // cluster ids come from the caller: anything outside [0, C) contributes nothing
        const int c = s_sel[sl / a.s];
        const long long r = (long long)c * a.s + sl % a.s;
        ok[u] = c >= 0 && r < a.Ts;
        row = ok[u] ? (int)r : 0;
      }
      const size_t off = ((size_t)row * D + li * EPL) * DT::kElt;
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
#pragma unroll
        for (int o = LPR / 2; o > 0; o >>= 1) p += __shfl_xor(p, o);
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
  if (a.splits == 1) return;

  // split-K: the last workgroup of the unit to finish merges the partials
  __threadfence();
  __syncthreads();
  if (tid == 0) s_last = atomicAdd(&a.counters[unit], 1) == a.splits - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  for (int t = tid; t < G * D; t += NW * kWave) {
    const int g = t / D, dim = t % D;
    const float* p0 = a.part + ((size_t)unit * a.splits * G + g) * (D + 2);
    const size_t stride = (size_t)G * (D + 2);
    float M = -1e30f;
    for (int i = 0; i < a.splits; ++i) M = fmaxf(M, __builtin_nontemporal_load(p0 + i * stride + D));
    float L = 0.f, O = 0.f;
    for (int i = 0; i < a.splits; ++i) {
      const float* p = p0 + i * stride;
      const float r = fast_exp2(__builtin_nontemporal_load(p + D) - M);
      L += __builtin_nontemporal_load(p + D + 1) * r;
      O += __builtin_nontemporal_load(p + dim) * r;
    }
    store_elt<DT>(a.out, (q_row0 + g) * D + dim, O / L);
    if (dim == 0 && a.lse) a.lse[q_row0 + g] = (M + __log2f(L)) * 0.69314718055994531f;
  }
  if (tid == 0) a.counters[unit] = 0;
}

template <class DT, int D, int G>
hipError_t launch_dt_d_g(const DecodeArgs& a, int units, hipStream_t st) {
  constexpr int NW = kDecodeWaves, U = 4;
  hipLaunchKernelGGL((k_sparse_decode<DT, D, G, NW, U>), dim3(units * a.splits), dim3(NW * kWave), 0,
                     st, a);
  return hipGetLastError();
}

template <class DT, int D>
hipError_t launch_dt_d(const DecodeArgs& a, int G, int units, hipStream_t st) {
  switch (G) {
    case 1: return launch_dt_d_g<DT, D, 1>(a, units, st);
    case 2: return launch_dt_d_g<DT, D, 2>(a, units, st);
    case 4: return launch_dt_d_g<DT, D, 4>(a, units, st);
    case 8: return launch_dt_d_g<DT, D, 8>(a, units, st);
  }
  return hipErrorInvalidValue;
}

template <class DT>
hipError_t launch_dt(const DecodeArgs& a, int D, int G, int units, hipStream_t st) {
  if (D == 64) return launch_dt_d<DT, 64>(a, G, units, st);
  if (D == 128) return launch_dt_d<DT, 128>(a, G, units, st);
  return hipErrorInvalidValue;
}

}  // namespace

int decode_splits(int units, int n_slot, int D, int elt) {
  const int lpr = D * elt / 16;
  const int rows_per_pass = kDecodeWaves * (kWave / lpr);
  int max_splits = n_slot / rows_per_pass;
  if (max_splits < 1) max_splits = 1;
  int s = (kDecodeTargetBlocks + units - 1) / units;
  if (s > max_splits) s = max_splits;
  if (s > 64) s = 64;
  return s < 1 ? 1 : s;
}

hipError_t launch_sparse_decode(const DecodeArgs& a, int dtype, int D, int G, int units,
                                hipStream_t st) {
  switch (dtype) {
    case MPC_FP32: return launch_dt<F32>(a, D, G, units, st);
    case MPC_FP16: return launch_dt<F16>(a, D, G, units, st);
    case MPC_BF16: return launch_dt<BF16>(a, D, G, units, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace mpc
