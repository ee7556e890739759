// Device code of the sparse decode attention, shared by the standalone kernel and the fused
// decode-step kernel.
#pragma once
#include "decode_attn.h"

namespace mpc {
namespace dev {

// A gathered K / V row chunk: plain, or with the non-temporal hint, so that a row read once per
// call streams through the caches without displacing what the next call reads again.
template <bool STREAM>
__device__ __forceinline__ uint4 kv_load(const void* p) {
  if constexpr (STREAM)
    return ldg16_stream(p);
  else
    return ldg16(p);
}

constexpr int kMaxSel = 1024;

// Byte offset of a unit's K/V block: (layer, sequence) of the unit, then its cache head.
template <int D, class DT>
__device__ __forceinline__ size_t cache_offset(const DecodeArgs& a, int unit) {
  const size_t cu = (size_t)(unit / a.Hkv) * a.cache_heads + (unit % a.Hkv) / a.cache_div;
  return cu * a.rows * D * DT::kElt;
}

// The unit's cluster list in LDS: its selected clusters, with ids outside [0, C) replaced by -1
// (they contribute nothing), then the clusters C, C + 1, ... that hold the tail rows
// [Ts, Ts + n_tail) (Ts is a multiple of s when there is a tail). Returns the list length.
// COH_SEL: the selection was written by another workgroup of the same launch, so it is read with
// device-coherent loads. pick: if not null, the selection computed by this workgroup (LDS).
template <int NW, bool COH_SEL>
__device__ __forceinline__ int load_list(const DecodeArgs& a, int unit, int32_t* s_sel, const int32_t* pick) {
  const int n_list = a.k_sel + (a.n_tail + a.s - 1) / a.s;
  for (int i = threadIdx.x; i < n_list; i += NW * kWave) {
    int c = a.C + (i - a.k_sel);
    if (i < a.k_sel) {
      const int32_t* src = a.sel + (size_t)unit * a.k_sel + i;
      if (pick)
        c = pick[i];
      else if constexpr (COH_SEL)
        c = __hip_atomic_load(src, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      else
        c = *src;
      if ((unsigned)c >= (unsigned)a.C) c = -1;
    }
    s_sel[i] = c;
  }
  return n_list;
}

// Cross-wave merge of one unit's (m, l, acc) from LDS, then the output (one split) or the split-K
// partial and, for the last split to arrive, the merge of all partials.
template <class DT, int D, int G, int NW>
__device__ __forceinline__ void finish_unit(const DecodeArgs& a, int unit, int split, size_t q_row0,
                                            const float (*s_m)[G], const float (*s_l)[G],
                                            const float (*s_acc)[G][D]) {
  const int tid = threadIdx.x;
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
      // partial of this split, written device-coherently for the split that merges
      float* p = a.part + (((size_t)unit * a.splits + split) * G + g) * (D + 2);
      st_coherent(p + dim, O);
      if (dim == 0) {
        st_coherent(p + D, M);
        st_coherent(p + D + 1, L);
      }
    }
  }
  if (a.splits == 1) return;

  // Split-K: the last split of the unit to arrive merges all partials. Every split's partial
  // stores have completed before its arrival is counted, and the merging split reads them with
  // device-coherent loads, so no cache write-back fence is needed.
  __shared__ int s_last;
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0) {
    const int c = __hip_atomic_fetch_add(&a.cnt[unit], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = c == a.splits - 1;
    if (s_last) __hip_atomic_store(&a.cnt[unit], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (!s_last) return;
  for (int t = tid; t < G * D; t += NW * kWave) {
    const int g = t / D, dim = t % D;
    const float* p0 = a.part + ((size_t)unit * a.splits * G + g) * (D + 2);
    const size_t stride = (size_t)G * (D + 2);
    // every split's (m, l, o) is requested before any is used: one memory round trip for the
    // merge instead of one per split and pass (these loads bypass the per-die caches)
    float mv[kMaxSplits], lv[kMaxSplits], ov[kMaxSplits];
#pragma unroll
    for (int i = 0; i < kMaxSplits; ++i) {
      if (i < a.splits) {
        const float* p = p0 + i * stride;
        mv[i] = ld_coherent(p + D);
        lv[i] = ld_coherent(p + D + 1);
        ov[i] = ld_coherent(p + dim);
      }
    }
    float M = -1e30f;
#pragma unroll
    for (int i = 0; i < kMaxSplits; ++i)
      if (i < a.splits) M = fmaxf(M, mv[i]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxSplits; ++i) {
      if (i < a.splits) {
        const float r = fast_exp2(mv[i] - M);
        L += lv[i] * r;
        O += ov[i] * r;
      }
    }
    store_elt<DT>(a.out, (q_row0 + g) * D + dim, O / L);
    if (dim == 0 && a.lse) a.lse[q_row0 + g] = (M + __log2f(L)) * 0.69314718055994531f;
  }
}

// Attention of one work unit (or one split of it). COH_SEL: read the selection with
// device-coherent loads (it was written by another workgroup of the same launch). The gathered V
// rows are loaded with the non-temporal hint; the K rows too when STREAM_K.
template <class DT, int D, int G, int NW, int U, bool COH_SEL, bool STREAM_K>
__device__ __forceinline__ void attend_unit(const DecodeArgs& a, int unit, int split, const int32_t* pick) {
  constexpr int EPL = DT::kVec;
  constexpr int LPR = D / EPL;
  constexpr int RPW = kWave / LPR;
  constexpr bool kDot2 = DT::kElt == 2;
  constexpr float kSlack = 8.f;
  static_assert(LPR <= kWave && kWave % LPR == 0, "row must fit a wave");

  __shared__ int32_t s_sel[kMaxSel];
  __shared__ float s_m[NW][G], s_l[NW][G];
  __shared__ float s_acc[NW][G][D];

  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  const int rg = lane / LPR, li = lane % LPR;

  // unit = (l * B + b) * Hkv + h ; q-heads h*G .. h*G+G-1 of the same (l, b)
  const size_t q_row0 = (size_t)(unit / a.Hkv) * a.Hq + (size_t)(unit % a.Hkv) * G;
  // 16-bit types: q stays packed and the dot products use the two-wide dot instructions (exact
  // bf16 / fp16 products, fp32 sums), scaled afterwards; fp32: q pre-scaled, fused multiply-adds
  uint4 qraw[G];
  float qf[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    qraw[g] = ldg16((const char*)a.q + ((q_row0 + g) * D + li * EPL) * DT::kElt);
    if constexpr (!kDot2) {
      float t[EPL];
      unpack<DT>(qraw[g], t);
#pragma unroll
      for (int e = 0; e < EPL; ++e) qf[g][e] = t[e] * a.qscale;
    }
  }
  // the cluster list after the query loads, so that both are in flight together
  const int n_list = load_list<NW, COH_SEL>(a, unit, s_sel, pick);
  __syncthreads();

  const int n_slot = n_list * a.s, rows_end = a.Ts + a.n_tail;
  const int chunk = (n_slot + a.splits - 1) / a.splits;
  const int lo = split * chunk, hi = min(n_slot, lo + chunk);
  const char* kbase = (const char*)a.k + cache_offset<D, DT>(a, unit);
  const char* vbase = (const char*)a.v + cache_offset<D, DT>(a, unit);

  float m[G], l[G], acc[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -1e30f;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[g][e] = 0.f;
  }

  // slot cursors: slot = cluster position * s + row; each step of the loop advances every
  // cursor by STEP slots without a division
  constexpr int STEP = NW * RPW * U;
  int cpos[U], crow[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int sl = lo + (u * NW + w) * RPW + rg;
    cpos[u] = sl / a.s;
    crow[u] = sl % a.s;
  }
  const int step_pos = STEP / a.s, step_row = STEP % a.s;

  // gathers the U rows of every lane for the step at slot `base` and advances the cursors
  auto fetch = [&](int base, uint4 (&kr)[U], uint4 (&vr)[U], bool (&ok)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      // a masked slot (past the list, a rejected id, past the cached rows) contributes nothing
      // and loads row 0 harmlessly
      const int sl = base + (u * NW + w) * RPW + rg;
      const int c = s_sel[min(cpos[u], n_list - 1)];
      const int r = c * a.s + crow[u];
      ok[u] = (sl < hi) & (c >= 0) & (r < rows_end);
      const unsigned off = (unsigned)(ok[u] ? r : 0) * (unsigned)(D * DT::kElt) + (unsigned)(li * 16);
      kr[u] = kv_load<STREAM_K>(kbase + off);
      vr[u] = kv_load<true>(vbase + off);
      crow[u] += step_row;
      cpos[u] += step_pos;
      if (crow[u] >= a.s) {
        crow[u] -= a.s;
        ++cpos[u];
      }
    }
  };

  for (int base = lo; base < hi; base += STEP) {
    uint4 kr[U], vr[U];
    bool ok[U];
    fetch(base, kr, vr, ok);
    float sc[U][G];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float kf[EPL];
      if constexpr (!kDot2) unpack<DT>(kr[u], kf);
#pragma unroll
      for (int g = 0; g < G; ++g) {
        float p = 0.f;
        if constexpr (kDot2) {
          p = dot2<DT>(qraw[g].x, kr[u].x, p);
          p = dot2<DT>(qraw[g].y, kr[u].y, p);
          p = dot2<DT>(qraw[g].z, kr[u].z, p);
          p = dot2<DT>(qraw[g].w, kr[u].w, p);
        } else {
#pragma unroll
          for (int e = 0; e < EPL; ++e) p += qf[g][e] * kf[e];
        }
        p = group_sum<LPR>(p);
        if constexpr (kDot2) p *= a.qscale;
        sc[u][g] = ok[u] ? p : -INFINITY;
      }
    }
    // The running maximum is refreshed only when a score exceeds it by more than kSlack (log2
    // units): exponentials stay below 2^kSlack, and the rescale of l and acc is skipped by the
    // whole wave in almost every step. Any reference maximum gives the same normalised result.
    float mx[G];
    bool up = false;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      mx[g] = m[g];
#pragma unroll
      for (int u = 0; u < U; ++u) mx[g] = fmaxf(mx[g], sc[u][g]);
      up |= mx[g] > m[g] + kSlack;
    }
    if (__any(up)) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float r = fast_exp2(m[g] - mx[g]);
        l[g] *= r;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[g][e] *= r;
        m[g] = mx[g];
      }
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

  finish_unit<DT, D, G, NW>(a, unit, split, q_row0, s_m, s_l, s_acc);
}

// Groups of four query heads over 16-bit rows: the scores come from the matrix cores
// (v_mfma_f32_16x16x32_{bf16,f16}: A = the group's four queries, each repeated on four rows,
// B = 16 gathered key rows), so every lane receives the four head scores of one token with no
// cross-lane reduction; p·V stays on the VALU in the row layout, each lane taking its row's
// probabilities from the score lane with one cross-lane read per head. The reference maximum is
// uniform over the wave (refreshed with a wave reduction only when a score exceeds it by more than
// the slack), so the row layout's partial sums need no rescale when they meet.
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));

template <class DT>
__device__ __forceinline__ f32x4_t mfma16(uint4 a, uint4 b, f32x4_t c);
template <>
__device__ __forceinline__ f32x4_t mfma16<BF16>(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c,
                                                 0, 0, 0);
}
template <>
__device__ __forceinline__ f32x4_t mfma16<F16>(uint4 a, uint4 b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a), __builtin_bit_cast(f16x8_t, b), c,
                                                0, 0, 0);
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

template <class DT, int D, int NW, bool COH_SEL, bool STREAM_K>
__device__ __forceinline__ void attend_unit_g4(const DecodeArgs& a, int unit, int split, const int32_t* pick) {
  constexpr int G = 4;
  constexpr int EPL = 8;              // 16-bit elements per 16-byte vector
  constexpr int LPR = D / EPL;        // lanes per row (row layout)
  constexpr int RPW = kWave / LPR;    // rows per row-layout load
  constexpr int UV = 16 / RPW;        // row-layout loads per 16 tokens
  constexpr int KK = D / 32;          // matrix-core steps over d
  constexpr int STEP = NW * 16;       // slots per workgroup step (16 per wave)
  constexpr float kSlack = 8.f;
  static_assert(DT::kElt == 2 && (D == 64 || D == 128), "16-bit rows, d = 64 or 128");

  __shared__ int32_t s_sel[kMaxSel];
  __shared__ float s_m[NW][G], s_l[NW][G];
  __shared__ float s_acc[NW][G][D];

  const int tid = threadIdx.x, lane = tid % kWave, w = tid / kWave;
  const int tk = lane % 16, kq = lane / 16;    // score layout: token of the 16, quarter of a 32-wide k step
  const int rg = lane / LPR, li = lane % LPR;  // row layout: row of the load, 16-byte column

  const size_t q_row0 = (size_t)(unit / a.Hkv) * a.Hq + (size_t)(unit % a.Hkv) * G;
  uint4 qa[KK];  // A operand: row tk holds head tk % 4
#pragma unroll
  for (int kk = 0; kk < KK; ++kk)
    qa[kk] = ldg16((const char*)a.q + ((q_row0 + tk % G) * D + kk * 32 + kq * 8) * DT::kElt);
  // the cluster list after the query loads, so that both are in flight together
  const int n_list = load_list<NW, COH_SEL>(a, unit, s_sel, pick);
  __syncthreads();

  const int n_slot = n_list * a.s, rows_end = a.Ts + a.n_tail;
  const int chunk = (n_slot + a.splits - 1) / a.splits;
  const int lo = split * chunk, hi = min(n_slot, lo + chunk);
  const char* kbase = (const char*)a.k + cache_offset<D, DT>(a, unit);
  const char* vbase = (const char*)a.v + cache_offset<D, DT>(a, unit);

  // slot cursors (cluster position, row), advanced by STEP slots per step without a division:
  // [0] the score-layout token of this lane, [1 + u] its row-layout rows
  int cpos[1 + UV], crow[1 + UV];
#pragma unroll
  for (int j = 0; j < 1 + UV; ++j) {
    const int sl = lo + w * 16 + (j == 0 ? tk : (j - 1) * RPW + rg);
    cpos[j] = sl / a.s;
    crow[j] = sl % a.s;
  }
  const int step_pos = STEP / a.s, step_row = STEP % a.s;
  // row of cursor j at step `base`; invalid slots read row 0 and are masked
  auto row_of = [&](int j, int sl, bool& ok) {
    const int c = s_sel[min(cpos[j], n_list - 1)];
    const int r = c * a.s + crow[j];
    ok = (sl < hi) & (c >= 0) & (r < rows_end);
    crow[j] += step_row;
    cpos[j] += step_pos;
    if (crow[j] >= a.s) {
      crow[j] -= a.s;
      ++cpos[j];
    }
    return (unsigned)(ok ? r : 0) * (unsigned)(D * DT::kElt);
  };

  float m[G], l[G], acc[G][EPL];
#pragma unroll
  for (int g = 0; g < G; ++g) {
    m[g] = -1e30f;
    l[g] = 0.f;
#pragma unroll
    for (int e = 0; e < EPL; ++e) acc[g][e] = 0.f;
  }

  for (int base = lo; base < hi; base += STEP) {
    bool okk;
    const unsigned koff = row_of(0, base + w * 16 + tk, okk);
    uint4 kr[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) kr[kk] = kv_load<STREAM_K>(kbase + koff + (kk * 32 + kq * 8) * DT::kElt);
    uint4 vr[UV];
#pragma unroll
    for (int u = 0; u < UV; ++u) {
      bool okv;
      const unsigned voff = row_of(1 + u, base + w * 16 + u * RPW + rg, okv);
      vr[u] = kv_load<true>(vbase + voff + li * 16);  // a masked row contributes p = 0
    }
    f32x4_t sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) sacc = mfma16<DT>(qa[kk], kr[kk], sacc);
    float sc[G];
    bool up = false;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      sc[g] = okk ? sacc[g] * a.qscale : -INFINITY;
      up |= sc[g] > m[g] + kSlack;
    }
    if (__any(up)) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float mx = wave_max(fmaxf(m[g], sc[g]));
        const float r = fast_exp2(m[g] - mx);
        l[g] *= r;
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[g][e] *= r;
        m[g] = mx;
      }
    }
    float p[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      p[g] = fast_exp2(sc[g] - m[g]);
      l[g] += p[g];
    }
#pragma unroll
    for (int u = 0; u < UV; ++u) {
      float vf[EPL];
      unpack<DT>(vr[u], vf);
      const int src = u * RPW + rg;  // score lane of this row's token
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const float pg = __shfl(p[g], src);
#pragma unroll
        for (int e = 0; e < EPL; ++e) acc[g][e] += pg * vf[e];
      }
    }
  }

  // the wave's rows meet: acc over the row groups, l over the 16 token lanes (each group of 16
  // lanes holds the same tokens' probabilities)
#pragma unroll
  for (int o = LPR; o < kWave; o <<= 1)
#pragma unroll
    for (int g = 0; g < G; ++g)
#pragma unroll
      for (int e = 0; e < EPL; ++e) acc[g][e] += __shfl_xor(acc[g][e], o);
#pragma unroll
  for (int g = 0; g < G; ++g) l[g] = group_sum<16>(l[g]);
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
  finish_unit<DT, D, G, NW>(a, unit, split, q_row0, s_m, s_l, s_acc);
}

// The attention path of a unit: matrix-core scores for four-head groups of 16-bit rows, the VALU
// path otherwise. pick: the unit's selection in LDS (computed by the same workgroup), or null to
// read it from a.sel.
template <class DT, int D, int G, int NW, int U, bool COH_SEL, bool STREAM_K>
__device__ __forceinline__ void attend(const DecodeArgs& a, int unit, int split, const int32_t* pick = nullptr) {
  if constexpr (G == 4 && DT::kElt == 2)
    attend_unit_g4<DT, D, NW, COH_SEL, STREAM_K>(a, unit, split, pick);
  else
    attend_unit<DT, D, G, NW, U, COH_SEL, STREAM_K>(a, unit, split, pick);
}

}  // namespace dev
}  // namespace mpc
