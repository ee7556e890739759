// Shared device helpers for the gfx950 kernels: element types, 16-byte vector loads, wave
// reductions. Wavefronts are 64 lanes wide.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "../../include/mpcache.h"

namespace mpc {

constexpr int kWave = 64;
constexpr int kNumCU = 256;         // compute units of an MI355X
constexpr size_t kMaxLds = 65536;   // LDS bytes one workgroup may allocate

// Element-type tags. A 16-byte vector holds kVec elements.
struct F32 {
  static constexpr int kElt = 4;
  static constexpr int kVec = 4;
  static constexpr int kCode = MPC_FP32;
};
struct F16 {
  static constexpr int kElt = 2;
  static constexpr int kVec = 8;
  static constexpr int kCode = MPC_FP16;
};
struct BF16 {
  static constexpr int kElt = 2;
  static constexpr int kVec = 8;
  static constexpr int kCode = MPC_BF16;
};

__device__ __forceinline__ float bf16_to_f32(uint32_t h) { return __uint_as_float(h << 16); }

__device__ __forceinline__ float f16_to_f32(uint32_t h) {
  _Float16 x = __builtin_bit_cast(_Float16, (uint16_t)h);
  return (float)x;
}

// Round-to-nearest-even conversions for stores.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ uint16_t f32_to_f16(float f) {
  return __builtin_bit_cast(uint16_t, (_Float16)f);
}

// Unpack one 16-byte vector into floats.
template <class DT>
__device__ __forceinline__ void unpack(const uint4& r, float* out);

template <>
__device__ __forceinline__ void unpack<F32>(const uint4& r, float* out) {
  out[0] = __uint_as_float(r.x);
  out[1] = __uint_as_float(r.y);
  out[2] = __uint_as_float(r.z);
  out[3] = __uint_as_float(r.w);
}
template <>
__device__ __forceinline__ void unpack<BF16>(const uint4& r, float* out) {
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(w[i] << 16);
    out[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}
template <>
__device__ __forceinline__ void unpack<F16>(const uint4& r, float* out) {
  const uint32_t w[4] = {r.x, r.y, r.z, r.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = f16_to_f32(w[i] & 0xFFFFu);
    out[2 * i + 1] = f16_to_f32(w[i] >> 16);
  }
}

// Scalar element load (used off the hot loops).
template <class DT>
__device__ __forceinline__ float load_elt(const void* base, size_t i);
template <>
__device__ __forceinline__ float load_elt<F32>(const void* base, size_t i) {
  return ((const float*)base)[i];
}
template <>
__device__ __forceinline__ float load_elt<BF16>(const void* base, size_t i) {
  return bf16_to_f32(((const uint16_t*)base)[i]);
}
template <>
__device__ __forceinline__ float load_elt<F16>(const void* base, size_t i) {
  return f16_to_f32(((const uint16_t*)base)[i]);
}


template <class DT>
__device__ __forceinline__ void store_elt(void* base, size_t i, float x);
template <>
__device__ __forceinline__ void store_elt<F32>(void* base, size_t i, float x) {
  ((float*)base)[i] = x;
}
template <>
__device__ __forceinline__ void store_elt<BF16>(void* base, size_t i, float x) {
  ((uint16_t*)base)[i] = f32_to_bf16(x);
}
template <>
__device__ __forceinline__ void store_elt<F16>(void* base, size_t i, float x) {
  ((uint16_t*)base)[i] = f32_to_f16(x);
}

__device__ __forceinline__ uint4 ldg16(const void* p) { return *(const uint4*)p; }

// The same with the non-temporal hint.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ldg16_stream(const void* p) {
  const u32x4_t v = __builtin_nontemporal_load((const u32x4_t*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Device-coherent (agent-scope) accesses for data exchanged between workgroups of one launch:
// they go through the coherent path of the per-die L2s without a cache write-back fence.
__device__ __forceinline__ void st_coherent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_coherent(const float* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Two-wide dot product of packed 16-bit pairs accumulated into fp32: c + a.lo * b.lo + a.hi * b.hi
// (the products of 16-bit values are exact in fp32).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
template <class DT>
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c);
template <>
__device__ __forceinline__ float dot2<BF16>(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c, false);
}
template <>
__device__ __forceinline__ float dot2<F16>(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2_t, a), __builtin_bit_cast(f16x2_t, b), c, false);
}
template <>
__device__ __forceinline__ float dot2<F32>(uint32_t, uint32_t, float c) {
  return c;  // not used: fp32 rows take the fused multiply-add path
}

// Owner layer of an absolute layer index (cross-layer index sharing).
__host__ __device__ __forceinline__ int owner_layer(int l, int period, int start) {
  if (period <= 1 || l < start) return l;
  return start + period * ((l - start) / period);
}

constexpr int kMaxLayers = 256;  // layers per call

// The owner layers of a block of layers [layer0, layer0 + n_layers), so that grids cover owner work
// only: every layer below `start` (or every layer when period <= 1), then start + period * j for
// j >= j0. Closed forms of a few scalars: a kernel indexing a table held in its arguments would pay
// a dependent memory round trip per lookup.
struct OwnerTable {
  int n;        // owner layers in the block
  int layer0, n_layers, period, start;
  int n_pre;    // owners below `start` (each its own owner): local layers [0, n_pre)
  int j0;       // first shared owner: absolute layer start + period * j0

  // local layer of owner o (0 <= o < n)
  __host__ __device__ int local(int o) const {
    return o < n_pre ? o : start + period * (j0 + o - n_pre) - layer0;
  }
  // owner index of local layer l, or -1 when its owner precedes the block
  __host__ __device__ int index_of(int l) const {
    const int abs = layer0 + l;
    if (period <= 1 || abs < start) return l;
    const int j = (abs - start) / period;
    return start + period * j < layer0 ? -1 : n_pre + j - j0;
  }
  // end (exclusive local layer) of the layers that share owner o's selection
  __host__ __device__ int end(int o) const {
    if (o < n_pre) return o + 1;
    const int e = local(o) + period;
    return e < n_layers ? e : n_layers;
  }
};

inline OwnerTable owner_table(int layer0, int n_layers, int period, int start) {
  OwnerTable t{};
  t.layer0 = layer0;
  t.n_layers = n_layers;
  t.period = period;
  t.start = start;
  if (period <= 1) {
    t.n_pre = t.n = n_layers;
    return t;
  }
  const int end = layer0 + n_layers, a0 = layer0 > start ? layer0 : start;
  t.n_pre = (end < start ? end : start) - layer0;
  if (t.n_pre < 0) t.n_pre = 0;
  t.j0 = (a0 - start + period - 1) / period;
  const int n_sh = end > start ? (end - start + period - 1) / period - t.j0 : 0;
  t.n = t.n_pre + (n_sh > 0 ? n_sh : 0);
  return t;
}

template <class T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Data-parallel-primitive (DPP) lane moves: plain VALU operations, no LDS round trip.
//   0x121..0x12F  row_ror:1..15   rotate right within each row of 16 lanes
//   0x141         row_half_mirror reverse the order within each half-row of 8 lanes
//   0x4E / 0xB1   quad_perm       lane ^ 2 / lane ^ 1 within each quad
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(x), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(x), CTRL, 0xF, 0xF, false);
  return __hiloint2double(hi, lo);
}

// Sum over aligned groups of N consecutive lanes; every lane of a group receives its group's sum.
// Each step adds a lane permutation that pairs partial sums, so after log2(N) steps every lane
// has seen all N inputs (rotations by 8, 4, 2, 1 within 16 lanes; mirror + quad swaps within 8).
template <int N, class T>
__device__ __forceinline__ T group_sum(T x) {
  static_assert(N == 1 || N == 2 || N == 4 || N == 8 || N == 16 || N == 32 || N == 64, "group size");
  auto mv = [](auto v, auto ctrl_tag) {
    constexpr int C = decltype(ctrl_tag)::value;
    if constexpr (sizeof(T) == 8) return dpp_f64<C>(v); else return dpp_f32<C>(v);
  };
  using I = int;
  if constexpr (N == 2) {
    x += mv(x, std::integral_constant<I, 0xB1>{});
  } else if constexpr (N == 4) {
    x += mv(x, std::integral_constant<I, 0x4E>{});
    x += mv(x, std::integral_constant<I, 0xB1>{});
  } else if constexpr (N == 8) {
    x += mv(x, std::integral_constant<I, 0x141>{});
    x += mv(x, std::integral_constant<I, 0x4E>{});
    x += mv(x, std::integral_constant<I, 0xB1>{});
  } else if constexpr (N >= 16) {
    x += mv(x, std::integral_constant<I, 0x128>{});
    x += mv(x, std::integral_constant<I, 0x124>{});
    x += mv(x, std::integral_constant<I, 0x122>{});
    x += mv(x, std::integral_constant<I, 0x121>{});
    if constexpr (N >= 32) x += __shfl_xor(x, 16);
    if constexpr (N == 64) x += __shfl_xor(x, 32);
  }
  return x;
}

}  // namespace mpc
