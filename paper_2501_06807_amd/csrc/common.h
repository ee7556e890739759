// Shared device helpers for the gfx950 kernels: element types, 16-byte vector loads, wave
// reductions. Wavefronts are 64 lanes wide.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/mpcache.h"

namespace mpc {

constexpr int kWave = 64;

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

// Owner layer of an absolute layer index (cross-layer index sharing).
__host__ __device__ __forceinline__ int owner_layer(int l, int period, int start) {
  if (period <= 1 || l < start) return l;
  return start + period * ((l - start) / period);
}

template <class T>
__device__ __forceinline__ T wave_sum(T v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

}  // namespace mpc
