// Measured ceilings for the roofline context (not part of the method). Read ceiling of the decode
// kernels:
// every workgroup reads `per_wg` contiguous chunks of `chunk_bytes`, taken in a caller-given
// (random) order, with 16-byte coalesced non-temporal loads, four in flight per thread — the access
// pattern of the sparse attention, which reads whole clusters of K / V rows with the same hint. One XOR per thread is written to
// `sink` so that the loads are kept. Matrix-core ceiling of the static-scoring passes: every wave
// runs chains of the bf16 32x32x16 matrix instruction on register operands, four independent
// accumulators in flight, and writes its accumulators to `sink`.
#include <hip/hip_runtime.h>
#include <cstdint>

namespace {

constexpr int kThreads = 256;
constexpr int kInFlight = 4;

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_stream(const uint4* p) {
  const u32x4_t v = __builtin_nontemporal_load((const u32x4_t*)p);
  return make_uint4(v.x, v.y, v.z, v.w);
}

__global__ __launch_bounds__(kThreads) void k_read_chunks(const uint4* __restrict__ buf,
                                                          const int32_t* __restrict__ order, int per_wg,
                                                          int chunk16, uint32_t* __restrict__ sink) {
  uint32_t acc = 0;
  const int n = per_wg * chunk16;  // 16-byte vectors of this workgroup
  const int32_t* mine = order + (size_t)blockIdx.x * per_wg;
  int j = threadIdx.x;
  for (; j + (kInFlight - 1) * kThreads < n; j += kInFlight * kThreads) {
    uint4 v[kInFlight];
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      const int jj = j + u * kThreads;
      v[u] = load_stream(buf + (size_t)mine[jj / chunk16] * chunk16 + jj % chunk16);
    }
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; j < n; j += kThreads) {
    const uint4 v = load_stream(buf + (size_t)mine[j / chunk16] * chunk16 + j % chunk16);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  sink[(size_t)blockIdx.x * kThreads + threadIdx.x] = acc;
}

typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
constexpr int kChains = 4;

__global__ __launch_bounds__(kThreads) void k_mfma(int iters, float seed, float* __restrict__ sink) {
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(seed * (float)(threadIdx.x + i));
    b[i] = (__bf16)(seed * (float)(blockIdx.x - i));
  }
  f32x16 acc[kChains];
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[c][i] = 0.f;
#pragma unroll 4
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
  }
  float t = 0.f;
#pragma unroll
  for (int c = 0; c < kChains; ++c)
#pragma unroll
    for (int i = 0; i < 16; ++i) t += acc[c][i];
  sink[(size_t)blockIdx.x * kThreads + threadIdx.x] = t;
}

}  // namespace

// grid workgroups of 256 threads, each wave running `iters` x 4 matrix instructions (32768 flop
// each); sink: grid * 256 floats. Returns a hipError_t code (0 = launched).
extern "C" int mpc_mfma_ceiling(int grid, int iters, float* sink, void* stream) {
  if (!sink || grid <= 0 || iters <= 0) return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_mfma, dim3(grid), dim3(kThreads), 0, (hipStream_t)stream, iters, 1e-3f, sink);
  return (int)hipGetLastError();
}

// buf: n_chunks * chunk_bytes bytes; order: grid * per_wg chunk ids in [0, n_chunks); sink: grid *
// 256 words. Returns a hipError_t code (0 = launched).
extern "C" int mpc_read_ceiling(const void* buf, int64_t n_chunks, int chunk_bytes, const int32_t* order, int grid,
                                int per_wg, uint32_t* sink, void* stream) {
  if (!buf || !order || !sink || chunk_bytes <= 0 || chunk_bytes % 16 || grid <= 0 || per_wg <= 0 ||
      (int64_t)grid * per_wg > n_chunks || (int64_t)per_wg * (chunk_bytes / 16) >= ((int64_t)1 << 31))
    return (int)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_read_chunks, dim3(grid), dim3(kThreads), 0, (hipStream_t)stream, (const uint4*)buf, order,
                     per_wg, chunk_bytes / 16, sink);
  return (int)hipGetLastError();
}
