// Decode-time append of one token's k and v to every (layer, sequence, kv head) of the kept
// cache: one 16-byte vector per thread, coalesced on both sides.
#include "append.h"

namespace mpc {
namespace {

constexpr int kAppendThreads = 256;

__global__ __launch_bounds__(kAppendThreads) void k_append_rows(AppendArgs a) {
  const int vec = a.row_bytes / 16;  // vectors per row
  const int64_t n = a.units * vec;   // vectors of k (then as many of v)
  const int64_t i = (int64_t)blockIdx.x * kAppendThreads + threadIdx.x;
  if (i >= 2 * n) return;
  const bool is_v = i >= n;
  const int64_t j = is_v ? i - n : i;
  const int64_t unit = j / vec;
  const int c = (int)(j % vec);
  const char* src = (const char*)(is_v ? a.v_new : a.k_new) + (size_t)j * 16;
  char* dst = (char*)(is_v ? a.v : a.k) + (((size_t)unit * a.rows + a.row) * vec + c) * 16;
  *(uint4*)dst = ldg16(src);
}

}  // namespace

hipError_t launch_append_rows(const AppendArgs& a, hipStream_t st) {
  const int64_t threads = 2 * a.units * (a.row_bytes / 16);
  const int64_t blocks = (threads + kAppendThreads - 1) / kAppendThreads;
  if (blocks >= ((int64_t)1 << 31)) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_append_rows, dim3((unsigned)blocks), dim3(kAppendThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace mpc
