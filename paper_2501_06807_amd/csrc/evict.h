// Launch interface of the static-eviction kernels.
#pragma once
#include "common.h"

namespace mpc {

constexpr int kNumXcd = 8;       // accelerator dies; workgroup i runs on die i % 8
constexpr int kRowBlock = 256;      // window rows per row-statistics workgroup
constexpr int kColBlockKeys = 256;  // keys per column-sum workgroup (its waves share each staged row tile)
constexpr int kColThreads16 = 256;  // column-sum workgroup for 16-bit inputs: 4 waves of 64 keys
constexpr int kRowThreads16 = 256;  // row-statistics workgroup for 16-bit inputs: 4 waves of 64 rows

struct EvictArgs {
  const void* q_win;   // [L][B][Hq][W][d]
  const void* k;       // [L][B][Hkv][T][d]
  const void* v;
  int32_t* kept;       // [L][B][Hkv][keep]
  void* k_out;         // [L][B][Hkv][out_rows][d], rows [0, keep) written
  void* v_out;
  float* score;        // [L][B][Hkv][T] accumulated attention (token_score or workspace)
  float2* rowstat;     // [L][B][Hq][W]: (whole-number offset b, every fma(c, score, b) <= 1; 1 / sum of exp2(fma(c, score, b)))
  float* row_lse;      // [L][B][Hq][W] natural log-sum-exp, optional
  int B, layer0, n_layers, Hq, Hkv, T, W, keep, local_keep, causal, period, start;
  int out_rows;        // row capacity of k_out / v_out per (layer, sequence, kv head)
  OwnerTable own;      // owner layers of the block
  uint64_t skip[kMaxLayers / 64];  // layers whose rows the gather leaves to the cluster build (bit l)
  float c32;           // fp32(sm_scale * log2(e)), the exponent scale of both scoring passes
};

hipError_t launch_rowstats(const EvictArgs& a, int dtype, int D, hipStream_t st);
hipError_t launch_colsum(const EvictArgs& a, int dtype, int D, hipStream_t st);
hipError_t launch_topk(const EvictArgs& a, hipStream_t st);
hipError_t launch_gather(const EvictArgs& a, int dtype, int D, hipStream_t st);

}  // namespace mpc
