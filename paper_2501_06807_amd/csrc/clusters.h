// Launch interface of the cluster-representative kernel.
#pragma once
#include "common.h"

namespace mpc {

struct BuildArgs {
  const void* k;   // [L][B][Hkv][Ts][d]
  float* cent;     // [L][B][Hkv][C][d]
  float* scent;    // [L][B][Hkv][S][d]
  int B, layer0, n_layers, Hkv, Ts, s, f, C, S, period, start;
  float alpha, beta;  // beta = fp32(1 - alpha)
  OwnerTable own;
};

hipError_t launch_build(const BuildArgs& a, int dtype, int D, hipStream_t st);

}  // namespace mpc
