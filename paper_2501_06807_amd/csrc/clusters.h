// Launch interface of the cluster-representative kernel.
#pragma once
#include "common.h"

namespace mpc {

struct BuildArgs {
  const void* k;   // [L][B][Hkv][rows][d]
  float* cent;     // [L][B][Hkv][cs][R][d]  (R = 2 for the max-product bound, else 1)
  float* scent;    // [L][B][Hkv][ss][R][d]
  int B, layer0, n_layers, Hkv, Ts, s, f, C, S, period, start;
  int rows, cs, ss;   // allocated rows / cluster slots / super-cluster slots per (layer, sequence, head)
  int sup0, n_sup;    // super-clusters [sup0, sup0 + n_sup) are (re)built
  int similarity;     // mpc_similarity
  float alpha, beta;  // beta = fp32(1 - alpha)
  OwnerTable own;
};

hipError_t launch_build(const BuildArgs& a, int dtype, int D, hipStream_t st);

}  // namespace mpc
