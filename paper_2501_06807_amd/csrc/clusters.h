// Launch interface of the cluster-representative kernel.
#pragma once
#include "common.h"

namespace mpc {

// Prefill mode: the rows of the kept cache are gathered from the prompt cache on their way into
// the representatives (one pass over the kept keys instead of a gather and a re-read).
struct BuildGather {
  int32_t* kept;         // [L][B][Hkv][keep]: a layer's kept set is read from its eviction owner's
                         // and, for a sharing layer, copied into its own slot
  const void* k_src;     // [L][B][Hkv][T][d] prompt cache
  const void* v_src;
  void* k_dst;           // [L][B][Hkv][rows][d] kept cache, rows [0, keep) written
  void* v_dst;
  int T, keep;
  int period, start;     // sharing rule of the kept sets
};

struct BuildArgs {
  const void* k;   // [L][B][Hkv][rows][d] (unused in prefill mode)
  float* cent;     // [L][B][Hkv][cs][R][d]  (R = 2 for the max-product bound, else 1)
  float* scent;    // [L][B][Hkv][ss][R][d]
  int B, layer0, n_layers, Hkv, Ts, s, f, C, S, period, start;
  int rows, cs, ss;   // allocated rows / cluster slots / super-cluster slots per (layer, sequence, head)
  int sup0, n_sup;    // super-clusters [sup0, sup0 + n_sup) are (re)built
  int similarity;     // mpc_similarity
  float alpha, beta;  // beta = fp32(1 - alpha)
  OwnerTable own;
  BuildGather g;      // prefill mode when g.kept is set (then Ts = keep, sup0 = 0, n_sup = S)
};

hipError_t launch_build(const BuildArgs& a, int dtype, int D, hipStream_t st);

}  // namespace mpc
