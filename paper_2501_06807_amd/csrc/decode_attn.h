// Launch interface of the sparse decode attention kernel.
#pragma once
#include "common.h"

namespace mpc {

constexpr int kDecodeWaves = 8;          // waves per workgroup
constexpr int kDecodeTargetBlocks = 1024; // split-K aims for at least this many workgroups

struct DecodeArgs {
  const void* q;       // [L][B][Hq][d]
  const void* k;       // [L][B][Hkv][Ts][d]
  const void* v;
  const int32_t* sel;  // [L][B][Hkv][k_sel]
  void* out;           // [L][B][Hq][d]
  float* lse;          // [L][B][Hq] or null
  float* part;         // split-K partials [units][splits][G][d + 2]
  int32_t* counters;   // [units], zero between calls
  int Ts, s, k_sel, Hq, Hkv, splits;
  float qscale;        // sm_scale * log2(e)
};

int decode_splits(int units, int n_slot, int D, int elt);
hipError_t launch_sparse_decode(const DecodeArgs& a, int dtype, int D, int G, int units,
                                hipStream_t st);

}  // namespace mpc
