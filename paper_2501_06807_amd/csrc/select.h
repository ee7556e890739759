// Launch interface of the two-level cluster selection kernel.
#pragma once
#include "common.h"

namespace mpc {

constexpr int kSelMaxSuper = 1024;  // S limit (LDS)
constexpr int kSelMaxCand = 1024;   // k_super * fanout limit (LDS)

struct SelectArgs {
  const void* q;        // [L][B][Hq][d]
  const float* cent;    // [L][B][Hkv][cs][R][d], the first C slots used
  const float* scent;   // [L][B][Hkv][ss][R][d], the first S slots used
  int32_t* sel;         // [L][B][Hsel][k_clusters]
  float* sel_score;     // same or null
  int B, layer0, n_layers, Hq, Hkv;
  int Hsel;     // selection units per (layer, sequence): Hq when every q-head selects, else Hkv
  int rep_div;  // selection unit h reads the representatives of kv head h / rep_div
  int C, S, f, NC, k_super, k_clusters;  // NC = k_super * f
  int cs, ss;                            // allocated cluster / super-cluster slots per head
  int period, start;
  int similarity;  // mpc_similarity: representatives of 2 rows (r^max, r^min) for the bound
  int group;       // mpc_group: how the q-heads of a unit combine (sum, maximum, one head)
  OwnerTable own;  // owner layers of the block (one workgroup per owner head)
};

size_t select_smem_bytes(int D, int S, int NC, int qrows);  // qrows: 1, or the unit's q-heads
int select_query_rows(const SelectArgs& a);  // query rows a unit keeps in LDS
hipError_t launch_select(const SelectArgs& a, int dtype, int D, hipStream_t st);

}  // namespace mpc
