// Launch interface of the sparse decode attention kernel.
#pragma once
#include "common.h"

namespace mpc {

constexpr int kMaxSplits = 16;   // split-K limit (workspace bound)

struct DecodeArgs {
  const void* q;       // [L][B][Hq][d]
  const void* k;       // [L][B][cache_heads][rows][d]
  const void* v;
  const int32_t* sel;  // [L][B][Hkv][k_sel] (one list per unit)
  void* out;           // [L][B][Hq][d]
  float* lse;          // [L][B][Hq] or null
  float* part;         // split-K partials [units][splits][G][d + 2]
  int* cnt;            // split-K arrival counters [units], zero between launches
  int Ts, s, C, k_sel, Hq, splits;  // C = ceil(Ts / s) selectable clusters
  int Hkv;          // selection lists (work units) per (layer, sequence): the kv heads, or the
                    // q-heads when every q-head has its own list (then G = 1 per unit)
  int cache_heads;  // kv heads of the cache per (layer, sequence)
  int cache_div;    // unit head h reads the rows of cache head h / cache_div
  int rows;            // allocated rows per (layer, sequence, kv head)
  int n_tail;          // rows [Ts, Ts + n_tail) attended by every head (Ts % s == 0 if n_tail > 0)
  float qscale;        // sm_scale * log2(e)
  int stream_kv;       // 1: the gathered K / V rows are loaded with the non-temporal hint
};

// Gathered K / V bytes of one call above which the rows are loaded with the non-temporal hint:
// half the 256 MB memory-side cache. Smaller calls keep them cached, since the next decode step
// selects many of the same clusters again; larger ones would only displace the representatives
// the next selection reads.
constexpr long long kStreamKvBytes = 128ll << 20;

struct DecodePlan {
  int waves;   // waves per workgroup
  int splits;  // workgroups per unit
};
DecodePlan decode_plan(int units, int n_slot, int D, int elt);
hipError_t launch_sparse_decode(const DecodeArgs& a, int dtype, int D, int G, int units, const DecodePlan& p,
                                hipStream_t st);

}  // namespace mpc
