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
  int stream_k;        // 1: the gathered K rows too are loaded with the non-temporal hint (V rows
                       // always are)
};

// Working set of one decode step above which the gathered K rows are loaded with the non-temporal
// hint: the 256 MB memory-side cache. The working set is the call's K rows plus the fine-cluster
// representatives of its units, which the next selection reads. While both fit, the K rows stay
// cacheable, since later steps select many of the same clusters again; beyond it they would only
// displace the representatives. V rows are read once, after their scores, and always stream.
constexpr long long kStreamKBytes = 256ll << 20;

struct DecodePlan {
  int waves;   // waves per workgroup
  int splits;  // workgroups per unit
};
DecodePlan decode_plan(int units, int n_slot, int D, int elt);
hipError_t launch_sparse_decode(const DecodeArgs& a, int dtype, int D, int G, int units, const DecodePlan& p,
                                hipStream_t st);

}  // namespace mpc
