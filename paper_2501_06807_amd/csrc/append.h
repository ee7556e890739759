// Launch interface of the decode-time row append.
#pragma once
#include "common.h"

namespace mpc {

struct AppendArgs {
  const void* k_new;  // [units][d]
  const void* v_new;
  void* k;            // [units][rows][d]
  void* v;
  int64_t units;      // (layer, sequence, kv head) triples
  int rows;           // allocated rows per unit
  int row;            // row written
  int row_bytes;      // d * element size (a multiple of 16)
};

hipError_t launch_append_rows(const AppendArgs& a, hipStream_t st);

}  // namespace mpc
