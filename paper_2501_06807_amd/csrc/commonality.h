// Launch interface of the commonality score of adjacent layers' top-k sets.
#pragma once
#include "common.h"

namespace mpc {

constexpr int kCommonMaxK = 1024;  // set size limit (the scan per membership test is O(k))

hipError_t launch_commonality(int L, int units, int k, int m, const int32_t* idx, double* out, hipStream_t st);

}  // namespace mpc
