// Launch interface of the fused decode-step kernel (selection + sparse attention, one launch).
#pragma once
#include "decode_attn.h"
#include "select.h"

namespace mpc {

// Workspace of the fused kernel: a sticky error word, then per owner head a state word
// (0 free, 1 being selected, 2 published) and a consumer count. Zero before first use; every
// completed launch leaves the per-head words at zero again.
struct FusedSync {
  int error;  // bit 0: an attention unit gave up waiting for its selection (never expected)
};

struct FusedArgs {
  SelectArgs s;
  DecodeArgs d;
  FusedSync* sync;
  int* state;  // [owner heads]
  int* cons;   // [owner heads]
};

struct FusedPlan {
  int units;
  size_t smem;
  bool self;  // every workgroup selects for its own unit (no waits; no workspace words used)
};

// splits: workgroups per attention unit of the block's attention plan.
FusedPlan fused_plan(const SelectArgs& s, int D, int splits);
// Whether the selection's LDS and the attention's fit one workgroup's LDS together.
bool fused_fits(const FusedPlan& p, int D, int G);
hipError_t launch_decode_step(const FusedArgs& f, const FusedPlan& p, int dtype, int D, int G,
                              hipStream_t st);

}  // namespace mpc
