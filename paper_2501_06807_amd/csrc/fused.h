// Launch interface of the fused decode-step kernel (selection + sparse attention, one launch).
#pragma once
#include "decode_attn.h"
#include "select.h"

namespace mpc {

// Ticket counters at the start of the fused workspace; zero before first use, left zero (with the
// epoch advanced) by every completed launch. Owner-head flags follow.
struct FusedSync {
  int ticket;
  int done;
  int epoch;
  int error;  // bit 0: an attention item gave up waiting (never expected)
};

struct FusedArgs {
  SelectArgs s;
  DecodeArgs d;
  FusedSync* sync;
  int* flags;  // [owner heads]
  int total;   // workgroups = tickets
};

struct FusedPlan {
  bool wave_select;
  int total;
  size_t smem;
};

FusedPlan fused_plan(const SelectArgs& s, int D);
hipError_t launch_decode_step(const FusedArgs& f, const FusedPlan& p, int dtype, int D, int G,
                              hipStream_t st);

}  // namespace mpc
