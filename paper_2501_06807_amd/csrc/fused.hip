// One decode step in one launch: two-level selection of every owner head and sparse attention of
// every (layer, sequence, kv head), gfx950.
//
// One workgroup per attention unit, in unit order. A unit whose layer is owned inside the block
// consumes its owner head's selection. The first consumer to arrive claims the head (state 0 -> 1
// by compare-and-swap), computes the selection, publishes it and then attends; later consumers
// wait until the head is published. A consumer only ever waits for a head claimed by a workgroup
// that is already running and waits on nothing itself, so every wait ends without any assumption
// on the order in which workgroups are dispatched. The selection is written with device-coherent
// stores (sc1, write-through of the per-die L2), their completion is awaited, then the state word
// is published with another device-coherent store; consumers poll it and read the selection with
// device-coherent loads, so no L2 write-back fence is needed. The last consumer of a head returns
// its words to zero for the next launch. A bounded poll turns a lost publication into an error
// bit and NaN outputs of the units that gave up, never a hang.
#include "decode_dev.h"
#include "fused.h"
#include "select_dev.h"

namespace mpc {
namespace {

constexpr int kFusedWaves = 8;
constexpr int kSpinLimit = 1 << 20;  // polls (each ~0.1-1 us) before a unit gives up

template <class DT, int D, int G, bool MP, bool GMAX>
__global__ __launch_bounds__(kFusedWaves* kWave) void k_decode_step(FusedArgs f) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int s_mode;  // 1 select then attend, 2 attend, 0 gave up
  const int tid = threadIdx.x;
  const SelectArgs& sa = f.s;
  const int BH = sa.B * sa.Hkv;
  const int unit = blockIdx.x;  // (l * B + b) * Hkv + h
  const int l = unit / BH;
  const int o = sa.own.index_of(l);  // owner index of layer l (-1: owned before the block, its
                                     // selection is an input)
  const int head = o >= 0 ? o * BH + unit % BH : -1;  // (owner index * B + b) * Hkv + h

  if (tid == 0) {
    int mode = 2;
    if (head >= 0) {
      int st = __hip_atomic_load(&f.state[head], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (st == 0 && __hip_atomic_compare_exchange_strong(&f.state[head], &st, 1, __ATOMIC_RELAXED,
                                                          __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
        mode = 1;
      } else {
        for (int it = 0; st != 2; ++it) {
          if (it == kSpinLimit) {
            atomicOr(&f.sync->error, 1);
            mode = 0;
            break;
          }
          __builtin_amdgcn_s_sleep(4);
          st = __hip_atomic_load(&f.state[head], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    }
    s_mode = mode;
  }
  __syncthreads();
  const int mode = s_mode;
  if (mode == 1) {
    // one row pass in flight per wave and the query in LDS keep the selection's registers near
    // the attention's
    dev::select_block<DT, D, kFusedWaves, true, 1, MP, false, GMAX>(sa, head, smem);
    __builtin_amdgcn_s_waitcnt(0);  // this thread's selection stores have completed
    __syncthreads();
    if (tid == 0) __hip_atomic_store(&f.state[head], 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  // K rows stream past the caches too: the representatives that selections of this same launch
  // are still reading stay resident
  if (mode != 0) {
    dev::attend<DT, D, G, kFusedWaves, 4, true, true>(f.d, unit, 0);
  } else {
    // the selection never arrived: the unit's outputs become NaN, so they cannot pass for a result
    const float nan = __builtin_nanf("");
    for (int i = tid; i < G * D; i += kFusedWaves * kWave) store_elt<DT>(f.d.out, (size_t)unit * G * D + i, nan);
    if (tid < G && f.d.lse) f.d.lse[(size_t)unit * G + tid] = nan;
  }

  if (head >= 0) {
    __syncthreads();
    if (tid == 0) {
      __builtin_amdgcn_s_waitcnt(0);  // the publication above has completed
      const int lb = sa.own.local(o), le = sa.own.end(o);
      const int c = __hip_atomic_fetch_add(&f.cons[head], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (c == le - lb - 1) {  // last consumer of the head
        __hip_atomic_store(&f.state[head], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&f.cons[head], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
}

// Self-selecting form (blocks of at most one attention unit per compute unit, attention not split):
// every workgroup computes the selection of its unit's owner head itself and attends over it from
// LDS. Workgroups never wait for one another; the two to four units that share an owner head
// compute the same selection side by side, reading its representatives through one L2.
constexpr int kDies = 8;  // compute dies (XCDs); workgroup p of a launch runs on die p % kDies

// Unit of workgroup p: ranks i of the owner-major order (all units of one owner head, then the next
// head) are dealt to the dies in contiguous runs, so the units that select alike share a die's L2.
// Returns -1 for the padding positions of the last run.
__device__ __forceinline__ int self_unit(const SelectArgs& s, int p) {
  const int BH = s.B * s.Hsel, n_units = s.n_layers * BH;
  const int per = (n_units + kDies - 1) / kDies;
  const int i = (p % kDies) * per + p / kDies;
  if (i >= n_units) return -1;
  // owner group of rank i: layers [lb, le) that share one selection (or, before the first owner
  // of the block, layers whose selection is an input); a group's ranks are [lb * BH, le * BH), so it
  // is the group of layer i / BH
  const int o = s.own.index_of(i / BH);
  const int lb = o >= 0 ? s.own.local(o) : 0;
  const int le = o >= 0 ? s.own.end(o) : (s.own.n > 0 ? s.own.local(0) : s.n_layers);
  const int il = i - lb * BH, n = le - lb;
  return (lb + il % n) * BH + il / n;
}

template <class DT, int D, int G, bool MP, bool GMAX, bool STREAM_K>
__global__ __launch_bounds__(kFusedWaves* kWave) void k_decode_self(FusedArgs f) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int32_t s_pick[dev::kMaxSel];
  const SelectArgs& sa = f.s;
  const int unit = self_unit(sa, blockIdx.x);  // (l * B + b) * Hsel + h
  if (unit < 0) return;
  const int BH = sa.B * sa.Hsel, l = unit / BH;
  const int o = sa.own.index_of(l);  // -1: owned before the block, its selection is an input
  if (o >= 0) {
    dev::select_block<DT, D, kFusedWaves, false, 2, MP, true, GMAX>(sa, o * BH + unit % BH, smem, s_pick, l);
    __syncthreads();
  }
  dev::attend<DT, D, G, kFusedWaves, 4, false, STREAM_K>(f.d, unit, 0, o >= 0 ? s_pick : nullptr);
}

template <class DT, int D, int G, bool MP, bool GMAX>
void launch_self(const FusedArgs& f, size_t smem, hipStream_t st) {
  const int units = f.s.n_layers * f.s.B * f.s.Hsel;
  const dim3 grid((units + kDies - 1) / kDies * kDies), block(kFusedWaves * kWave);
  if (f.d.stream_k)
    hipLaunchKernelGGL((k_decode_self<DT, D, G, MP, GMAX, true>), grid, block, smem, st, f);
  else
    hipLaunchKernelGGL((k_decode_self<DT, D, G, MP, GMAX, false>), grid, block, smem, st, f);
}

template <class DT, int D, int G>
hipError_t launch_claim(const FusedArgs& f, size_t smem, hipStream_t st) {
  const dim3 grid(f.s.n_layers * f.s.B * f.s.Hkv), block(kFusedWaves * kWave);
  const bool mp = f.s.similarity == MPC_SIM_MAXPROD;
  if constexpr (G > 1) {
    if (f.s.group == MPC_GROUP_MAX) {
      if (mp)
        hipLaunchKernelGGL((k_decode_step<DT, D, G, true, true>), grid, block, smem, st, f);
      else
        hipLaunchKernelGGL((k_decode_step<DT, D, G, false, true>), grid, block, smem, st, f);
      return hipGetLastError();
    }
  }
  if (mp)
    hipLaunchKernelGGL((k_decode_step<DT, D, G, true, false>), grid, block, smem, st, f);
  else
    hipLaunchKernelGGL((k_decode_step<DT, D, G, false, false>), grid, block, smem, st, f);
  return hipGetLastError();
}

template <class DT, int D, int G>
hipError_t launch_g(const FusedArgs& f, const FusedPlan& p, hipStream_t st) {
  const size_t smem = p.smem;
  const bool mp = f.s.similarity == MPC_SIM_MAXPROD;
  const bool gmax = G > 1 && f.s.group == MPC_GROUP_MAX;
  if (p.self) {
    if constexpr (G > 1) {
      if (gmax) {
        mp ? launch_self<DT, D, G, true, true>(f, smem, st) : launch_self<DT, D, G, false, true>(f, smem, st);
        return hipGetLastError();
      }
    }
    mp ? launch_self<DT, D, G, true, false>(f, smem, st) : launch_self<DT, D, G, false, false>(f, smem, st);
    return hipGetLastError();
  }
  return launch_claim<DT, D, G>(f, smem, st);
}

template <class DT, int D>
hipError_t launch_d(const FusedArgs& f, int G, const FusedPlan& p, hipStream_t st) {
  switch (G) {
    case 1: return launch_g<DT, D, 1>(f, p, st);
    case 2: return launch_g<DT, D, 2>(f, p, st);
    case 4: return launch_g<DT, D, 4>(f, p, st);
    case 8: return launch_g<DT, D, 8>(f, p, st);
  }
  return hipErrorInvalidValue;
}

template <class DT>
hipError_t launch_dt(const FusedArgs& f, int D, int G, const FusedPlan& p, hipStream_t st) {
  if (D == 64) return launch_d<DT, 64>(f, G, p, st);
  if (D == 128) return launch_d<DT, 128>(f, G, p, st);
  return hipErrorInvalidValue;
}

}  // namespace

FusedPlan fused_plan(const SelectArgs& s, int D, int splits) {
  FusedPlan p{};
  p.units = s.n_layers * s.B * s.Hsel;
  p.smem = dev::select_smem_bytes_dev(D, s.S, s.NC, select_query_rows(s));
  p.self = p.units <= kNumCU && splits == 1;
  return p;
}

bool fused_fits(const FusedPlan& p, int D, int G) {
  // the attention's static LDS: selection ids, per-wave (m, l) and partial outputs, a few words;
  // the self-selecting form holds its selection ids once more
  const size_t att = 4 * dev::kMaxSel * (p.self ? 2 : 1) + (size_t)kFusedWaves * G * (2 + D) * 4 + 64;
  return p.smem + att <= kMaxLds;
}

hipError_t launch_decode_step(const FusedArgs& f, const FusedPlan& p, int dtype, int D, int G,
                              hipStream_t st) {
  switch (dtype) {
    case MPC_FP32: return launch_dt<F32>(f, D, G, p, st);
    case MPC_FP16: return launch_dt<F16>(f, D, G, p, st);
    case MPC_BF16: return launch_dt<BF16>(f, D, G, p, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace mpc
