// One decode step in one launch: two-level selection of every owner head and sparse attention of
// every (layer, sequence, kv head), gfx950.
//
// Every workgroup takes a ticket when it starts. The selection items of all owner heads hold the
// first tickets, the attention items follow in layer order (layers whose owner precedes the block
// first: their selection is an input). An attention item waits for its owner head's flag; that
// head's selection item holds a smaller ticket, so it was taken by a workgroup that is already
// running and never waits: the wait always ends. The selection is published with device-coherent stores (sc1, which write through the
// per-die L2), their completion awaited, then the flag is raised with another device-coherent
// store; readers poll the flag and read the selection with device-coherent loads. No L2
// write-back fence is needed. A bounded poll turns a lost flag into an error bit, never a hang.
#include "decode_dev.h"
#include "fused.h"
#include "select_dev.h"

namespace mpc {
namespace {

constexpr int kFusedWaves = 8;
constexpr int kSpinLimit = 1 << 20;  // polls (each ~0.1-1 us) before an item gives up

template <class DT, int D, int G, bool WAVE_SELECT>
__global__ __launch_bounds__(kFusedWaves* kWave) void k_decode_step(FusedArgs f) {
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int s_ticket, s_epoch, s_go;
  const int tid = threadIdx.x;
  if (tid == 0) {
    s_ticket = atomicAdd(&f.sync->ticket, 1);
    s_epoch = __hip_atomic_load(&f.sync->epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_go = 1;
  }
  __syncthreads();
  const int epoch = s_epoch;
  const SelectArgs& sa = f.s;
  const int BH = sa.B * sa.Hkv;
  const int hps = WAVE_SELECT ? kFusedWaves : 1;  // owner heads per selection item
  const int n_heads = sa.own.n * BH;               // owner heads, (owner index * B + b) * Hkv + h
  const int t = s_ticket;

  // decode the ticket: [selection items of every owner head][attention items in layer order]
  int kind, unit = 0, head = -1, ou0 = 0;
  const int sel_items = (n_heads + hps - 1) / hps;
  if (t < sel_items) {
    kind = 0;
    ou0 = t * hps;
  } else {
    kind = 1;
    unit = t - sel_items;
    const int l = unit / BH;
    int o = -1;  // owner index of layer l (none: owned before the block, selection is an input)
    for (int i = 0; i < sa.own.n && sa.own.l[i] <= l; ++i) o = i;
    if (o >= 0) head = o * BH + unit % BH;
  }

  if (kind == 0) {
    if constexpr (WAVE_SELECT)
      dev::select_waves<DT, D, true>(sa, ou0, smem);
    else
      dev::select_block<DT, D, kFusedWaves, true>(sa, ou0, smem);
    __builtin_amdgcn_s_waitcnt(0);  // this thread's selection stores have completed
    __syncthreads();
    if (tid == 0)
      for (int i = 0; i < hps && ou0 + i < n_heads; ++i)
        __hip_atomic_store(&f.flags[ou0 + i], epoch + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  } else if (kind == 1) {
    if (head >= 0 && tid == 0) {
      int it = 0;
      while (__hip_atomic_load(&f.flags[head], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != epoch + 1) {
        __builtin_amdgcn_s_sleep(4);
        if (++it > kSpinLimit) {
          atomicOr(&f.sync->error, 1);
          s_go = 0;
          break;
        }
      }
    }
    __syncthreads();
    if (s_go) dev::attend_unit<DT, D, G, kFusedWaves, 4, true>(f.d, unit, 0);
  }

  // the last workgroup to finish resets the ticket counters for the next launch
  __syncthreads();
  if (tid == 0) {
    const int d = atomicAdd(&f.sync->done, 1);
    if (d == f.total - 1) {
      __hip_atomic_store(&f.sync->ticket, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&f.sync->done, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&f.sync->epoch, epoch + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

template <class DT, int D, int G>
hipError_t launch_g(const FusedArgs& f, bool wave, size_t smem, hipStream_t st) {
  if (wave)
    hipLaunchKernelGGL((k_decode_step<DT, D, G, true>), dim3(f.total), dim3(kFusedWaves * kWave), smem, st, f);
  else
    hipLaunchKernelGGL((k_decode_step<DT, D, G, false>), dim3(f.total), dim3(kFusedWaves * kWave), smem, st, f);
  return hipGetLastError();
}

template <class DT, int D>
hipError_t launch_d(const FusedArgs& f, int G, bool wave, size_t smem, hipStream_t st) {
  switch (G) {
    case 1: return launch_g<DT, D, 1>(f, wave, smem, st);
    case 2: return launch_g<DT, D, 2>(f, wave, smem, st);
    case 4: return launch_g<DT, D, 4>(f, wave, smem, st);
    case 8: return launch_g<DT, D, 8>(f, wave, smem, st);
  }
  return hipErrorInvalidValue;
}

template <class DT>
hipError_t launch_dt(const FusedArgs& f, int D, int G, bool wave, size_t smem, hipStream_t st) {
  if (D == 64) return launch_d<DT, 64>(f, G, wave, smem, st);
  if (D == 128) return launch_d<DT, 128>(f, G, wave, smem, st);
  return hipErrorInvalidValue;
}

}  // namespace

FusedPlan fused_plan(const SelectArgs& s, int D) {
  FusedPlan p{};
  const int BH = s.B * s.Hkv;
  const int heads = s.own.n * BH;
  p.wave_select = heads >= 512 && s.S <= dev::kWaveMaxSuper && s.NC <= dev::kWaveMaxCand;
  const int hps = p.wave_select ? kFusedWaves : 1;
  p.total = s.n_layers * BH + (s.own.n * BH + hps - 1) / hps;
  p.smem = p.wave_select ? kFusedWaves * dev::wave_region_bytes(s.S, s.NC)
                         : dev::select_smem_bytes_dev(D, s.S, s.NC);
  return p;
}

hipError_t launch_decode_step(const FusedArgs& f, const FusedPlan& p, int dtype, int D, int G,
                              hipStream_t st) {
  switch (dtype) {
    case MPC_FP32: return launch_dt<F32>(f, D, G, p.wave_select, p.smem, st);
    case MPC_FP16: return launch_dt<F16>(f, D, G, p.wave_select, p.smem, st);
    case MPC_BF16: return launch_dt<BF16>(f, D, G, p.wave_select, p.smem, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace mpc
