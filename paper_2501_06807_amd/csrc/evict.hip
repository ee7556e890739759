// Look-once static eviction on gfx950: accumulated window attention, top-k, gather.
//
// The accumulated attention of key j is A[j] = sum over the group's window rows t of
// softmax_j(sm_scale * q_t . k_j). It needs every row's normaliser before any column can be
// summed, so it takes two passes over the scores, both on the matrix cores (16-bit inputs:
// v_mfma_f32_16x16x32_{bf16,f16} blocks; fp32 inputs: v_mfma_f32_32x32x2f32):
//   pass 1 (k_rowstats16, k_rowstats for fp32): window rows stay in registers as the B operand,
//     key tiles stream through LDS as the A operand; each lane owns one query column of its
//     blocks, so a row's sum needs no exchange until the end. Output per row: a whole-number
//     offset b >= -ceil(fp32(c * m)) for the row max m with every exponent fma(c, s, b) at most 1
//     (b = -ceil(fp32(c * m)) for fp32 inputs), and 1 / sum of exp2(fma(c, s, b)),
//     c = fp32(sm_scale * log2(e)).
//   pass 2 (k_colsum16 for 16-bit inputs, k_colsum for fp32): keys stay in registers as the B
//     operand, window-row tiles (all query heads of the group) stream through LDS as the A
//     operand; each lane owns one key column, so the column sum needs no exchange within a tile.
//     p = exp2(fma(c, s, b)) / sum, summed over a lane's rows of a tile in fp32 and accumulated
//     across tiles in fp64. For 16-bit inputs both passes use 16x16 blocks and 64-row (64-key)
//     tiles, so that each block's exponentials overlap the next block's matrix chain within the
//     wave and a barrier serves 64 rows. Both passes form the exponent with one fused multiply-add
//     against the same offset, so the offset is a common factor of a row's terms and of its sum
//     and cancels in p; it only has to keep every exponent at or below about 1. Being a whole
//     number, a move of the offset rescales pass 1's sums by an exact power of two (ldexp). The
//     exponents of the terms near the max lie in (-1, 1], so their rounding, and that of c
//     (proportional to |c * (s - m)|), stay smallest on the terms that carry the sums.
// The top-k is a 4-pass, 8-bit LDS radix select on the fp32 score bits followed by an ordered
// block compaction, each thread's run of scores held in registers up to 32K older tokens; the
// gather copies kept rows with 16-byte lanes (all layers, or those whose representatives are not
// built in the same pass).
#include "evict.h"

#include <type_traits>

namespace mpc {
namespace {

typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef _Float16 f16x8 __attribute__((__vector_size__(8 * sizeof(_Float16))));

// Matrix-core operation per element type: reduction length K per instruction, KL elements per
// lane. Lane l feeds row (l % 32) of A / column (l % 32) of B with the k-slice
// [ks * K + (l / 32) * KL, + KL); any k-permutation works as long as A and B share it.
template <class DT>
struct Mma;
template <>
struct Mma<BF16> {
  static constexpr int K = 16, KL = 8;
  using Op = bf16x8;
  __device__ static f32x16 run(Op a, Op b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  __device__ static Op load(const void* p) { return __builtin_bit_cast(Op, *(const uint4*)p); }
};
template <>
struct Mma<F16> {
  static constexpr int K = 16, KL = 8;
  using Op = f16x8;
  __device__ static f32x16 run(Op a, Op b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
  }
  __device__ static Op load(const void* p) { return __builtin_bit_cast(Op, *(const uint4*)p); }
};
template <>
struct Mma<F32> {
  static constexpr int K = 2, KL = 1;
  using Op = float;
  __device__ static f32x16 run(Op a, Op b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  __device__ static Op load(const void* p) { return *(const float*)p; }
};

// 16x16x32 matrix-core operation for 16-bit inputs: lane l feeds row (l % 16) of A / column
// (l % 16) of B with the k-slice [(l / 16) * 8, + 8) of each 32-wide step, and receives the output
// rows 4 (l / 16) + r, r = 0..3, of column l % 16.
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));
template <class DT>
__device__ __forceinline__ f32x4 mma16(uint4 a, uint4 b, f32x4 c);
template <>
__device__ __forceinline__ f32x4 mma16<BF16>(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
template <>
__device__ __forceinline__ f32x4 mma16<F16>(uint4 a, uint4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// Row of the 32x32 output held in accumulator register r of `lane` (the column is lane % 32).
__device__ __forceinline__ int acc_row(int r, int lane) {
  return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
}

// Workgroup ids are dealt round-robin over the dies; renumber them so that each die gets one
// contiguous range of work items (all tiles of a head share that die's L2).
__device__ __forceinline__ int xcd_remap(int bid, int n) {
  const int q = n / kNumXcd, r = n % kNumXcd;
  const int x = bid % kNumXcd, slot = bid / kNumXcd;
  return x < r ? x * (q + 1) + slot : r * (q + 1) + (x - r) * q + slot;
}

// Tiles of ROWS rows of a [rows][D] matrix staged through LDS with 16-byte chunks; the row stride
// is padded by 16 bytes to spread the rows of a fragment read over the LDS banks.
template <class DT, int D, int NT = 256, int ROWS = 32>
struct Tile {
  static constexpr int RB = D * DT::kElt;
  static constexpr int RS = RB + 16;
  static constexpr int CH = RB / 16;
  static constexpr int CHUNKS = ROWS * CH;
  static constexpr int PER = (CHUNKS + NT - 1) / NT;  // chunks per thread (NT threads)
  static constexpr int BYTES = ROWS * RS;
};

// The PER 16-byte chunks a thread stages from each tile: chunk i is row row[i] of the
// tile, at byte mem[i] from the tile's first row in memory and byte lds[i] of an LDS buffer. The
// offsets are the same for every tile, so they are computed once per thread.
template <class TL, int NT>
struct TileChunks {
  unsigned row[TL::PER], mem[TL::PER], lds[TL::PER];
  int tid;
  __device__ explicit TileChunks(int t) : tid(t) {
#pragma unroll
    for (int i = 0; i < TL::PER; ++i) {
      const int ch = t + i * NT;
      row[i] = ch / TL::CH;
      mem[i] = row[i] * TL::RB + (ch % TL::CH) * 16;
      lds[i] = row[i] * TL::RS + (ch % TL::CH) * 16;
    }
  }
  // whether chunk i exists (always, when the threads cover the tile's chunks exactly)
  __device__ bool ok(int i) const { return (i + 1) * NT <= TL::CHUNKS || tid + i * NT < TL::CHUNKS; }
};

// Shape of the 32x32 scoring passes (fp32 inputs; 16-bit inputs take the 16x16 kernels): a
// workgroup covers 256 window rows (pass 1) or 256 keys (pass 2) as NBK register blocks of 32 per
// wave and 8 / NBK waves; fp32 fragments keep one block per wave.
template <class DT>
struct PassShape {
  static_assert(DT::kElt == 4, "16-bit inputs take k_rowstats16 / k_colsum16");
  static constexpr int NBK = 1;
  static constexpr int WAVES = kRowBlock / 32 / NBK;
  static constexpr int THREADS = WAVES * kWave;
  static constexpr int MIN_WAVES = 1;  // waves per SIMD the register budget keeps
};
static_assert(kRowBlock == kColBlockKeys, "both passes cover 256 rows / keys per workgroup");

// Row pass on 32x32 matrix instructions (fp32 inputs; 16-bit inputs take k_rowstats16 below):
// the offset follows the running max, so every exponent is at most 0.
template <class DT, int D>
__global__ __launch_bounds__(PassShape<DT>::THREADS, PassShape<DT>::MIN_WAVES) void k_rowstats(EvictArgs a) {
  using M = Mma<DT>;
  using PS = PassShape<DT>;
  constexpr int NBK = PS::NBK, NT = PS::THREADS;
  using TL = Tile<DT, D, NT>;
  constexpr int KS = D / M::K;
  __shared__ __align__(16) unsigned char s_k[2][TL::BYTES];

  const int n_rb = (a.W + kRowBlock - 1) / kRowBlock;
  const int id = xcd_remap(blockIdx.x, gridDim.x);
  const int rb = id % n_rb;
  const int ou = id / n_rb;  // (owner index * B + b) * Hq + hq
  const int l = a.own.local(ou / (a.B * a.Hq));
  const int b = (ou / a.Hq) % a.B, hq = ou % a.Hq;
  const size_t qunit = ((size_t)l * a.B + b) * a.Hq + hq;
  const int G = a.Hq / a.Hkv;
  const size_t kvunit = ((size_t)l * a.B + b) * a.Hkv + hq / G;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, c32 = lane & 31, hl = lane >> 5;

  // block u of this wave holds window rows row0 + 32 u .. + 31; lane column c32 is row t[u]
  const int row0 = rb * kRowBlock + w * 32 * NBK;
  int t[NBK], pos[NBK];
  typename M::Op qf[NBK][KS];
#pragma unroll
  for (int u = 0; u < NBK; ++u) {
    t[u] = row0 + 32 * u + c32;
    const int tc = t[u] < a.W ? t[u] : a.W - 1;
    pos[u] = a.T - a.W + tc;
    const char* qrow = (const char*)a.q_win + ((size_t)qunit * a.W + tc) * TL::RB;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[u][ks] = M::load(qrow + (ks * M::K + hl * M::KL) * DT::kElt);
  }

  const char* kh = (const char*)a.k + kvunit * a.T * TL::RB;
  const int last_row = min(a.W - 1, rb * kRowBlock + kRowBlock - 1);
  const int jend = a.causal ? min(a.T, a.T - a.W + last_row + 1) : a.T;
  const int ntile = (jend + 31) / 32;

  const TileChunks<TL, NT> tc(tid);
  uint4 pre[TL::PER];
  // key tiles lying wholly inside the cache load without per-chunk row tests or zero fills
  auto fetch = [&](int tile) {
    const char* tb = kh + (size_t)tile * (32 * TL::RB);
    if (tile * 32 + 32 <= a.T) {
#pragma unroll
      for (int i = 0; i < TL::PER; ++i)
        if (tc.ok(i)) pre[i] = ldg16(tb + tc.mem[i]);
    } else {
#pragma unroll
      for (int i = 0; i < TL::PER; ++i)
        pre[i] = tc.ok(i) && tile * 32 + (int)tc.row[i] < a.T ? ldg16(tb + tc.mem[i]) : make_uint4(0, 0, 0, 0);
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < TL::PER; ++i)
      if (tc.ok(i)) *(uint4*)&s_k[buf][tc.lds[i]] = pre[i];
  };
  fetch(0);
  stash(0);
  // the row operands are in registers before the loop, so that no wait for them lands inside it
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  const float cf = a.c32;
  float m[NBK], nb[NBK];  // running max and its whole-number offset -ceil(c * m), per block
  double ell[NBK];        // sum of exp2(fma(c, s, nb)) so far
#pragma unroll
  for (int u = 0; u < NBK; ++u) {
    m[u] = -INFINITY;
    nb[u] = INFINITY;
    ell[u] = 0.0;
  }
  for (int it = 0; it < ntile; ++it) {
    const int buf = it & 1;
    if (it + 1 < ntile) fetch(it + 1);
    f32x16 acc[NBK] = {};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const typename M::Op af =
          M::load(&s_k[buf][c32 * TL::RS + (ks * M::K + hl * M::KL) * DT::kElt]);
#pragma unroll
      for (int u = 0; u < NBK; ++u) acc[u] = M::run(af, qf[u][ks], acc[u]);
    }
    const int j0 = it * 32;
#pragma unroll
    for (int u = 0; u < NBK; ++u) {
      // a tile wholly inside the causal triangle and the key range needs no per-element mask
      // (uniform over the wave: the block's smallest row bounds every row's last visible key)
      const bool full = j0 + 31 < a.T && (!a.causal || j0 + 31 <= a.T - a.W + row0 + 32 * u);
      float tmax = -INFINITY;
      if (full) {
#pragma unroll
        for (int r = 0; r < 16; ++r) tmax = fmaxf(tmax, acc[u][r]);
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = j0 + acc_row(r, lane);
          if (j < a.T && (!a.causal || j <= pos[u])) tmax = fmaxf(tmax, acc[u][r]);
        }
      }
      if (tmax > m[u]) {
        // offsets are whole numbers, so moving one rescales the sum by a power of two (exact)
        const float nb_new = -ceilf(cf * tmax);
        if (ell[u] > 0.0 && nb_new != nb[u]) ell[u] = ldexp(ell[u], (int)(nb_new - nb[u]));
        m[u] = tmax;
        nb[u] = nb_new;
      }
      float ps = 0.f;
      if (full) {
#pragma unroll
        for (int r = 0; r < 16; ++r) ps += fast_exp2(fmaf(cf, acc[u][r], nb[u]));
      } else {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j = j0 + acc_row(r, lane);
          if (j < a.T && (!a.causal || j <= pos[u])) ps += fast_exp2(fmaf(cf, acc[u][r], nb[u]));
        }
      }
      ell[u] += (double)ps;
    }
    if (it + 1 < ntile) stash(buf ^ 1);
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < NBK; ++u) {
    // the two half-waves' sums meet at the offset of the larger max (the smaller offset)
    const double eo = __shfl_xor(ell[u], 32);
    const float nbo = __shfl_xor(nb[u], 32);
    const float nbx = fminf(nb[u], nbo);
    double L = 0.0;
    if (ell[u] > 0.0) L += ldexp(ell[u], (int)(nbx - nb[u]));
    if (eo > 0.0) L += ldexp(eo, (int)(nbx - nbo));
    if (hl == 0 && t[u] < a.W) {
      a.rowstat[(size_t)qunit * a.W + t[u]] = make_float2(nbx, (float)(1.0 / L));
      // log-sum-exp of the scaled scores: log2 of sum exp2(c * s) = log2(L) - offset
      if (a.row_lse) a.row_lse[(size_t)qunit * a.W + t[u]] = (float)((log2(L) - (double)nbx) * 0.69314718055994531);
    }
  }
}

// Column pass on 32x32 matrix instructions (fp32 inputs; 16-bit inputs take k_colsum16 below).
template <class DT, int D>
__global__ __launch_bounds__(PassShape<DT>::THREADS, PassShape<DT>::MIN_WAVES) void k_colsum(EvictArgs a) {
  using M = Mma<DT>;
  using PS = PassShape<DT>;
  constexpr int NBK = PS::NBK, NT = PS::THREADS;
  using TL = Tile<DT, D, NT>;
  constexpr int KS = D / M::K;
  __shared__ __align__(16) unsigned char s_q[2][TL::BYTES];
  __shared__ __align__(16) float s_nb[2][32], s_il[2][32];  // offset and 1 / sum of the staged rows

  const int n_kb = (a.T + kColBlockKeys - 1) / kColBlockKeys;
  const int id = xcd_remap(blockIdx.x, gridDim.x);
  const int kb = id % n_kb;
  const int ou = id / n_kb;  // (owner index * B + b) * Hkv + h
  const int l = a.own.local(ou / (a.B * a.Hkv));
  const int b = (ou / a.Hkv) % a.B, h = ou % a.Hkv;
  const size_t kvunit = ((size_t)l * a.B + b) * a.Hkv + h;
  const int G = a.Hq / a.Hkv;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, c32 = lane & 31, hl = lane >> 5;

  // block u of this wave holds keys jw + 32 u .. + 31; lane column c32 is key jw + 32 u + c32
  const int jw = kb * kColBlockKeys + w * 32 * NBK;
  const float cf = a.c32;
  const char* kh = (const char*)a.k + (size_t)kvunit * a.T * TL::RB;
  typename M::Op kf[NBK][KS];
#pragma unroll
  for (int u = 0; u < NBK; ++u) {
    const int j = min(jw + 32 * u + c32, a.T - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      kf[u][ks] = M::load(kh + (size_t)j * TL::RB + (ks * M::K + hl * M::KL) * DT::kElt);
  }

  const int j_lo = kb * kColBlockKeys;
  const int t_start = a.causal ? (max(0, j_lo - (a.T - a.W)) & ~31) : 0;
  const int n_t = (a.W - t_start + 31) / 32;
  const int ntile = G * n_t;
  const size_t qunit0 = ((size_t)l * a.B + b) * a.Hq + (size_t)h * G;

  const TileChunks<TL, NT> tc(tid);
  uint4 pre[TL::PER];
  float2 pre_b = make_float2(0.f, 0.f);
  // tiles run through the group's heads, each from row t_start to t_end; the next one to fetch is
  // head fg's rows ft0 .. ft0 + 31 (a counter, not a division per tile)
  const int t_end = t_start + n_t * 32;
  int fg = 0, ft0 = t_start;
  auto fetch = [&]() {
    const size_t r0 = (qunit0 + fg) * a.W + ft0;
    const char* tb = (const char*)a.q_win + r0 * TL::RB;
    if (ft0 + 32 <= a.W) {
#pragma unroll
      for (int i = 0; i < TL::PER; ++i)
        if (tc.ok(i)) pre[i] = ldg16(tb + tc.mem[i]);
    } else {
#pragma unroll
      for (int i = 0; i < TL::PER; ++i)
        pre[i] = tc.ok(i) && ft0 + (int)tc.row[i] < a.W ? ldg16(tb + tc.mem[i]) : make_uint4(0, 0, 0, 0);
    }
    if (tid < 32) pre_b = ft0 + tid < a.W ? a.rowstat[r0 + tid] : make_float2(0.f, 0.f);
    ft0 += 32;
    if (ft0 == t_end) {
      ft0 = t_start;
      ++fg;
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < TL::PER; ++i)
      if (tc.ok(i)) *(uint4*)&s_q[buf][tc.lds[i]] = pre[i];
    if (tid < 32) {
      s_nb[buf][tid] = pre_b.x;
      s_il[buf][tid] = pre_b.y;
    }
  };
  fetch();
  stash(0);
  // the key operands are in registers before the loop, so that no wait for them lands inside it
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  double cacc[NBK];
#pragma unroll
  for (int u = 0; u < NBK; ++u) cacc[u] = 0.0;
  int t0 = t_start;  // first window row of the tile being scored
  for (int it = 0; it < ntile; ++it) {
    const int buf = it & 1;
    if (it + 1 < ntile) fetch();
    f32x16 acc[NBK] = {};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const typename M::Op af =
          M::load(&s_q[buf][c32 * TL::RS + (ks * M::K + hl * M::KL) * DT::kElt]);
#pragma unroll
      for (int u = 0; u < NBK; ++u) acc[u] = M::run(af, kf[u][ks], acc[u]);
    }
    // every row of the tile valid and every key of the wave's last block visible to its first row
    const bool full = t0 + 31 < a.W && (!a.causal || jw + 32 * NBK - 1 <= a.T - a.W + t0);
    float ps[NBK];
#pragma unroll
    for (int u = 0; u < NBK; ++u) ps[u] = 0.f;
    if (full) {
      // the tile's rows of this lane: 8 g + 4 hl + (0..3), g = 0..3, read four at a time
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const float4 nb4 = *(const float4*)&s_nb[buf][8 * g4 + 4 * hl];
        const float4 il4 = *(const float4*)&s_il[buf][8 * g4 + 4 * hl];
        const float nbv[4] = {nb4.x, nb4.y, nb4.z, nb4.w}, ilv[4] = {il4.x, il4.y, il4.z, il4.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
#pragma unroll
          for (int u = 0; u < NBK; ++u)
            ps[u] = fmaf(fast_exp2(fmaf(cf, acc[u][4 * g4 + q], nbv[q])), ilv[q], ps[u]);
        }
      }
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rr = acc_row(r, lane);
        const int trow = t0 + rr;
        if (trow >= a.W) continue;
        const float nbv = s_nb[buf][rr], ilv = s_il[buf][rr];
#pragma unroll
        for (int u = 0; u < NBK; ++u) {
          const int j = jw + 32 * u + c32;
          if (!a.causal || j <= a.T - a.W + trow) ps[u] = fmaf(fast_exp2(fmaf(cf, acc[u][r], nbv)), ilv, ps[u]);
        }
      }
    }
#pragma unroll
    for (int u = 0; u < NBK; ++u) cacc[u] += (double)ps[u];
    if (it + 1 < ntile) stash(buf ^ 1);
    t0 = t0 + 32 == t_end ? t_start : t0 + 32;
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < NBK; ++u) {
    const double tot = cacc[u] + __shfl_xor(cacc[u], 32);
    const int j = jw + 32 * u + c32;
    if (hl == 0 && j < a.T) a.score[(size_t)kvunit * a.T + j] = (float)tot;
  }
}

// Row pass for 16-bit inputs on 16x16x32 matrix instructions. A wave holds 64 window rows in
// registers as four 16-row B operands (query groups) and takes each 64-key tile from LDS as four
// 16-key A operands, so a tile is sixteen 16x16 blocks; a lane holds keys 4 (lane / 16) + r of one
// row per block. Each block's exponentials are taken against the row's current offset, with no
// running max, beside the next block's matrix chain (one basic block, so the two interleave). A
// block whose four terms sum to at most 2 has every exponent at most 1, as accurate as an offset
// at the max; a larger sum takes the slow path: the offset moves to the block's max if that is
// higher (the running sums rescaled by an exact power of two) and the block is summed again. The
// four lanes of a row meet once at the end at the smallest offset, so no exponent of pass 2 exceeds 1.
template <class DT, int D>
__global__ __launch_bounds__(kRowThreads16, 3) void k_rowstats16(EvictArgs a) {
  constexpr int NT = kRowThreads16;
  constexpr int KT = 64;  // keys per staged tile
  using TL = Tile<DT, D, NT, KT>;
  constexpr int KS = D / 32;
  static_assert(DT::kElt == 2, "16-bit inputs");
  static_assert(NT / kWave * 64 == kRowBlock, "four waves of 64 rows");
  __shared__ __align__(16) unsigned char s_k[2][TL::BYTES];

  const int n_rb = (a.W + kRowBlock - 1) / kRowBlock;
  const int id = xcd_remap(blockIdx.x, gridDim.x);
  const int rb = id % n_rb;
  const int ou = id / n_rb;  // (owner index * B + b) * Hq + hq
  const int l = a.own.local(ou / (a.B * a.Hq));
  const int b = (ou / a.Hq) % a.B, hq = ou % a.Hq;
  const size_t qunit = ((size_t)l * a.B + b) * a.Hq + hq;
  const int G = a.Hq / a.Hkv;
  const size_t kvunit = ((size_t)l * a.B + b) * a.Hkv + hq / G;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, c16 = lane & 15, q4 = lane >> 4;

  // query group g of this wave holds window rows row0 + 16 g + lane % 16
  const int row0 = rb * kRowBlock + w * 64;
  int t[4], pos[4];
  uint4 qf[4][KS];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    t[g] = row0 + 16 * g + c16;
    const int tc = t[g] < a.W ? t[g] : a.W - 1;
    pos[g] = a.T - a.W + tc;
    const char* qrow = (const char*)a.q_win + ((size_t)qunit * a.W + tc) * TL::RB;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[g][ks] = ldg16(qrow + (ks * 32 + q4 * 8) * DT::kElt);
  }

  const char* kh = (const char*)a.k + kvunit * a.T * TL::RB;
  const int last_row = min(a.W - 1, rb * kRowBlock + kRowBlock - 1);
  const int jend = a.causal ? min(a.T, a.T - a.W + last_row + 1) : a.T;
  const int ntile = (jend + KT - 1) / KT;

  const TileChunks<TL, NT> tc(tid);
  uint4 pre[TL::PER];
  // key tiles lying wholly inside the cache load without per-chunk row tests or zero fills
  auto fetch = [&](int tile) {
    const char* tb = kh + (size_t)tile * (KT * TL::RB);
    if (tile * KT + KT <= a.T) {
#pragma unroll
      for (int i = 0; i < TL::PER; ++i)
        if (tc.ok(i)) pre[i] = ldg16(tb + tc.mem[i]);
    } else {
#pragma unroll
      for (int i = 0; i < TL::PER; ++i)
        pre[i] = tc.ok(i) && tile * KT + (int)tc.row[i] < a.T ? ldg16(tb + tc.mem[i]) : make_uint4(0, 0, 0, 0);
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < TL::PER; ++i)
      if (tc.ok(i)) *(uint4*)&s_k[buf][tc.lds[i]] = pre[i];
  };
  fetch(0);
  stash(0);
  // the row operands are in registers before the loop, so that no wait for them lands inside it
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  const float cf = a.c32;
  float nb[4];    // whole-number offset of each query group's row (this lane's keys)
  double ell[4];  // sum of exp2(fma(c, s, nb)) so far
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    nb[g] = INFINITY;
    ell[g] = 0.0;
  }
  // one tile; block b = (key quarter b / 4, query group b % 4). FULL: every key of the tile visible
  // to every row of the wave
  auto tile = [&](auto full_tag, int buf, int j0) {
    constexpr bool FULL = decltype(full_tag)::value;
    float psg[4] = {0.f, 0.f, 0.f, 0.f};
    uint4 af[KS];
    auto load_af = [&](int kq) {
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        af[ks] = *(const uint4*)&s_k[buf][(16 * kq + c16) * TL::RS + (ks * 32 + q4 * 8) * DT::kElt];
    };
    auto chain = [&](int g) {
      f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) c = mma16<DT>(af[ks], qf[g][ks], c);
      return c;
    };
    auto visible = [&](int kq, int g, int r) {
      if constexpr (FULL) return true;
      const int j = j0 + 16 * kq + 4 * q4 + r;
      return j < a.T && (!a.causal || j <= pos[g]);
    };
    auto sum4 = [&](const f32x4& c, int kq, int g) {
      float ps = 0.f;
#pragma unroll
      for (int r = 0; r < 4; ++r)
        if (visible(kq, g, r)) ps += fast_exp2(fmaf(cf, c[r], nb[g]));
      return ps;
    };
    auto finish = [&](const f32x4& c, int kq, int g, float ps) {
      if (ps > 2.f) {  // an exponent may exceed 1 (or the row's first terms): offset at the max
        float tmax = -INFINITY;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (visible(kq, g, r)) tmax = fmaxf(tmax, c[r]);
        const float nb_new = -ceilf(cf * tmax);
        if (nb_new < nb[g]) {
          const int d = (int)(nb_new - nb[g]);
          if (ell[g] > 0.0) ell[g] = ldexp(ell[g], d);
          if (psg[g] > 0.f) psg[g] = ldexpf(psg[g], d);
          nb[g] = nb_new;
        }
        ps = sum4(c, kq, g);
      }
      psg[g] += ps;
    };
    load_af(0);
    f32x4 cp = chain(0);
#pragma unroll
    for (int bb = 1; bb < 4 * (KT / 16); ++bb) {
      if ((bb & 3) == 0) load_af(bb >> 2);
      const f32x4 cc = chain(bb & 3);
      const int kp = (bb - 1) >> 2, gp = (bb - 1) & 3;
      finish(cp, kp, gp, sum4(cp, kp, gp));
      cp = cc;
    }
    finish(cp, KT / 16 - 1, 3, sum4(cp, KT / 16 - 1, 3));
#pragma unroll
    for (int g = 0; g < 4; ++g) ell[g] += (double)psg[g];
  };
  // a wave whose rows all lie past the window (the last workgroup of a ragged window) only helps
  // stage the tiles
  const bool rows_live = row0 < a.W;
  for (int it = 0; it < ntile; ++it) {
    const int buf = it & 1;
    if (it + 1 < ntile) fetch(it + 1);
    const int j0 = it * KT;
    if (rows_live) {
      if (j0 + KT - 1 < a.T && (!a.causal || j0 + KT - 1 <= a.T - a.W + row0))
        tile(std::true_type{}, buf, j0);
      else
        tile(std::false_type{}, buf, j0);
    }
    if (it + 1 < ntile) stash(buf ^ 1);
    __syncthreads();
  }
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    // the four lanes of a row (lane % 16 equal) meet at the smallest offset, in two pairwise steps
    double e = ell[g];
    float o = nb[g];
#pragma unroll
    for (int x = 16; x <= 32; x <<= 1) {
      const double eo = __shfl_xor(e, x);
      const float oo = __shfl_xor(o, x);
      const float ox = fminf(o, oo);
      double L = 0.0;
      if (e > 0.0) L += ldexp(e, (int)(ox - o));
      if (eo > 0.0) L += ldexp(eo, (int)(ox - oo));
      e = L;
      o = ox;
    }
    if (q4 == 0 && t[g] < a.W) {
      a.rowstat[(size_t)qunit * a.W + t[g]] = make_float2(o, (float)(1.0 / e));
      // log-sum-exp of the scaled scores: log2 of sum exp2(c * s) = log2(L) - offset
      if (a.row_lse) a.row_lse[(size_t)qunit * a.W + t[g]] = (float)((log2(e) - (double)o) * 0.69314718055994531);
    }
  }
}

// Column pass for 16-bit inputs on 16x16x32 matrix instructions. A wave holds 64 keys in
// registers as four 16-key B operands and takes each 64-row window tile from LDS as four 16-row A
// operands, so a tile is sixteen 16x16 blocks of four accumulators each; every block's
// exponentials and sums run while the next block's four matrix instructions execute (a block's
// vector work, twelve instructions, matches its matrix work), with no second accumulator set, and
// a barrier, a tile load and a row-statistics stash serve 64 rows. A lane holds rows
// 4 (lane / 16) + r of one key per block; its fp32 sum over a tile's sixteen rows goes into an fp64
// total, and the four lanes of a key meet once at the end.
template <class DT, int D>
__global__ __launch_bounds__(kColThreads16, 3) void k_colsum16(EvictArgs a) {
  constexpr int NT = kColThreads16;
  constexpr int RT = 64;  // window rows per staged tile
  using TL = Tile<DT, D, NT, RT>;
  constexpr int KS = D / 32;
  static_assert(DT::kElt == 2, "16-bit inputs");
  static_assert(NT / kWave * 64 == kColBlockKeys, "four waves of 64 keys");
  __shared__ __align__(16) unsigned char s_q[2][TL::BYTES];
  __shared__ __align__(16) float s_nb[2][RT], s_il[2][RT];  // offset and 1 / sum of the staged rows

  const int n_kb = (a.T + kColBlockKeys - 1) / kColBlockKeys;
  const int id = xcd_remap(blockIdx.x, gridDim.x);
  const int kb = id % n_kb;
  const int ou = id / n_kb;  // (owner index * B + b) * Hkv + h
  const int l = a.own.local(ou / (a.B * a.Hkv));
  const int b = (ou / a.Hkv) % a.B, h = ou % a.Hkv;
  const size_t kvunit = ((size_t)l * a.B + b) * a.Hkv + h;
  const int G = a.Hq / a.Hkv;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, c16 = lane & 15, q4 = lane >> 4;

  // key group g of this wave holds keys jw + 16 g + lane % 16
  const int jw = kb * kColBlockKeys + w * 64;
  const float cf = a.c32;
  const char* kh = (const char*)a.k + (size_t)kvunit * a.T * TL::RB;
  uint4 kf[4][KS];
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const int j = min(jw + 16 * g + c16, a.T - 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) kf[g][ks] = ldg16(kh + (size_t)j * TL::RB + (ks * 32 + q4 * 8) * DT::kElt);
  }

  const int j_lo = kb * kColBlockKeys;
  const int t_start = a.causal ? (max(0, j_lo - (a.T - a.W)) & ~31) : 0;
  const int n_t = (a.W - t_start + RT - 1) / RT;
  const int ntile = G * n_t;
  const size_t qunit0 = ((size_t)l * a.B + b) * a.Hq + (size_t)h * G;

  const TileChunks<TL, NT> tc(tid);
  uint4 pre[TL::PER];
  float2 pre_b = make_float2(0.f, 0.f);
  // tiles run through the group's heads, each from row t_start to t_end; the next one to fetch is
  // head fg's rows ft0 .. ft0 + RT - 1
  const int t_end = t_start + n_t * RT;
  int fg = 0, ft0 = t_start;
  auto fetch = [&]() {
    const size_t r0 = (qunit0 + fg) * a.W + ft0;
    const char* tb = (const char*)a.q_win + r0 * TL::RB;
    if (ft0 + RT <= a.W) {
#pragma unroll
      for (int i = 0; i < TL::PER; ++i)
        if (tc.ok(i)) pre[i] = ldg16(tb + tc.mem[i]);
    } else {
#pragma unroll
      for (int i = 0; i < TL::PER; ++i)
        pre[i] = tc.ok(i) && ft0 + (int)tc.row[i] < a.W ? ldg16(tb + tc.mem[i]) : make_uint4(0, 0, 0, 0);
    }
    if (tid < RT) pre_b = ft0 + tid < a.W ? a.rowstat[r0 + tid] : make_float2(0.f, 0.f);
    ft0 += RT;
    if (ft0 == t_end) {
      ft0 = t_start;
      ++fg;
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < TL::PER; ++i)
      if (tc.ok(i)) *(uint4*)&s_q[buf][tc.lds[i]] = pre[i];
    if (tid < RT) {
      s_nb[buf][tid] = pre_b.x;
      s_il[buf][tid] = pre_b.y;
    }
  };
  fetch();
  stash(0);
  // the key operands are in registers before the loop, so that no wait for them lands inside it
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  double cacc[4] = {0.0, 0.0, 0.0, 0.0};
  int t0 = t_start;  // first window row of the tile being scored
  // one tile; FULL: every row valid and every key of the wave visible to the tile's first row
  auto tile = [&](auto full_tag, int buf) {
    constexpr bool FULL = decltype(full_tag)::value;
    float ps[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int rh = 0; rh < RT / 16; ++rh) {
      // this lane's rows of the quarter: t0 + 16 rh + 4 (lane / 16) + r
      const float4 nb4 = *(const float4*)&s_nb[buf][16 * rh + 4 * q4];
      const float4 il4 = *(const float4*)&s_il[buf][16 * rh + 4 * q4];
      const float nbv[4] = {nb4.x, nb4.y, nb4.z, nb4.w}, ilv[4] = {il4.x, il4.y, il4.z, il4.w};
      uint4 af[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        af[ks] = *(const uint4*)&s_q[buf][(16 * rh + c16) * TL::RS + (ks * 32 + q4 * 8) * DT::kElt];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) c = mma16<DT>(af[ks], kf[g][ks], c);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          if constexpr (FULL) {
            ps[g] = fmaf(fast_exp2(fmaf(cf, c[r], nbv[r])), ilv[r], ps[g]);
          } else {
            const int t = t0 + 16 * rh + 4 * q4 + r, j = jw + 16 * g + c16;
            if (t < a.W && (!a.causal || j <= a.T - a.W + t))
              ps[g] = fmaf(fast_exp2(fmaf(cf, c[r], nbv[r])), ilv[r], ps[g]);
          }
        }
      }
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) cacc[g] += (double)ps[g];
  };
  for (int it = 0; it < ntile; ++it) {
    const int buf = it & 1;
    if (it + 1 < ntile) fetch();
    if (t0 + RT - 1 < a.W && (!a.causal || jw + 63 <= a.T - a.W + t0))
      tile(std::true_type{}, buf);
    else
      tile(std::false_type{}, buf);
    if (it + 1 < ntile) stash(buf ^ 1);
    t0 = t0 + RT == t_end ? t_start : t0 + RT;
    __syncthreads();
  }
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    double tot = cacc[g] + __shfl_xor(cacc[g], 16);
    tot += __shfl_xor(tot, 32);
    const int j = jw + 16 * g + c16;
    if (q4 == 0 && j < a.T) a.score[(size_t)kvunit * a.T + j] = (float)tot;
  }
}

// Exclusive prefix sum over the 1024 threads of a workgroup.
__device__ int block_excl_scan(int v, int* wsum) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) wsum[w] = x;
  __syncthreads();
  if (w == 0) {
    int s = lane < 16 ? wsum[lane] : 0;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      const int y = __shfl_up(s, o);
      if (lane >= o) s += y;
    }
    if (lane < 16) wsum[lane] = s;
  }
  __syncthreads();
  const int res = (w > 0 ? wsum[w - 1] : 0) + x - v;
  __syncthreads();
  return res;
}

constexpr int kTopkThreads = 1024;

// The radix digit (bins in descending order) at which the running count of tot[] reaches rem, by
// the 64 lanes of wave 0 (four bins each, a wave prefix sum): writes prefix | digit << shift to
// *s_prefix and rem minus the count of the higher bins to *s_rem. Requires sum(tot) >= rem >= 1.
__device__ __forceinline__ void pick_digit(const uint32_t* tot, int rem, uint32_t prefix, int shift,
                                           uint32_t* s_prefix, int* s_rem) {
  const int lane = threadIdx.x & 63;
  uint32_t c[4], sum = 0;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    c[u] = tot[255 - 4 * lane - u];
    sum += c[u];
  }
  uint32_t x = sum;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  uint32_t cum = x - sum;  // count of the bins above this lane's first
  const uint32_t r = (uint32_t)rem;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (cum < r && r <= cum + c[u]) {
      *s_prefix = prefix | ((uint32_t)(255 - 4 * lane - u) << shift);
      *s_rem = (int)(r - cum);
    }
    cum += c[u];
  }
}

__global__ __launch_bounds__(kTopkThreads) void k_topk(EvictArgs a) {
  __shared__ uint32_t hist[kTopkThreads / 64][256];
  __shared__ uint32_t tot[256];
  __shared__ uint32_t s_prefix;
  __shared__ int s_rem;
  __shared__ int wsum[16];

  const int ou = blockIdx.x;  // (owner index * B + b) * Hkv + h
  const int l = a.own.local(ou / (a.B * a.Hkv));
  const size_t unit = (size_t)l * a.B * a.Hkv + ou % (a.B * a.Hkv);
  const int tid = threadIdx.x, w = tid >> 6;
  const int loc = min(a.local_keep, a.keep);
  const int n_old = a.T - loc, n_sel = a.keep - loc;
  const uint32_t* key = (const uint32_t*)(a.score + (size_t)unit * a.T);
  int32_t* out = a.kept + (size_t)unit * a.keep;

  // radix select: the n_sel-th largest key (non-negative floats order like their bits)
  uint32_t prefix = 0, mask = 0;
  int rem = n_sel;
  if (n_sel > 0) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < (kTopkThreads / 64) * 256; i += kTopkThreads) hist[i / 256][i % 256] = 0;
      __syncthreads();
      for (int j = tid; j < n_old; j += kTopkThreads) {
        const uint32_t u = key[j];
        if ((u & mask) == prefix) atomicAdd(&hist[w][(u >> shift) & 255u], 1u);
      }
      __syncthreads();
      if (tid < 256) {
        uint32_t s = 0;
        for (int i = 0; i < kTopkThreads / 64; ++i) s += hist[i][tid];
        tot[tid] = s;
      }
      __syncthreads();
      if (tid < 64) pick_digit(tot, rem, prefix, shift, &s_prefix, &s_rem);
      __syncthreads();
      prefix = s_prefix;
      rem = s_rem;
      mask |= 255u << shift;
      __syncthreads();
    }
  }
  // ordered compaction: keys above the threshold, then the lowest-index ties up to `rem`
  const int chk = (n_old + kTopkThreads - 1) / kTopkThreads;
  const int j0 = min(n_old, tid * chk), j1 = min(n_old, j0 + chk);
  int gt = 0, eq = 0;
  if (n_sel > 0)
    for (int j = j0; j < j1; ++j) {
      const uint32_t u = key[j];
      gt += u > prefix;
      eq += u == prefix;
    }
  const int eq_before = block_excl_scan(eq, wsum);
  const int take = n_sel > 0 ? max(0, min(eq, rem - eq_before)) : 0;
  int off = block_excl_scan(gt + take, wsum);
  if (n_sel > 0) {
    int taken = 0;
    for (int j = j0; j < j1; ++j) {
      const uint32_t u = key[j];
      if (u > prefix || (u == prefix && taken < take)) {
        taken += u == prefix;
        out[off++] = j;
      }
    }
  }
  for (int i = tid; i < loc; i += kTopkThreads) out[n_sel + i] = n_old + i;
}

// The same selection with each thread's run of KPT scores held in registers from one read on:
// the radix passes and the compaction read registers, not the score buffer (which otherwise is
// re-read from memory by every pass once the heads in flight outgrow the L2).
template <int KPT>
__global__ __launch_bounds__(kTopkThreads) void k_topk_reg(EvictArgs a) {
  __shared__ uint32_t hist[kTopkThreads / 64][256];
  __shared__ uint32_t tot[256];
  __shared__ uint32_t s_prefix;
  __shared__ int s_rem;
  __shared__ int wsum[16];

  const int ou = blockIdx.x;  // (owner index * B + b) * Hkv + h
  const int l = a.own.local(ou / (a.B * a.Hkv));
  const size_t unit = (size_t)l * a.B * a.Hkv + ou % (a.B * a.Hkv);
  const int tid = threadIdx.x, w = tid >> 6;
  const int loc = min(a.local_keep, a.keep);
  const int n_old = a.T - loc, n_sel = a.keep - loc;
  const uint32_t* key = (const uint32_t*)(a.score + (size_t)unit * a.T);
  int32_t* out = a.kept + (size_t)unit * a.keep;

  // this thread's run [j0, j0 + nv) of the older tokens' scores
  const int j0 = tid * KPT;
  const int nv = max(0, min(KPT, n_old - j0));
  uint32_t kv[KPT];
  if (nv == KPT && (((uintptr_t)(key + j0)) & 15) == 0) {
#pragma unroll
    for (int i = 0; i < KPT; i += 4) {
      const uint4 v = *(const uint4*)(key + j0 + i);
      kv[i] = v.x;
      kv[i + 1] = v.y;
      kv[i + 2] = v.z;
      kv[i + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < KPT; ++i) kv[i] = i < nv ? key[j0 + i] : 0u;
  }

  // radix select: the n_sel-th largest key (non-negative floats order like their bits)
  uint32_t prefix = 0, mask = 0;
  int rem = n_sel;
  if (n_sel > 0) {
    for (int shift = 24; shift >= 0; shift -= 8) {
      for (int i = tid; i < (kTopkThreads / 64) * 256; i += kTopkThreads) hist[i / 256][i % 256] = 0;
      __syncthreads();
#pragma unroll
      for (int i = 0; i < KPT; ++i)
        if (i < nv && (kv[i] & mask) == prefix) atomicAdd(&hist[w][(kv[i] >> shift) & 255u], 1u);
      __syncthreads();
      if (tid < 256) {
        uint32_t s = 0;
        for (int i = 0; i < kTopkThreads / 64; ++i) s += hist[i][tid];
        tot[tid] = s;
      }
      __syncthreads();
      if (tid < 64) pick_digit(tot, rem, prefix, shift, &s_prefix, &s_rem);
      __syncthreads();
      prefix = s_prefix;
      rem = s_rem;
      mask |= 255u << shift;
      __syncthreads();
    }
  }
  // ordered compaction: keys above the threshold, then the lowest-index ties up to `rem`
  int gt = 0, eq = 0;
  if (n_sel > 0) {
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      gt += i < nv && kv[i] > prefix;
      eq += i < nv && kv[i] == prefix;
    }
  }
  const int eq_before = block_excl_scan(eq, wsum);
  const int take = n_sel > 0 ? max(0, min(eq, rem - eq_before)) : 0;
  int off = block_excl_scan(gt + take, wsum);
  if (n_sel > 0) {
    int taken = 0;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      if (i < nv && (kv[i] > prefix || (kv[i] == prefix && taken < take))) {
        taken += kv[i] == prefix;
        out[off++] = j0 + i;
      }
    }
  }
  for (int i = tid; i < loc; i += kTopkThreads) out[n_sel + i] = n_old + i;
}

template <int RB>
__global__ __launch_bounds__(256) void k_gather(EvictArgs a) {
  constexpr int CH = RB / 16;
  constexpr int RPP = 256 / CH;
  constexpr int ROWS = 64;
  const int n_chunks = (a.keep + ROWS - 1) / ROWS;
  const int chunk = blockIdx.x % n_chunks;
  const size_t unit = blockIdx.x / n_chunks;
  const int l = (int)(unit / ((size_t)a.B * a.Hkv));
  if ((a.skip[l >> 6] >> (l & 63)) & 1) return;
  const int o = owner_layer(a.layer0 + l, a.period, a.start) - a.layer0;
  const int src_l = o >= 0 ? o : l;
  const size_t src_unit = unit - (size_t)(l - src_l) * a.B * a.Hkv;
  const int r_in = threadIdx.x / CH, c16 = threadIdx.x % CH;
  const int end = min(a.keep, chunk * ROWS + ROWS);
  for (int i = chunk * ROWS + r_in; i < end; i += RPP) {
    int idx = a.kept[src_unit * a.keep + i];
    if (src_l != l && c16 == 0) a.kept[unit * a.keep + i] = idx;
    idx = min(max(idx, 0), a.T - 1);  // indices supplied by the caller are clamped into the cache
    const size_t so = (unit * a.T + idx) * RB + c16 * 16;
    const size_t dst = (unit * a.out_rows + i) * RB + c16 * 16;
    *(uint4*)((char*)a.k_out + dst) = ldg16((const char*)a.k + so);
    *(uint4*)((char*)a.v_out + dst) = ldg16((const char*)a.v + so);
  }
}

template <class DT, int D>
hipError_t launch_pass(const EvictArgs& a, bool rows, hipStream_t st) {
  if (rows) {
    const int n_rb = (a.W + kRowBlock - 1) / kRowBlock;
    if constexpr (DT::kElt == 2)
      hipLaunchKernelGGL((k_rowstats16<DT, D>), dim3(a.own.n * a.B * a.Hq * n_rb), dim3(kRowThreads16), 0, st, a);
    else
      hipLaunchKernelGGL((k_rowstats<DT, D>), dim3(a.own.n * a.B * a.Hq * n_rb), dim3(PassShape<DT>::THREADS), 0, st, a);
  } else {
    const int n_kb = (a.T + kColBlockKeys - 1) / kColBlockKeys;
    if constexpr (DT::kElt == 2)
      hipLaunchKernelGGL((k_colsum16<DT, D>), dim3(a.own.n * a.B * a.Hkv * n_kb), dim3(kColThreads16), 0, st, a);
    else
      hipLaunchKernelGGL((k_colsum<DT, D>), dim3(a.own.n * a.B * a.Hkv * n_kb), dim3(PassShape<DT>::THREADS), 0, st, a);
  }
  return hipGetLastError();
}

template <class DT>
hipError_t launch_pass_dt(const EvictArgs& a, int D, bool rows, hipStream_t st) {
  if (D == 64) return launch_pass<DT, 64>(a, rows, st);
  if (D == 128) return launch_pass<DT, 128>(a, rows, st);
  return hipErrorInvalidValue;
}

hipError_t launch_pass_any(const EvictArgs& a, int dtype, int D, bool rows, hipStream_t st) {
  switch (dtype) {
    case MPC_FP32: return launch_pass_dt<F32>(a, D, rows, st);
    case MPC_FP16: return launch_pass_dt<F16>(a, D, rows, st);
    case MPC_BF16: return launch_pass_dt<BF16>(a, D, rows, st);
  }
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_rowstats(const EvictArgs& a, int dtype, int D, hipStream_t st) {
  return launch_pass_any(a, dtype, D, true, st);
}

hipError_t launch_colsum(const EvictArgs& a, int dtype, int D, hipStream_t st) {
  return launch_pass_any(a, dtype, D, false, st);
}

hipError_t launch_topk(const EvictArgs& a, hipStream_t st) {
  // a run of up to 32 scores per thread stays in registers; longer prompts stream the scores
  const dim3 grid(a.own.n * a.B * a.Hkv), block(kTopkThreads);
  const int n_old = a.T - min(a.local_keep, a.keep);
  if (n_old <= 4 * kTopkThreads)
    hipLaunchKernelGGL(k_topk_reg<4>, grid, block, 0, st, a);
  else if (n_old <= 8 * kTopkThreads)
    hipLaunchKernelGGL(k_topk_reg<8>, grid, block, 0, st, a);
  else if (n_old <= 16 * kTopkThreads)
    hipLaunchKernelGGL(k_topk_reg<16>, grid, block, 0, st, a);
  else if (n_old <= 32 * kTopkThreads)
    hipLaunchKernelGGL(k_topk_reg<32>, grid, block, 0, st, a);
  else
    hipLaunchKernelGGL(k_topk, grid, block, 0, st, a);
  return hipGetLastError();
}

hipError_t launch_gather(const EvictArgs& a, int dtype, int D, hipStream_t st) {
  const int rb = D * (dtype == MPC_FP32 ? 4 : 2);
  const int blocks = a.n_layers * a.B * a.Hkv * ((a.keep + 63) / 64);
  switch (rb) {
    case 128: hipLaunchKernelGGL(k_gather<128>, dim3(blocks), dim3(256), 0, st, a); break;
    case 256: hipLaunchKernelGGL(k_gather<256>, dim3(blocks), dim3(256), 0, st, a); break;
    case 512: hipLaunchKernelGGL(k_gather<512>, dim3(blocks), dim3(256), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace mpc
