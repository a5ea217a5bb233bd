// Early-exit prefetch head on gfx950 (wave64, MFMA): the approximate
// next-token distribution p = softmax(W h) of an intermediate hidden state
// (Eq. 13) and its K most likely tokens (Eq. 14), which are the candidates
// the cache prefetch consumes.
//
// For up to 64 rows (and K at most the number of compute units) one launch,
// k_head_fused (below, with its design); otherwise two launches:
//   k_head_logits  logits = W h for up to 64 rows h per block: a dense
//                  contraction, so it runs on the matrix cores
//                  (v_mfma_f32_16x16x32_bf16).  W ([V x D] bf16, 311 MB for
//                  the 151936 x 1024 head) is streamed from HBM exactly once
//                  per 64 rows; the 64 hidden rows are staged in LDS and read
//                  by every wave.  One wave computes three 16-token x
//                  64-row tiles at a time (single tiles for the rest of a
//                  block's range), which share each read of the staged
//                  rows: W is read 128 contiguous bytes per row and load
//                  instruction, a few chunks of every row in flight
//                  together, then passed through a small per-wave LDS
//                  staging tile into the MFMA operand layout.
//                  The epilogue writes the fp32 logits and, per (row,
//                  16-token tile), the largest (logit, id) key and the sum of
//                  exp(logit - tile max).
//   k_head_rows    per row: the log-sum-exp from the tile statistics, a
//                  radix select over the tile keys down to a set of at least
//                  K tiles (every top-K logit lies in one of the K tiles with
//                  the largest maxima), then those tiles' logits ranked in
//                  LDS.
// Ties in logit go to the lower token id, so the answer is unique.  The K
// output probabilities use the full-accuracy expf (about 1 ulp); the chunk
// sums of exp(l - max) use the hardware exponential, whose relative error
// (about |l - max| 2^-24 plus an ulp) is negligible in a sum dominated by
// terms near the maximum.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tfe_head.h"

namespace tfe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

#ifndef TFE_HEAD_WAVES
#define TFE_HEAD_WAVES 8
#endif
#ifndef TFE_HEAD_NT
#define TFE_HEAD_NT 1
#endif

constexpr int kLogitWaves = TFE_HEAD_WAVES;  // waves per logits block (tuning knob)
constexpr int kCols = 64;        // hidden rows per logits block (4 MFMA column tiles)

// Order-preserving float -> uint32 map (larger float, larger key).
__device__ __forceinline__ uint32_t f2key(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key2f(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7FFFFFFFu) : ~k);
}
// 64-bit unsigned max (the generic max/min overloads can resolve to
// floating point for mixed integer types, which would round the keys).
__device__ __forceinline__ uint64_t umax64(uint64_t x, uint64_t y) { return x > y ? x : y; }
// (logit, token) -> 64-bit key: higher logit first, then lower token id.
// Keys are distinct, and 0 is below every real key.
__device__ __forceinline__ uint64_t tkey64(float l, uint32_t id) {
  return ((uint64_t)f2key(l) << 32) | (uint64_t)(0xFFFFFFFFu - id);
}

// Reductions over the four lanes r, r + 16, r + 32, r + 48 that hold one
// MFMA output column: permlane16_swap pairs rows 0-1 and 2-3 of the wave,
// permlane32_swap pairs the two halves; combining both outputs of each swap
// leaves every lane with the reduction in a fixed order.
__device__ __forceinline__ uint64_t col_max64(uint64_t k) {
  uint32_t hi = (uint32_t)(k >> 32), lo = (uint32_t)k;
  const auto h16 = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
  const auto l16 = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
  k = umax64(((uint64_t)h16[0] << 32) | l16[0], ((uint64_t)h16[1] << 32) | l16[1]);
  hi = (uint32_t)(k >> 32);
  lo = (uint32_t)k;
  const auto h32 = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
  const auto l32 = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
  return umax64(((uint64_t)h32[0] << 32) | l32[0], ((uint64_t)h32[1] << 32) | l32[1]);
}
__device__ __forceinline__ float col_sum(float x) {
  uint32_t u = __float_as_uint(x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  u = __float_as_uint(__uint_as_float(a[0]) + __uint_as_float(a[1]));
  const auto b = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Stores one 16-token x 64-row tile of logits and its statistics.  Logits
// are tile-major: logits[((grp * tpitch + t) * 64 + c) * 16 + i] for column
// c = j - 64 grp and token 16 t + i, so a tile is one contiguous 4 KB block
// (each store instruction writes 1 KB of whole lines) and a row's 16 logits
// of a tile are 64 contiguous bytes.  Statistics are blocked by 16 tiles:
// entry (t, c) at ((grp * tblocks + t / 16) * 64 + c) * 16 + t % 16, so 16
// consecutive tiles of a row fill one 128-byte line (written by the block's
// waves close together in time, read whole by the top-K kernel).
// D operand: lane (r, g) holds tokens t*16 + 4 g + q, q = 0..3, of column r.
// The scratch is padded (whole 32-token super-tiles, rows up to a multiple
// of 64), so the logits stores are in bounds and unconditional (columns
// past B and tokens past V hold junk that nothing reads).
__device__ __forceinline__ void tile_epilogue(const HeadArgs& a, uint32_t t, int r, int g,
                                              const f32x4* acc, uint64_t* bm) {
  const uint32_t i0 = t * 16 + 4 * g;
  const size_t tile = (size_t)blockIdx.y * a.tpitch + t;
#pragma unroll
  for (int bt = 0; bt < 4; ++bt) {
    const uint32_t c = bt * 16 + r;
    // Streamed past the L2 (read back only for the few candidate tiles).
    __builtin_nontemporal_store(acc[bt], (f32x4*)(a.logits + (tile * 64 + c) * 16 + 4 * g));
    // Tile statistics of column c: the largest (logit, id) key of the 16
    // tokens and the sum of exp(logit - tile max); all four lanes of the
    // column hold the same values and the first one writes them.
    uint64_t best = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      best = umax64(best, i0 + q < a.V ? tkey64(acc[bt][q], i0 + q) : (uint64_t)0);
    best = col_max64(best);
    bm[bt] = umax64(bm[bt], best);  // the wave's largest key of column c so far
    const float m = key2f((uint32_t)(best >> 32));
    float sum = 0.f;
#pragma unroll
    for (int q = 0; q < 4; ++q) sum += i0 + q < a.V ? __expf(acc[bt][q] - m) : 0.f;
    sum = col_sum(sum);
    if (g == 0) {
      const size_t o = (((size_t)blockIdx.y * a.tblocks + (t >> 4)) * 64 + c) * 16 + (t & 15);
      a.tkey[o] = best;
      a.tsum[o] = sum;
    }
  }
}

// One wave's logits for TPW consecutive 16-token tiles from t, accumulated
// in acc (a tile at or past t_hi re-reads tile t's rows; its accumulators
// are junk that the callers skip).  The tiles share each B-operand read of the
// staged hidden rows, so the LDS traffic per token falls with TPW; the W
// rows stream PC 64-element chunks per pass (PC x 2 TPW x 1 KB in flight
// per wave).
// W rows are read 128 contiguous bytes per row and instruction (8 lanes x
// 16 B, 8 rows): lane l holds row (l >> 3) (even group) or 8 + (l >> 3)
// (odd group) of a tile, elements 64 c + 8 (l & 7) .. + 8 of chunk c.  The
// MFMA wants lane (g, i) to hold row i, so each chunk of each tile passes
// through the wave's LDS staging tile (16 rows x 64 elements) and is read
// back in MFMA layout: step x of the chunk takes elements 64 c + 32 x +
// 8 g .. + 8.
template <int KS, int TPW, int PC>
__device__ __forceinline__ void logits_acc(const HeadArgs& a, uint32_t t, uint32_t t_hi,
                                           const __bf16* hs, __bf16* st, int hoff, int lane,
                                           int r, int g, f32x4 (&acc)[TPW][4]) {
  constexpr int D = KS * 32;
  constexpr int STRIDE = D + 8;  // staged hidden row pitch (elements)
  constexpr int NCH = D / 64;    // 64-element chunks per W row
  constexpr int SP = 72;         // W staging row pitch (elements)
  static_assert(NCH % PC == 0, "passes of whole chunks");
  const u32x4* wr[2 * TPW];
#pragma unroll
  for (int q = 0; q < 2 * TPW; ++q) {
    const uint32_t tt = t + (uint32_t)(q >> 1) < t_hi ? t + (uint32_t)(q >> 1) : t;
    const uint32_t row = tt * 16 + 8 * (q & 1) + (lane >> 3);
    wr[q] = (const u32x4*)a.w + ((size_t)min(row, a.V - 1) * D) / 8 + (lane & 7);
  }
#pragma unroll
  for (int i = 0; i < TPW; ++i)
#pragma unroll
    for (int bt = 0; bt < 4; ++bt) acc[i][bt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int h = 0; h < NCH / PC; ++h) {
    u32x4 v[2 * TPW][PC];
#pragma unroll
    for (int cc = 0; cc < PC; ++cc)
#pragma unroll
      for (int q = 0; q < 2 * TPW; ++q)
#if TFE_HEAD_NT
        v[q][cc] = __builtin_nontemporal_load(wr[q] + 8 * (h * PC + cc));
#else
        v[q][cc] = wr[q][8 * (h * PC + cc)];
#endif
    // Keep the pass's loads together ahead of its MFMAs (left alone, the
    // scheduler interleaves them and keeps only a few in flight).
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int cc = 0; cc < PC; ++cc) {
      const int c = h * PC + cc;
      u32x4 av[TPW][2];
#pragma unroll
      for (int i = 0; i < TPW; ++i) {
        *(u32x4*)(st + (lane >> 3) * SP + (lane & 7) * 8) = v[2 * i][cc];
        *(u32x4*)(st + (8 + (lane >> 3)) * SP + (lane & 7) * 8) = v[2 * i + 1][cc];
#pragma unroll
        for (int x = 0; x < 2; ++x) av[i][x] = *(const u32x4*)(st + r * SP + (4 * x + g) * 8);
      }
#pragma unroll
      for (int x = 0; x < 2; ++x) {
        u32x4 bv[4];
#pragma unroll
        for (int bt = 0; bt < 4; ++bt)
          bv[bt] = *(const u32x4*)(hs + hoff + bt * 16 * STRIDE + 64 * c + 32 * x);
#pragma unroll
        for (int bt = 0; bt < 4; ++bt)
#pragma unroll
          for (int i = 0; i < TPW; ++i)
            acc[i][bt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, av[i][x]), __builtin_bit_cast(bf16x8, bv[bt]),
                acc[i][bt], 0, 0, 0);
      }
    }
  }
}

// logits_acc, then the epilogue of every tile below t_hi.
template <int KS, int TPW, int PC>
__device__ __forceinline__ void logits_tiles(const HeadArgs& a, uint32_t t, uint32_t t_hi,
                                             const __bf16* hs, __bf16* st, int hoff, int lane,
                                             int r, int g, uint64_t* bm) {
  f32x4 acc[TPW][4];
  logits_acc<KS, TPW, PC>(a, t, t_hi, hs, st, hoff, lane, r, g, acc);
#pragma unroll
  for (int i = 0; i < TPW; ++i)
    if (t + (uint32_t)i < t_hi) tile_epilogue(a, t + i, r, g, acc[i], bm);
}

// Tiles per wave and chunks per pass of the logits kernel: three tiles
// with two-chunk passes (12 KB in flight per wave), then single tiles with
// four-chunk passes for the rest of a block's range.  (Measured on the
// 151936 x 1024 head at B = 64: 88.6 us per call against 93.0 for single
// tiles with eight-chunk passes; 2, 4 or 5 tiles, or longer passes, were
// slower.)
constexpr int kTileGroup = 3;
constexpr int kGroupChunks = 2;
constexpr int kSingleChunks = 4;

template <int KS>  // KS = D / 32 k-steps
__global__ __launch_bounds__(kLogitWaves * 64) void k_head_logits(const HeadArgs a) {
  constexpr int D = KS * 32;
  constexpr int STRIDE = D + 8;  // staged hidden row pitch (elements): conflict-free b128 reads
  constexpr int SP = 72;         // W staging row pitch (elements): conflict-free b128 reads
  __shared__ __attribute__((aligned(16))) __bf16 hs[kCols * STRIDE];
  __shared__ __attribute__((aligned(16))) __bf16 stage[kLogitWaves][16 * SP];
  __shared__ uint32_t s_next, s_next1;
  __shared__ unsigned long long s_bmax[kCols];  // the block's largest tile key per column
  if (threadIdx.x < kCols) s_bmax[threadIdx.x] = 0;
  const uint32_t col0 = blockIdx.y * kCols;
  const int ncols = (int)min((uint32_t)kCols, a.B - col0);
  for (int e = threadIdx.x; e < kCols * (D / 8); e += kLogitWaves * 64) {
    const int j = e / (D / 8), c = e - j * (D / 8);
    u32x4 v = {0u, 0u, 0u, 0u};
    if (j < ncols) v = *((const u32x4*)a.hidden + ((size_t)(col0 + j) * D) / 8 + c);
    *(u32x4*)(hs + j * STRIDE + c * 8) = v;
  }
  // The block owns a contiguous range of 16-token tiles; its waves claim
  // groups of kTileGroup tiles while whole groups remain, then single
  // tiles, so every wave stays busy until the range is done.
  const uint32_t nt = (a.V + 15) >> 4;
  const uint32_t t_lo = (uint32_t)((uint64_t)nt * blockIdx.x / gridDim.x);
  const uint32_t t_hi = (uint32_t)((uint64_t)nt * (blockIdx.x + 1) / gridDim.x);
  const uint32_t t_grp = t_lo + (t_hi - t_lo) / kTileGroup * kTileGroup;
  if (threadIdx.x == 0) {
    s_next = t_lo;
    s_next1 = t_grp;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r = lane & 15, g = lane >> 4;
  __bf16* st = stage[wave];
  // The staged hidden rows do not change across tiles; hiding the offset
  // from the optimiser keeps their LDS reads inside the loop (hoisted, the
  // whole 128 KB B operand would be held in registers and spill).
  int hoff = r * STRIDE + 8 * g;
  uint64_t bm[4] = {0, 0, 0, 0};  // column bt * 16 + r (lanes g = 0 hold it)
  for (;;) {
    uint32_t t = 0;
    if (lane == 0) t = atomicAdd(&s_next, (uint32_t)kTileGroup);
    t = __builtin_amdgcn_readfirstlane(t);
    if (t >= t_grp) break;
    asm volatile("" : "+v"(hoff));
    logits_tiles<KS, kTileGroup, kGroupChunks>(a, t, t_hi, hs, st, hoff, lane, r, g, bm);
  }
  for (;;) {
    uint32_t t = 0;
    if (lane == 0) t = atomicAdd(&s_next1, 1u);
    t = __builtin_amdgcn_readfirstlane(t);
    if (t >= t_hi) break;
    asm volatile("" : "+v"(hoff));
    logits_tiles<KS, 1, kSingleChunks>(a, t, t_hi, hs, st, hoff, lane, r, g, bm);
  }
  // The block's largest tile key per row (0 for a block without tiles),
  // from which the top-K kernel certifies a lower bound of each row's K-th
  // largest logit.
  if (g == 0) {
#pragma unroll
    for (int bt = 0; bt < 4; ++bt)
      if (bm[bt]) atomicMax(&s_bmax[bt * 16 + r], (unsigned long long)bm[bt]);
  }
  __syncthreads();
  if (threadIdx.x < kCols)
    a.bmax[((size_t)blockIdx.y * a.nblk + blockIdx.x) * kCols + threadIdx.x] = s_bmax[threadIdx.x];
}

// Wave-wide reductions and scans with DPP (rows of 16 lanes) and readlane,
// in a fixed order, without LDS round trips.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}

__device__ __forceinline__ float wave_add(float x) {
  x += __uint_as_float(dpp_u32<0xB1>(__float_as_uint(x)));   // quad_perm [1,0,3,2]
  x += __uint_as_float(dpp_u32<0x4E>(__float_as_uint(x)));   // quad_perm [2,3,0,1]
  x += __uint_as_float(dpp_u32<0x141>(__float_as_uint(x)));  // row_half_mirror
  x += __uint_as_float(dpp_u32<0x140>(__float_as_uint(x)));  // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return (r0 + r1) + (r2 + r3);
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x) {
  x = max(x, dpp_u32<0xB1>(x));
  x = max(x, dpp_u32<0x4E>(x));
  x = max(x, dpp_u32<0x141>(x));
  x = max(x, dpp_u32<0x140>(x));
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)x, 0);
  const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 16);
  const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)x, 32);
  const uint32_t r3 = (uint32_t)__builtin_amdgcn_readlane((int)x, 48);
  return max(max(r0, r1), max(r2, r3));
}

// Inclusive sum over the lanes up to this one: shifts within each 16-lane
// row, then the totals of the rows below.
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  const int lane = threadIdx.x & 63;
  x += dpp_u32<0x111>(x);  // row_shr:1
  x += dpp_u32<0x112>(x);  // row_shr:2
  x += dpp_u32<0x114>(x);  // row_shr:4
  x += dpp_u32<0x118>(x);  // row_shr:8
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)x, 15);
  const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 31);
  const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)x, 47);
  const int row = lane >> 4;
  return x + (row >= 1 ? r0 : 0u) + (row >= 2 ? r1 : 0u) + (row >= 3 ? r2 : 0u);
}

// Bitonic sort of a[0, N2) in LDS, descending; N2 a power of two.
template <int NT>
__device__ void lds_sort_desc(uint64_t* a, uint32_t N2) {
  for (uint32_t size = 2; size <= N2; size <<= 1) {
    for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
      for (uint32_t e = threadIdx.x; e < N2 / 2; e += NT) {
        const uint32_t i = 2 * e - (e & (stride - 1));
        const uint32_t j = i + stride;
        const bool desc = (i & size) == 0;
        const uint64_t x = a[i], y = a[j];
        if ((x < y) == desc) {
          a[i] = y;
          a[j] = x;
        }
      }
      __syncthreads();
    }
  }
}

__device__ __forceinline__ uint32_t pow2_ceil(uint32_t x) {
  uint32_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

constexpr int kRowThreads = 1024;
constexpr int kRowTiles = kHeadMaxTiles / kRowThreads;  // tile entries per thread
constexpr int kRowCand = 16 * kHeadMaxK;                // logits of the candidate tiles

// Appends the tiles whose masked key reaches lo ((key & msk) >= lo) to
// s_tiles, in no particular order (the ranking does not depend on it): each
// wave appends its tiles with one LDS atomic.  *s_n counts every such tile;
// the list is cut at its capacity.
template <int NI, int NT_>
__device__ __forceinline__ void list_tiles(const uint64_t (&key)[NI], uint32_t NT, uint64_t msk,
                                           uint64_t lo, uint32_t* s_tiles, uint32_t* s_n) {
  const int tid = threadIdx.x, lane = tid & 63;
  const uint64_t below = (1ull << lane) - 1ull;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const uint32_t t = tid + i * NT_;
    const bool in = t < NT && (key[i] & msk) >= lo;
    const uint64_t m = __builtin_amdgcn_ballot_w64(in);
    if (m) {
      uint32_t base = 0;
      if (lane == 0) base = atomicAdd(s_n, (uint32_t)__builtin_popcountll(m));
      base = __builtin_amdgcn_readfirstlane(base);
      const uint32_t off = base + (uint32_t)__builtin_popcountll(m & below);
      if (in && off < (uint32_t)kHeadMaxK) s_tiles[off] = t;
    }
  }
}

// Per row: the K most likely tokens and their probabilities from the tile
// statistics and the logits.
//   1. M = max logit, S = sum over tiles of tsum * exp(tile max - M).
//   2. A lower bound of the K-th largest logit from the logits blocks'
//      largest keys (one 8-bit histogram of 256 values) usually lists the
//      candidate tiles in one pass.  Otherwise a radix select over the
//      tile-max keys (8-bit digits from the highest bit in which they
//      differ; one LDS histogram per pass) narrows the tiles to the bins at
//      and above the one holding the K-th largest key; it stops when those
//      hold at most 192 tiles (or exactly K).  The K tiles with the largest
//      maxima are among them and hold every top-K logit, and every top-K
//      logit is at or above the bins' lower bound.
//   3. The logits of those tiles at or above that bound are ranked in LDS,
//      by counting when there are at most 1024 of them, else by a bitonic
//      sort; the first K are the answer.  The tile and logit lists are
//      built with wave-aggregated LDS appends in no particular order (the
//      ranking does not depend on it; keys are distinct), which took the
//      call from 87.5 to 81.9 us against block-wide scans per round.
__global__ __launch_bounds__(kRowThreads) void k_head_rows(const HeadArgs a) {
  __shared__ uint64_t s_cand[kRowCand];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t s_tiles[kHeadMaxK];
  __shared__ uint32_t s_wave[kRowThreads / 64];
  __shared__ uint32_t s_wmin[kRowThreads / 64];
  __shared__ uint32_t s_bwmax[kRowThreads / 64], s_bwmin[kRowThreads / 64];
  __shared__ float s_red[kRowThreads / 64];
  __shared__ uint32_t s_bin, s_above, s_cnt, s_ntile, s_nc;
  __shared__ unsigned long long s_lo;
  const uint32_t b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) {
    s_ntile = 0;
    s_nc = 0;
    s_lo = 0;
  }
  const uint32_t NT = (a.V + 15) >> 4;
  // Statistics of tile t of this row: block t / 16 of the row's 64-row
  // group, column c, slot t % 16.
  const size_t grp = b >> 6, c = b & 63;
  const uint64_t* tk = a.tkey + (grp * a.tblocks * 64 + c) * 16;
  const float* ts = a.tsum + (grp * a.tblocks * 64 + c) * 16;
  auto sidx = [](uint32_t t) { return (size_t)(t >> 4) * 1024 + (t & 15); };

  // Tile keys and sums, and the logits blocks' largest keys of this row
  // (step 2a), are loaded together (one round trip).
  const uint32_t take = min(a.K, NT);
  const bool bound = take < NT && a.K <= a.nblk && a.nblk <= (uint32_t)kRowThreads;
  const uint64_t bmv = bound && (uint32_t)tid < a.nblk
                           ? a.bmax[(grp * a.nblk + (uint32_t)tid) * 64 + c] : 0;  // 0: none
  uint64_t key[kRowTiles];
  float tsv[kRowTiles];
#pragma unroll
  for (int i = 0; i < kRowTiles; ++i) {
    const uint32_t t = tid + i * kRowThreads;
    key[i] = t < NT ? tk[sidx(t)] : 0;
    tsv[i] = t < NT ? ts[sidx(t)] : 0.f;
  }
  // High key words of this thread's tiles (absent tiles hold key 0, below
  // every real one, so they only count for the minimum when skipped).
  uint32_t hmax = 0, hmin = 0xFFFFFFFFu;
#pragma unroll
  for (int i = 0; i < kRowTiles; ++i) {
    const uint32_t hw = (uint32_t)(key[i] >> 32);
    hmax = max(hmax, hw);
    hmin = min(hmin, key[i] ? hw : 0xFFFFFFFFu);
  }
  // 1. Log-sum-exp over the tiles.  The largest logit is the largest high
  // key word; the tile terms use the hardware exponential (the tile sums do
  // too; relative error about an ulp per term).
  hmax = wave_max_u32(hmax);
  hmin = ~wave_max_u32(~hmin);
  uint32_t bhmax = wave_max_u32((uint32_t)(bmv >> 32));
  uint32_t bhmin = ~wave_max_u32(bmv ? ~(uint32_t)(bmv >> 32) : 0u);
  if (lane == 0) {
    s_wave[wave] = hmax;
    s_wmin[wave] = hmin;
    s_bwmax[wave] = bhmax;
    s_bwmin[wave] = bhmin;
  }
  __syncthreads();
  hmax = bhmax = 0;
  hmin = bhmin = 0xFFFFFFFFu;
  for (int w = 0; w < kRowThreads / 64; ++w) {
    hmax = max(hmax, s_wave[w]);
    hmin = min(hmin, s_wmin[w]);
    bhmax = max(bhmax, s_bwmax[w]);
    bhmin = min(bhmin, s_bwmin[w]);
  }
  const float M = key2f(hmax);
  // Each wave's part of S = sum over tiles of tsum * exp(tile max - M); the
  // parts are added up after a later barrier (step 3).
  {
    float part = 0.f;
#pragma unroll
    for (int i = 0; i < kRowTiles; ++i) {
      const uint32_t t = tid + i * kRowThreads;
      if (t < NT) part += tsv[i] * __expf(key2f((uint32_t)(key[i] >> 32)) - M);
    }
    part = wave_add(part);
    if (lane == 0) s_red[wave] = part;
  }

  // 2. Candidate tiles.  Every top-K logit lies in a tile whose largest key
  // reaches the row's K-th largest logit key, and reaches it itself, so for
  // any lower bound tau of that key the tiles with a key >= tau hold every
  // answer, and their logits >= tau include it.
  uint64_t tau = 0;
  bool listed = false;
  // 2a. A certified bound, when K is at most the number of logits blocks:
  // at least K of the blocks' largest keys reach it, and they are distinct
  // logit keys, so the row's K-th largest logit key reaches it too.  One
  // 8-bit histogram of the block maxima (from the highest bit in which they
  // differ) gives the bin holding their K-th largest; its lower edge is the
  // bound.  One pass lists the tiles that reach it; if they overflow the
  // list, the radix select below takes over.
  if (bound) {
    const uint32_t dh = bhmin ^ bhmax;
    const int top = dh ? 63 - __builtin_clz(dh) : 31;
    const int sh = max(top - 7, 0);
    const uint64_t cm =
        sh + 8 < 64 ? ((uint64_t)bhmax << 32) & ~((1ull << (sh + 8)) - 1ull) : 0ull;
    if (tid < 256) hist[tid] = 0u;
    __syncthreads();
    if (bmv) atomicAdd(&hist[(uint32_t)(bmv >> sh) & 255u], 1u);
    __syncthreads();
    if (wave == 0) {  // the bin where the count from the top reaches K
      uint32_t v[4], sum = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        v[k] = hist[255 - 4 * lane - k];
        sum += v[k];
      }
      const uint32_t inc = wave_incl_scan(sum);
      uint32_t ex = inc - sum;
      if (ex < a.K && a.K <= inc) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          if (ex < a.K && a.K <= ex + v[k])
            s_lo = cm | ((uint64_t)(255u - 4u * (uint32_t)lane - (uint32_t)k) << sh);
          ex += v[k];
        }
      }
    }
    __syncthreads();
    const uint64_t lo = s_lo;  // 0: fewer than K blocks with tiles
    if (lo != 0) {
      list_tiles<kRowTiles, kRowThreads>(key, NT, ~0ull, lo, s_tiles, &s_ntile);
      __syncthreads();
      const uint32_t n = s_ntile;
      __syncthreads();  // every thread has read s_ntile
      if (n <= (uint32_t)kHeadMaxK) {
        listed = true;
        tau = lo;
      } else if (tid == 0) {
        s_ntile = 0;  // the radix select's first barrier orders this
      }
    }
  }
  if (!listed) {
    // 2b. The K-th largest tile key (all tiles when there are at most K).
    uint64_t prefix = 0, mask = 0, common = 0;
    if (take < NT) {
      // Radix select from the highest bit in which the tile keys differ (the
      // high words of all keys lie between hmin and hmax, so they agree above
      // the top bit of hmin ^ hmax), 8 bits per pass.  It stops once the bins
      // at and above the chosen one hold at most kStopCand tiles: every
      // answer lies in those tiles, so the K-th largest key itself is not
      // needed.
      constexpr uint32_t kStopCand = 192;
      static_assert(kStopCand <= kHeadMaxK, "candidate tiles must fit s_tiles");
      const uint32_t dhi = hmin ^ hmax;
      const int top = dhi ? 63 - __builtin_clz(dhi) : 31;  // highest differing bit (low word: 31)
      const int shift0 = max(top - 7, 0);
      // Bits above the first digit, shared by every key (all in the high word).
      if (shift0 + 8 < 64) common = ((uint64_t)hmax << 32) & ~((1ull << (shift0 + 8)) - 1ull);
      uint32_t need = take, above = 0;
      const uint64_t lt = (1ull << lane) - 1ull;
      for (int shift = shift0;; shift = max(shift - 8, 0)) {
        if (tid < 256) hist[tid] = 0u;
        __syncthreads();
        // The lanes holding the first active lane's digit add their number
        // with one atomic (the top digits of tile maxima are mostly equal).
#pragma unroll
        for (int i = 0; i < kRowTiles; ++i) {
          if (tid + i * kRowThreads < NT && (key[i] & mask) == prefix) {
            const uint32_t d = (uint32_t)(key[i] >> shift) & 255u;
            const uint32_t d0 = __builtin_amdgcn_readfirstlane(d);
            const uint64_t m = __builtin_amdgcn_ballot_w64(d == d0);
            if (d != d0) atomicAdd(&hist[d], 1u);
            else if ((m & lt) == 0) atomicAdd(&hist[d0], (uint32_t)__builtin_popcountll(m));
          }
        }
        __syncthreads();
        // Wave 0 finds the bin holding the need-th largest key: lane l holds
        // bins 255 - 4 l - k, k = 0..3 (descending order).
        if (wave == 0) {
          uint32_t v[4], sum = 0;
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            v[k] = hist[255 - 4 * lane - k];
            sum += v[k];
          }
          const uint32_t inc = wave_incl_scan(sum);
          uint32_t ex = inc - sum;
          if (ex < need && need <= inc) {
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              if (ex < need && need <= ex + v[k]) {
                s_bin = 255u - 4u * (uint32_t)lane - (uint32_t)k;
                s_above = ex;
                s_cnt = v[k];
              }
              ex += v[k];
            }
          }
        }
        __syncthreads();
        need -= s_above;
        above += s_above;
        prefix |= (uint64_t)s_bin << shift;  // bits below the previous digit only
        mask |= (uint64_t)0xFF << shift;
        // Every thread has read s_bin / s_above / s_cnt before wave 0 can
        // write them again (two barriers of the next pass come first).
        if (s_cnt == need || above + s_cnt <= kStopCand || shift == 0) break;
      }
    }
    // Candidate tiles: the keys whose masked bits reach the prefix (at most
    // max(K, kStopCand) of them, the keys being distinct); every answer
    // logit is at or above the prefix.  The list is cut at its capacity all
    // the same, so that statistics that were never written (equal keys)
    // cannot make the block write past it.
    list_tiles<kRowTiles, kRowThreads>(key, NT, mask, prefix, s_tiles, &s_ntile);
    // (With all tiles taken, every logit is a candidate.)
    tau = take == NT ? 0 : (common | prefix);
    __syncthreads();
  }
  const uint32_t ntile = min(s_ntile, (uint32_t)kHeadMaxK);
  const uint64_t below = (1ull << lane) - 1ull;

  // 3. Gather the candidate tiles' logits at or above tau, sort, emit.
  const float* lg = a.logits + (grp * a.tpitch * 64 + c) * 16;  // tile t at lg[1024 t]
  // All candidate logits are loaded first (16 per tile, kRowThreads per
  // round; the logits scratch holds whole tiles, so the reads past V stay
  // in it), and the logits at or above tau are appended, wave by wave, to
  // the candidates.
  constexpr int kRounds = kRowCand / kRowThreads;
  const uint32_t nlog = 16 * ntile;  // <= kRowCand
  float lv[kRounds];
#pragma unroll
  for (int j = 0; j < kRounds; ++j) {
    const uint32_t e = j * kRowThreads + tid;
    lv[j] = 0.f;
    if (e < nlog) lv[j] = lg[1024 * (size_t)s_tiles[e >> 4] + (e & 15)];
  }
#pragma unroll
  for (int j = 0; j < kRounds; ++j) {
    const uint32_t e = j * kRowThreads + tid;
    uint64_t ck = 0;
    bool keep = false;
    if (e < nlog) {
      const uint32_t v = 16 * s_tiles[e >> 4] + (e & 15);
      if (v < a.V) {
        ck = tkey64(lv[j], v);
        keep = ck >= tau;
      }
    }
    const uint64_t m = __builtin_amdgcn_ballot_w64(keep);
    if (m) {
      uint32_t base = 0;
      if (lane == 0) base = atomicAdd(&s_nc, (uint32_t)__builtin_popcountll(m));
      base = __builtin_amdgcn_readfirstlane(base);
      if (keep) s_cand[base + (uint32_t)__builtin_popcountll(m & below)] = ck;
    }
  }
  __syncthreads();
  float S = 0.f;
  for (int w = 0; w < kRowThreads / 64; ++w) S += s_red[w];
  const uint32_t n_c = s_nc;
  const float invS = 1.0f / S;
  auto emit = [&](uint32_t i, uint64_t k) {
    a.top_ids[(size_t)b * a.K + i] = (int32_t)(0xFFFFFFFFu - (uint32_t)k);
    a.top_prob[(size_t)b * a.K + i] = expf(key2f((uint32_t)(k >> 32)) - M) * invS;
  };
  if (n_c <= (uint32_t)kRowThreads) {
    // Usually a little over K candidates: each thread ranks its own by
    // counting the larger ones (keys are distinct; every thread reads the
    // same LDS word at a time), with no sorting network.
    if ((uint32_t)tid < n_c) {
      const uint64_t k = s_cand[tid];
      uint32_t rank = 0;
      for (uint32_t u = 0; u < n_c; ++u) rank += s_cand[u] > k ? 1u : 0u;
      if (rank < a.K) emit(rank, k);
    }
    return;
  }
  const uint32_t N2 = pow2_ceil(n_c);
  for (uint32_t e = n_c + tid; e < N2; e += kRowThreads) s_cand[e] = 0;
  __syncthreads();
  lds_sort_desc<kRowThreads>(s_cand, N2);
  for (uint32_t i = tid; i < a.K; i += kRowThreads) emit(i, s_cand[i]);
}


// ---------------------------------------------------------------------------
// One launch for up to 64 rows (K at most the number of blocks).
//
// The two launches above write every logit (39 MB for the 151936-token head
// at B = 64) so that the second can select from them, and read back about 2%
// of them.  Here each wave keeps the logits of its tile groups (at most two)
// in registers, and two grid barriers take the place of that write:
//   A. the logits as in k_head_logits (one block per compute unit, the same
//      tiles; claiming the second tile groups device-wide instead, first
//      come first served, made the call slower, 93.2 against 73.4 us: the
//      compute units that finish early take too many); after each tile
//      group the wave folds its logits into a
//      running per-row maximum and sum of exp(logit - maximum), which hides
//      that arithmetic under the other waves' loads; each block publishes
//      per row its largest logit (as a key) and its sum;
//   B. after the first barrier every block derives, per row, a lower bound
//      of the row's K-th largest logit: split the blocks into G >= K
//      disjoint non-empty groups; each group holds a logit at least as
//      large as the smallest of the G group maxima, and these G logits are
//      distinct entries of the row, so the G-th largest logit, and with it
//      the K-th, reaches that minimum;
//   C. each block writes the (logit, id) keys of its logits at or above the
//      bound (a few per row) to its own segment of the row's candidate list;
//   D. after the second barrier block r ranks row r: M and S from the
//      published maxima and sums, then a radix select of the K largest
//      candidates in LDS (first over the segments in memory when more than
//      LDS holds, which only heavy ties produce), emitted with exp(l - M) / S.
// Data that crosses blocks is stored and loaded with device scope (cache
// policy sc1: the stores write through the XCD's L2 and the loads do not
// take stale L2 lines), and each wave's stores have completed before its
// block counts itself in at a barrier.
// The barriers need all blocks resident at once: one block per compute
// unit fits (the LDS allows no second), and the launch is an ordinary one
// (a cooperative launch, which guarantees residency, cost about 15 us more
// per call).  So a call must not overlap on the device with other work that
// holds compute units while it waits for this call, such as a one-launch
// head call of another head on another stream.  The waits are bounded
// (about a second); if one runs out, that call answers every row with ids
// -1 and probabilities 0.
constexpr int kFuseThreads = kLogitWaves * 64;
constexpr int kFuseGroups = 2;      // tile groups a wave computes and holds
constexpr uint32_t kFuseMaxBlocks = 256;

template <typename T>
__device__ __forceinline__ void st_agent(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T ld_agent(const T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// 16 bytes at base + off with device scope (buffer load, cache policy sc1).
__device__ __forceinline__ u32x4 ld_agent16(const void* base, uint32_t off) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, 0x7FFFFFFF, 0x00020000);
  return __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 16);
}

// The call's epoch (one-launch calls made before it on this scratch) lives
// in device memory, so that a captured graph replays correctly: every block
// adds one to counter b mod 16 of ectl (each in a 128-byte line of its own)
// as it leaves, without waiting for the result, and the next call -- which
// starts only once this one has ended, its additions included -- takes the
// sum of the counters over the number of blocks as its epoch.
constexpr uint32_t kLeaveCtrs = 16;

__device__ __forceinline__ uint64_t call_epoch(const HeadArgs& a) {
  unsigned long long n = 0;
#pragma unroll
  for (uint32_t i = 0; i < kLeaveCtrs; ++i)
    n += __hip_atomic_load(a.ectl + 16 * i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return n / a.nblk;
}

__device__ __forceinline__ void leave_call(const HeadArgs& a) {
  if (threadIdx.x == 0)
    (void)__hip_atomic_fetch_add(a.ectl + 16 * (blockIdx.x % kLeaveCtrs), 1ull, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
}

// Barrier j (1 or 2) of the call with epoch e, called by every thread, as a
// two-level tree: block b counts into the counter of its group b % 16 (each
// counter in a 128-byte line of its own), the last block of a group into the
// root counter, and the last group releases every group's flag; a block
// then waits on its group's flag.  Every launch passes each barrier once per
// block, so a group of n blocks is complete at barrier j once its counter
// reaches (2 e + j) n, and the release value is 2 e + j.  (One counter that
// every block counts into and polls took 9-13 us from the last arrival to
// the release: its reads and atomics queue behind each other.)  Thread 0
// counts the block in after all its waves' stores have completed
// (s_waitcnt vmcnt(0)); with `wait`, it then waits for the release.
constexpr uint32_t kBarGroups = 16;
constexpr uint32_t kBarLine = 16;  // 64-bit words per 128-byte line

__device__ __forceinline__ void grid_barrier(const HeadArgs& a, uint64_t epoch, uint32_t j,
                                             bool wait) {
  __builtin_amdgcn_s_waitcnt(0x0F70);
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t nb = a.nblk, grp = blockIdx.x % kBarGroups;
    const uint32_t ngrp = min(nb, kBarGroups);
    const uint64_t gsize = nb / kBarGroups + (grp < nb % kBarGroups ? 1u : 0u);
    const uint64_t phase = 2ull * epoch + j;
    unsigned long long* cnt = a.bar + kBarLine * (1 + grp);
    unsigned long long* root = a.bar;
    unsigned long long* flag = a.bar + kBarLine * (1 + kBarGroups);
    const unsigned long long old =
        __hip_atomic_fetch_add(cnt, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old + 1 == phase * gsize) {
      const unsigned long long r =
          __hip_atomic_fetch_add(root, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (r + 1 == phase * ngrp)
        for (uint32_t q = 0; q < ngrp; ++q) st_agent(flag + kBarLine * q, (unsigned long long)phase);
    }
    if (wait) {
      const unsigned long long* f = flag + kBarLine * grp;
      for (uint32_t n = 0; ld_agent(f) < phase; ++n) {
        if (n == a.wait_limit) {
          atomicMax(a.fault, (unsigned long long)epoch + 1ull);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
      }
    }
  }
  __syncthreads();
}

// (m, s) <- the merge of two partial softmax sums: m the largest logit, s
// the sum of exp(logit - m); (-inf, 0) is empty.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -INFINITY) return;
  s = s * __expf(m - mm) + s2 * __expf(m2 - mm);
  m = mm;
}

// lse_merge over the four lanes of one MFMA output column (as col_sum).
__device__ __forceinline__ void col_lse(float& m, float& s) {
  uint32_t um = __float_as_uint(m), us = __float_as_uint(s);
  const auto m16 = __builtin_amdgcn_permlane16_swap(um, um, false, false);
  const auto s16 = __builtin_amdgcn_permlane16_swap(us, us, false, false);
  m = __uint_as_float(m16[0]);
  s = __uint_as_float(s16[0]);
  lse_merge(m, s, __uint_as_float(m16[1]), __uint_as_float(s16[1]));
  um = __float_as_uint(m);
  us = __float_as_uint(s);
  const auto m32 = __builtin_amdgcn_permlane32_swap(um, um, false, false);
  const auto s32 = __builtin_amdgcn_permlane32_swap(us, us, false, false);
  m = __uint_as_float(m32[0]);
  s = __uint_as_float(s32[0]);
  lse_merge(m, s, __uint_as_float(m32[1]), __uint_as_float(s32[1]));
}

// Wave 0 finds the histogram bin that holds the need-th largest key (lane l
// holds bins 255 - 4 l - k, k = 0..3, in descending order) and leaves the
// bin, the count above it and its own count in s_sel[0..2].
__device__ __forceinline__ void pick_bin(const uint32_t* hist, uint32_t need, uint32_t* s_sel) {
  const int lane = threadIdx.x & 63;
  uint32_t v[4], sum = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[k] = hist[255 - 4 * lane - k];
    sum += v[k];
  }
  const uint32_t inc = wave_incl_scan(sum);
  uint32_t ex = inc - sum;
  if (ex < need && need <= inc) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (ex < need && need <= ex + v[k]) {
        s_sel[0] = 255u - 4u * (uint32_t)lane - (uint32_t)k;
        s_sel[1] = ex;
        s_sel[2] = v[k];
      }
      ex += v[k];
    }
  }
}

// Adds a key to the radix histogram of the current pass if it agrees with
// the decided bits (lanes holding the first active lane's digit add their
// number with one atomic).
__device__ __forceinline__ void hist_key(uint32_t* hist, bool in, uint64_t key, uint64_t dm,
                                         uint64_t lo, int sh) {
  in = in && (key & dm) == lo;
  const uint64_t act = __builtin_amdgcn_ballot_w64(in);
  if (!act) return;
  const uint32_t d = (uint32_t)(key >> sh) & 255u;
  const int first = __builtin_ctzll(act);
  const uint32_t d0 = (uint32_t)__builtin_amdgcn_readlane((int)d, first);
  const uint64_t same = __builtin_amdgcn_ballot_w64(in && d == d0);
  const int lane = threadIdx.x & 63;
  if (in && d != d0) atomicAdd(&hist[d], 1u);
  else if (lane == first) atomicAdd(&hist[d0], (uint32_t)__builtin_popcountll(same));
}

template <int KS>
__global__ __launch_bounds__(kFuseThreads) void k_head_fused(const HeadArgs a) {
  constexpr int D = KS * 32;
  constexpr int STRIDE = D + 8;
  constexpr int SP = 72;
  // The staged hidden rows; in phase D the candidates of the block's row.
  __shared__ __attribute__((aligned(16))) __bf16 hs[kCols * STRIDE];
  __shared__ __attribute__((aligned(16))) __bf16 stage[kLogitWaves][16 * SP];
  __shared__ float s_wm[kLogitWaves][kCols], s_ws[kLogitWaves][kCols];
  __shared__ uint32_t s_bound[kCols], s_cnt[kCols];
  __shared__ uint32_t s_off[kFuseMaxBlocks + 1];
  __shared__ uint32_t hist[256];
  __shared__ unsigned long long s_top[kHeadMaxK];
  __shared__ uint32_t s_wtot[kLogitWaves], s_wmax[kLogitWaves];
  __shared__ float s_red[kLogitWaves];
  __shared__ uint32_t s_next, s_n, s_sel[3];
  constexpr uint32_t kLds = sizeof(hs) / 8;  // candidates selected in LDS
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r = lane & 15, g = lane >> 4;
  const uint32_t b = blockIdx.x, nblk = a.nblk, B = a.B, K = a.K;

  // A. Logits of the block's tiles, held in registers; per (lane, row) the
  // running maximum rm and sum rs of exp(logit - rm).
  if (tid < kCols) s_cnt[tid] = 0;
  for (int e = tid; e < kCols * (D / 8); e += kFuseThreads) {
    const int j = e / (D / 8), c = e - j * (D / 8);
    u32x4 v = {0u, 0u, 0u, 0u};
    if ((uint32_t)j < B) v = *((const u32x4*)a.hidden + ((size_t)j * D) / 8 + c);
    *(u32x4*)(hs + j * STRIDE + c * 8) = v;
  }
  const uint32_t nt = (a.V + 15) >> 4;
  const uint32_t t_lo = (uint32_t)((uint64_t)nt * b / nblk);
  const uint32_t t_hi = (uint32_t)((uint64_t)nt * (b + 1) / nblk);
  // The epoch is read now and first used at the first barrier (thread 0
  // takes part in both); the other threads get it through LDS there.
  uint64_t ep = 0;
  if (tid == 0) {
    s_next = t_lo;
    ep = call_epoch(a);
  }
  __syncthreads();
  __bf16* st = stage[wave];
  int hoff = r * STRIDE + 8 * g;
  f32x4 acc[kFuseGroups][kTileGroup][4];
  uint32_t tg[kFuseGroups];
  float rm[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY}, rs[4] = {0.f, 0.f, 0.f, 0.f};
  // Held logit (k, i, bt, q): tile tg[k] + i, token 16 (tg[k] + i) + 4 g + q,
  // row bt * 16 + r; it exists if the tile is below t_hi and the token
  // below V (tile-uniform tests first).
  auto held = [&](int k, int i) { return tg[k] < t_hi && tg[k] + (uint32_t)i < t_hi; };
  auto whole = [&](int k, int i) { return (tg[k] + (uint32_t)i) * 16 + 16 <= a.V; };
#pragma unroll
  for (int k = 0; k < kFuseGroups; ++k) {
    uint32_t t = 0;
    if (lane == 0) t = atomicAdd(&s_next, (uint32_t)kTileGroup);
    tg[k] = __builtin_amdgcn_readfirstlane(t);
#pragma unroll
    for (int i = 0; i < kTileGroup; ++i)
#pragma unroll
      for (int bt = 0; bt < 4; ++bt) acc[k][i][bt] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (tg[k] < t_hi) {
      asm volatile("" : "+v"(hoff));
      logits_acc<KS, kTileGroup, kGroupChunks>(a, tg[k], t_hi, hs, st, hoff, lane, r, g, acc[k]);
#pragma unroll
      for (int bt = 0; bt < 4; ++bt) {
        float x[kTileGroup][4];
        float gmx = -INFINITY;
#pragma unroll
        for (int i = 0; i < kTileGroup; ++i)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t id = (tg[k] + i) * 16 + 4 * g + q;
            x[i][q] = held(k, i) && (whole(k, i) || id < a.V) ? acc[k][i][bt][q] : -INFINITY;
            gmx = fmaxf(gmx, x[i][q]);
          }
        const float mm = fmaxf(rm[bt], gmx);
        if (mm != -INFINITY) {
          float s = rs[bt] * __expf(rm[bt] - mm);
#pragma unroll
          for (int i = 0; i < kTileGroup; ++i)
#pragma unroll
            for (int q = 0; q < 4; ++q) s += __expf(x[i][q] - mm);
          rs[bt] = s;
          rm[bt] = mm;
        }
      }
    }
  }
  // The block's maximum and sum per row: the four lanes of each column,
  // then the eight waves in a fixed order.
#pragma unroll
  for (int bt = 0; bt < 4; ++bt) {
    col_lse(rm[bt], rs[bt]);
    if (g == 0) {
      s_wm[wave][bt * 16 + r] = rm[bt];
      s_ws[wave][bt * 16 + r] = rs[bt];
    }
  }
  __syncthreads();
  if ((uint32_t)tid < B) {
    float m = -INFINITY, s = 0.f;
    for (int w = 0; w < kLogitWaves; ++w) lse_merge(m, s, s_wm[w][tid], s_ws[w][tid]);
    st_agent(a.bhi + (size_t)tid * nblk + b, m == -INFINITY ? 0u : f2key(m));
    st_agent(a.bsum + (size_t)tid * nblk + b, __float_as_uint(s));
  }
  if (tid == 0) s_top[0] = ep;  // s_top is next written in phase D
  grid_barrier(a, ep, 1, true);
  ep = s_top[0];

  // B. Per row, the smallest of G group maxima (high key words; 0 for a
  // block without logits), G the least power of two >= K (G >= K groups
  // bound the G-th largest logit, which is at most the K-th): groups of
  // nblk / G consecutive blocks, nblk a power of two.  Wave w takes rows
  // 8 w .. 8 w + 7; lane l loads blocks 4 l .. 4 l + 3 of a row with one
  // 16-byte load.  A block that ranks a row in phase D also loads that
  // row's block maxima and sums here, for M and S.
  uint32_t fbh = 0;
  float fbs = 0.f;
  {
    uint32_t G = 1;
    while (G < K) G <<= 1;
    const uint32_t sg = nblk / G;  // blocks per group, a power of two
    const uint32_t om = (4u * K + nblk - 1u) / nblk;
    const bool mine = 4u * (uint32_t)lane < nblk;
    u32x4 v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const uint32_t row = (uint32_t)wave * 8 + q;
      v[q] = u32x4{0u, 0u, 0u, 0u};
      if (row < B && mine) v[q] = ld_agent16(a.bhi, (row * nblk + 4u * (uint32_t)lane) * 4u);
    }
    if (b < B && (uint32_t)tid < nblk) {
      fbh = ld_agent(a.bhi + (size_t)b * nblk + tid);
      fbs = __uint_as_float(ld_agent(a.bsum + (size_t)b * nblk + tid));
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const u32x4 x = v[q];
      const uint32_t a0 = max(x[0], x[1]), a1 = max(x[2], x[3]);
      uint32_t m;
      if (sg == 1) {
        m = min(min(x[0], x[1]), min(x[2], x[3]));
      } else if (sg == 2) {
        m = min(a0, a1);
      } else {  // a group spans sg / 4 aligned lanes
        m = max(a0, a1);
        for (uint32_t o = 1; o < sg / 4; o <<= 1) m = max(m, (uint32_t)__shfl_xor((int)m, (int)o));
      }
      m = ~wave_max_u32(mine ? ~m : 0u);
      // A second bound, the larger one is kept: blocks in groups of four
      // (one lane); the om largest maxima of a group, om = ceil(4 K / nblk)
      // <= 4, are distinct logits of the row, (nblk / 4) om >= K of them,
      // each at least the group's om-th largest.  (Groups of eight, with a
      // sort across lane pairs, halved the candidates again but cost as
      // much in this step as they saved later.)
      if (om == 2u || om == 3u) {
        const uint32_t lo0 = min(x[0], x[1]), lo1 = min(x[2], x[3]);
        const uint32_t ms = om == 2u ? max(min(a0, a1), max(lo0, lo1))   // second largest
                                     : min(max(lo0, lo1), min(a0, a1));  // third largest
        m = max(m, ~wave_max_u32(mine ? ~ms : 0u));
      }
      if (lane == 0) s_bound[wave * 8 + q] = m;
    }
    const uint32_t wm = wave_max_u32(fbh);
    if (lane == 0) s_wmax[wave] = wm;
  }
  __syncthreads();
  // Row b's largest logit M and its part of S = sum over blocks of
  // bsum exp(block max - M) (added up in phase D).
  uint32_t hmax = 0;
  for (int w = 0; w < kLogitWaves; ++w) hmax = max(hmax, s_wmax[w]);
  const float M = key2f(hmax);
  {
    float part = fbh ? fbs * __expf(key2f(fbh) - M) : 0.f;
    part = wave_add(part);
    if (lane == 0) s_red[wave] = part;
  }

  // C. Keys of the held logits that reach their row's bound (compared as
  // floats: a superset of the keys at or above it, which differs only by
  // -0 at a bound of +0).  The four logits of a lane, tile and row are
  // tested against the bound through their maximum first.  (Counting each
  // lane's candidates first and reserving their places with one atomic per
  // row was slower: 75.0 against 73.8 us per call.)
  {
    float lbf[4];
#pragma unroll
    for (int bt = 0; bt < 4; ++bt) {
      const uint32_t lb = s_bound[bt * 16 + r];
      lbf[bt] = (uint32_t)(bt * 16 + r) >= B ? INFINITY : lb ? key2f(lb) : -INFINITY;
    }
#pragma unroll
    for (int k = 0; k < kFuseGroups; ++k)
#pragma unroll
      for (int i = 0; i < kTileGroup; ++i)
        if (held(k, i)) {
          const uint32_t i0 = (tg[k] + i) * 16 + 4 * g;
#pragma unroll
          for (int bt = 0; bt < 4; ++bt) {
            const f32x4 v = acc[k][i][bt];
            if (fmaxf(fmaxf(v[0], v[1]), fmaxf(v[2], v[3])) >= lbf[bt]) {
              const uint32_t c = bt * 16 + r;
#pragma unroll
              for (int q = 0; q < 4; ++q)
                if (v[q] >= lbf[bt] && (whole(k, i) || i0 + q < a.V)) {
                  const uint32_t p = atomicAdd(&s_cnt[c], 1u);
                  st_agent(a.cand + ((size_t)c * nblk + b) * a.ccap + 1 + p, tkey64(v[q], i0 + q));
                }
            }
          }
        }
  }
  // The counts are final once every wave's LDS atomics have returned (an
  // LDS-only barrier: the segment stores complete before the block counts
  // itself in below).
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  if ((uint32_t)tid < B)
    st_agent(a.cand + ((size_t)tid * nblk + b) * a.ccap, (uint64_t)s_cnt[tid]);
  grid_barrier(a, ep, 2, b < B);
  if (b >= B) {
    leave_call(a);
    return;
  }

  // D. Row b.
  const uint32_t row = b;
  if (ld_agent((const unsigned long long*)a.fault) == (unsigned long long)ep + 1ull) {
    for (uint32_t i = tid; i < K; i += kFuseThreads) {
      a.top_ids[(size_t)row * K + i] = -1;
      a.top_prob[(size_t)row * K + i] = 0.f;
    }
    leave_call(a);
    return;
  }
  // Segment t of the row: word 0 its number of keys, words 1.. the keys.
  // Each thread loads the first line (count and up to 15 keys) of its
  // segment.
  const uint64_t* seg = a.cand + (size_t)row * nblk * a.ccap;
  uint64_t line[16];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if ((uint32_t)tid < nblk) v = ld_agent16(seg, (uint32_t)(((size_t)tid * a.ccap + 2 * k) * 8));
    line[2 * k] = ((uint64_t)v[1] << 32) | v[0];
    line[2 * k + 1] = ((uint64_t)v[3] << 32) | v[2];
  }
  const uint32_t cnt = (uint32_t)min(line[0], (uint64_t)(a.ccap - 1));
  const uint32_t inc = wave_incl_scan(cnt);
  if (lane == 63) s_wtot[wave] = inc;
  __syncthreads();
  uint32_t base = 0, n = 0;
  for (int w = 0; w < kLogitWaves; ++w) {
    base += w < wave ? s_wtot[w] : 0u;
    n += s_wtot[w];
  }
  const uint32_t off = base + inc - cnt;
  if ((uint32_t)tid < nblk) s_off[tid] = off;
  if (tid == 0) {
    s_off[nblk] = n;
    s_n = 0;
  }
  __syncthreads();
  // Every key that decides the answer lies in [bound, largest key of the
  // row], so those keys agree above the highest bit in which the two
  // differ (keys below the bound drop out of every histogram).
  const uint32_t lbnd = s_bound[row];
  const uint64_t kmax = ((uint64_t)hmax << 32) | 0xFFFFFFFFull, kmin = (uint64_t)lbnd << 32;
  const uint64_t dk = kmax ^ kmin;
  const int top = dk ? 63 - __builtin_clzll(dk) : 0;
  const int sh0 = max(top - 7, 0);
  const uint64_t dm0 = sh0 + 8 < 64 ? ~((1ull << (sh0 + 8)) - 1ull) : 0ull;
  uint64_t* s_c = (uint64_t*)hs;
  uint32_t nl = n;
  if (n > kLds) {
    // Heavy ties: narrow in memory until at most kLds keys remain at or
    // above the chosen bin, then gather those.
    uint64_t lo = kmax & dm0, dm = dm0;
    uint32_t need = K, above = 0;
    for (int sh = sh0;; sh = max(sh - 8, 0)) {
      if (tid < 256) hist[tid] = 0u;
      __syncthreads();
      for (uint32_t t = wave; t < nblk; t += kLogitWaves) {
        const uint32_t c = s_off[t + 1] - s_off[t];
        const uint64_t* p = seg + (size_t)t * a.ccap + 1;
        for (uint32_t j = lane; j < (c + 63) / 64 * 64; j += 64)
          hist_key(hist, j < c, j < c ? ld_agent(p + j) : 0ull, dm, lo, sh);
      }
      __syncthreads();
      if (wave == 0) pick_bin(hist, need, s_sel);
      __syncthreads();
      const uint32_t bin = s_sel[0], ab = s_sel[1], cb = s_sel[2];
      need -= ab;
      above += ab;
      lo |= (uint64_t)bin << sh;
      dm |= 0xFFull << sh;
      __syncthreads();  // s_sel read by every thread before it is written again
      if (cb == need || above + cb <= kLds || sh == 0) break;
    }
    for (uint32_t t = wave; t < nblk; t += kLogitWaves) {
      const uint32_t c = s_off[t + 1] - s_off[t];
      const uint64_t* p = seg + (size_t)t * a.ccap + 1;
      for (uint32_t j = lane; j < (c + 63) / 64 * 64; j += 64) {
        const uint64_t key = j < c ? ld_agent(p + j) : 0ull;
        const bool in = j < c && key >= lo;
        const uint64_t m = __builtin_amdgcn_ballot_w64(in);
        if (m) {
          uint32_t o = 0;
          if (lane == 0) o = atomicAdd(&s_n, (uint32_t)__builtin_popcountll(m));
          o = __builtin_amdgcn_readfirstlane(o);
          const uint32_t at = o + (uint32_t)__builtin_popcountll(m & ((1ull << lane) - 1ull));
          if (in && at < kLds) s_c[at] = key;
        }
      }
    }
    __syncthreads();
    nl = min(s_n, kLds);
    __syncthreads();
    if (tid == 0) s_n = 0;
  } else if ((uint32_t)tid < nblk) {
#pragma unroll
    for (uint32_t i = 1; i < 16; ++i)
      if (i <= cnt) s_c[off + i - 1] = line[i];
    for (uint32_t i = 16; i <= cnt; ++i) s_c[off + i - 1] = ld_agent(seg + (size_t)tid * a.ccap + i);
  }
  __syncthreads();
  // Exact K-th largest key of the nl >= K candidates in LDS: afterwards the
  // keys >= lo are exactly the K largest.
  uint64_t lo = 0;
  if (nl > K) {
    lo = kmax & dm0;
    uint64_t dm = dm0;
    uint32_t need = K;
    for (int sh = sh0;; sh = max(sh - 8, 0)) {
      if (tid < 256) hist[tid] = 0u;
      __syncthreads();
      for (uint32_t e0 = 0; e0 < nl; e0 += kFuseThreads) {
        const uint32_t e = e0 + tid;
        hist_key(hist, e < nl, e < nl ? s_c[e] : 0ull, dm, lo, sh);
      }
      __syncthreads();
      if (wave == 0) pick_bin(hist, need, s_sel);
      __syncthreads();
      const uint32_t bin = s_sel[0], ab = s_sel[1], cb = s_sel[2];
      need -= ab;
      lo |= (uint64_t)bin << sh;
      dm |= 0xFFull << sh;
      __syncthreads();
      if (cb == need || sh == 0) break;
    }
  }
  const uint64_t below = (1ull << lane) - 1ull;
  for (uint32_t e0 = 0; e0 < nl; e0 += kFuseThreads) {
    const uint32_t e = e0 + tid;
    const uint64_t key = e < nl ? s_c[e] : 0ull;
    const bool in = e < nl && key >= lo;
    const uint64_t m = __builtin_amdgcn_ballot_w64(in);
    if (m) {
      uint32_t o = 0;
      if (lane == 0) o = atomicAdd(&s_n, (uint32_t)__builtin_popcountll(m));
      o = __builtin_amdgcn_readfirstlane(o);
      const uint32_t at = o + (uint32_t)__builtin_popcountll(m & below);
      if (in && at < (uint32_t)kHeadMaxK) s_top[at] = key;
    }
  }
  __syncthreads();
  float S = 0.f;
  for (int w = 0; w < kLogitWaves; ++w) S += s_red[w];
  const float invS = 1.0f / S;
  // The K largest ranked by counting, P consecutive lanes per key.
  const uint32_t lp = K <= 64 ? 3u : K <= 128 ? 2u : 1u;  // log2 P
  const uint32_t ki = (uint32_t)tid >> lp, part = (uint32_t)tid & ((1u << lp) - 1u);
  const uint64_t key = ki < K ? s_top[ki] : ~0ull;
  uint32_t rank = 0;
#pragma unroll 8
  for (uint32_t u = part; u < K; u += 1u << lp) rank += s_top[u] > key ? 1u : 0u;
  for (uint32_t o = 1; o < (1u << lp); o <<= 1) rank += (uint32_t)__shfl_xor((int)rank, (int)o, 8);
  if (ki < K && part == 0) {
    a.top_ids[(size_t)row * K + rank] = (int32_t)(0xFFFFFFFFu - (uint32_t)key);
    a.top_prob[(size_t)row * K + rank] = expf(key2f((uint32_t)(key >> 32)) - M) * invS;
  }
  leave_call(a);
}

}  // namespace

bool head_dim_supported(int D) { return D == 256 || D == 512 || D == 1024; }

uint32_t head_lds_bytes(int D) {
  return (uint32_t)(kCols * (D + 8) * 2 + kLogitWaves * 16 * 72 * 2 + 8 + kCols * 8);
}

hipError_t launch_head_logits(const HeadArgs& a, hipStream_t s) {
  const dim3 grid(a.nblk, (a.B + kCols - 1) / kCols);
  switch (a.D) {
    case 256: hipLaunchKernelGGL(k_head_logits<8>, grid, dim3(kLogitWaves * 64), 0, s, a); break;
    case 512: hipLaunchKernelGGL(k_head_logits<16>, grid, dim3(kLogitWaves * 64), 0, s, a); break;
    case 1024: hipLaunchKernelGGL(k_head_logits<32>, grid, dim3(kLogitWaves * 64), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_head_rows(const HeadArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(k_head_rows, dim3(a.B), dim3(kRowThreads), 0, s, a);
  return hipGetLastError();
}

uint32_t head_fused_ccap(uint32_t V, uint32_t nblk) {
  const uint32_t nt = (V + 15) / 16;
  return ((nt + nblk - 1) / nblk * 16 + 1 + 15) / 16 * 16;
}

bool head_fused_fits(const HeadArgs& a) {
  if (!head_dim_supported((int)a.D) || a.B < 1 || a.B > (uint32_t)kCols || a.B > a.nblk ||
      a.nblk > kFuseMaxBlocks || (a.nblk & (a.nblk - 1)) != 0 || a.K < 1 || a.K > a.nblk ||
      a.K > (uint32_t)kHeadMaxK)
    return false;
  // Tile groups per block within what the waves hold.
  const uint32_t tiles = ((a.V + 15) / 16 + a.nblk - 1) / a.nblk;
  return (tiles + kTileGroup - 1) / kTileGroup <= (uint32_t)(kFuseGroups * kLogitWaves);
}

bool head_fused_resident(int D) {
  const void* f = D == 256 ? (const void*)k_head_fused<8>
                : D == 512 ? (const void*)k_head_fused<16>
                           : (const void*)k_head_fused<32>;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, kFuseThreads, 0) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return n >= 1;
}

hipError_t launch_head_fused(const HeadArgs& a, hipStream_t s) {
  const dim3 grid(a.nblk), block(kFuseThreads);
  switch (a.D) {
    case 256: hipLaunchKernelGGL(k_head_fused<8>, grid, block, 0, s, a); break;
    case 512: hipLaunchKernelGGL(k_head_fused<16>, grid, block, 0, s, a); break;
    case 1024: hipLaunchKernelGGL(k_head_fused<32>, grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace tfe
