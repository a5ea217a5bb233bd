// Early-exit prefetch head on gfx950 (wave64, MFMA): the approximate
// next-token distribution p = softmax(W h) of an intermediate hidden state
// (Eq. 13) and its K most likely tokens (Eq. 14), which are the candidates
// the cache prefetch consumes.
//
// Two launches:
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

// One wave's logits for TPW consecutive 16-token tiles from t (a tile at or
// past t_hi is not stored, and its loads re-read tile t's rows; the
// kernel's claims never produce one).  The tiles share each B-operand read of the
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
__device__ __forceinline__ void logits_tiles(const HeadArgs& a, uint32_t t, uint32_t t_hi,
                                             const __bf16* hs, __bf16* st, int hoff, int lane,
                                             int r, int g, uint64_t* bm) {
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
  f32x4 acc[TPW][4];
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

}  // namespace tfe
