// Offline phrase-table construction on the GPU: the most frequent distinct
// n-grams of a token stream (Sec. 4.2: candidate phrases selected by corpus
// frequency; n-gram extraction dominates the construction time reported in
// the evaluation).
//
// Steps, all on the device:
//   1. key formation: every window of n tokens becomes one 64-bit key, the
//      tokens in 18-bit fields, oldest in the highest field, so that key
//      order is tuple order; a window with a token outside [0, vocab) gets
//      a mark above every valid key: vocab in the oldest field when vocab <
//      2^18 (the keys keep 18 n bits), else 2^(18 n) (formed by the first
//      pass of the sort, from the tokens);
//   2. LSD radix sort of the keys, 9-bit digits (an 18-bit token field is
//      two digits) over the key bits (the valid keys end up first; a binary
//      search counts them): per pass a digit histogram per tile (4096 keys;
//      3072 with a payload), one exclusive scan of the digit-major
//      histogram, and a stable scatter
//      (each wave ranks its keys with ballot-based digit matching, the tile
//      is reordered in LDS and written out in digit runs);
//   3. run-length count: per-block counts of run starts, their scan, the
//      starts written at their ranks into a unique-key array; a run's count
//      is the distance to the next start;
//   4. selection of ranks [0, skip + top): the (skip+top)-th largest count
//      c* from a histogram of the small counts (a radix select over the
//      counts when c* is large), then an order-preserving compaction of the
//      runs with count > c* and the first needed ones with count == c* (key
//      order = tuple order, which breaks the ties);
//   5. ranking: a stable radix sort of the selected runs by descending count
//      (payload: the run index), which keeps tuple order among equal counts;
//   6. ranks [skip, skip + top) are unpacked into tuples and counts.
// 4-grams need 72 key bits: the three newest tokens form the low word and
// the oldest token the high word; the LSD sort runs over the low word (high
// word as a 32-bit payload) and then stably over the high word.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "../../include/tfe.h"
#include "tfe_internal.h"

namespace tfe {
namespace {

// Radix tiles: the scatter runs 512 threads per tile (one per digit), 8
// keys per thread for keys alone (4096 keys: 52 KB of LDS with the 512-bin
// counts, so three tiles share a CU and one tile's ranking overlaps the
// others' memory traffic) and 6 with a 64-bit payload (68 KB, two tiles per
// CU).  Measured on MI355X with 8-bit digits for keys alone: 5120-key tiles
// beat 4096 (2.71 against 2.73 ms for the 2^26-token 2-gram table) and 8192
// (2.83 ms), whose 74 KB allow two tiles per CU; with 9-bit digits the 36-bit
// 2-gram keys take four passes instead of five (2.50 ms).  The histogram of
// a tile is counted by 1024 threads.
constexpr int kTileThreads = 512;
constexpr int kTileWaves = kTileThreads / 64;
constexpr int kHistThreads = 1024;
template <class K, bool PAIRS, class V>
constexpr int tile_items() { return (sizeof(K) + (PAIRS ? sizeof(V) : 0)) > 8 ? 6 : 8; }
template <class K, bool PAIRS, class V>
constexpr int tile_keys() { return kTileThreads * tile_items<K, PAIRS, V>(); }
constexpr int kMinTile = kTileThreads * 6;  // smallest tile: sizes the histogram matrix
// Radix digits: 9 bits (512 bins), so that 18-bit token fields take two
// digits each.
constexpr int kDigitBits = 9;
constexpr uint32_t kBins = 1u << kDigitBits;
static_assert(kBins <= (uint32_t)kTileThreads, "one scatter thread per digit");
constexpr int kScanThreads = 1024;
constexpr int kScanItems = 16;
constexpr int kScanBlock = kScanThreads * kScanItems;

// ---- 1. keys -----------------------------------------------------------------

// One key per window, in window order (no compaction: the sort moves the
// invalid windows, marked with a key just above every valid one, to the end).
// The keys are formed from the tokens by the first radix pass itself.
struct TokSrc {
  const int32_t* tok;
  int n;
  int32_t vocab;
  uint64_t mark;   // key of an invalid window: just above every valid key
  uint32_t mark4;  // 4-grams: high word of an invalid window
};

// Key sources: the key array, windows of 1, 2 or 3 tokens (the source is
// the window length, known at compile time so that the token loads of all
// of a thread's windows are in flight together), or 4-gram words.
enum { kSrcKeys = 0, kSrcNgram4 = 4 };

// Tokens a tile of windows [w0, w0 + TILE) needs: [w0, w0 + TILE + 3),
// clipped to the stream (n windows of `ts.n` tokens: n + ts.n - 1 tokens),
// staged in LDS with coalesced loads (16 bytes per lane when the stream is
// 16-byte aligned) so that each window's tokens are read from LDS instead of
// with one global load per token and window.  Past the stream: -1.
template <int TILE, int NT>
__device__ __forceinline__ void stage_tokens(const TokSrc& ts, uint64_t n, uint64_t w0,
                                             int32_t* s_tok) {
  constexpr int CNT = TILE + 3;
  const uint64_t ntok = n + (uint64_t)ts.n - 1;
  const uint64_t avail = ntok > w0 ? ntok - w0 : 0;
  const int32_t* src = ts.tok + w0;
  if ((((uintptr_t)src) & 15u) == 0) {
    typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
    for (int v = threadIdx.x; v < (CNT + 3) / 4; v += NT) {
      const uint64_t e = 4ull * (uint64_t)v;
      if (e + 4 <= avail) {
        const i32x4 x = *(const i32x4*)(src + e);
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (e + q < (uint64_t)CNT) s_tok[e + q] = x[q];
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (e + q < (uint64_t)CNT) s_tok[e + q] = e + q < avail ? src[e + q] : -1;
      }
    }
  } else {
    for (int e = threadIdx.x; e < CNT; e += NT) s_tok[e] = (uint64_t)e < avail ? src[e] : -1;
  }
}

// Key of the window starting at staged token j (NG <= 3 tokens, oldest in
// the highest field); an invalid window gets ts.mark.  4-grams: 72 key bits
// in two words, lo = the three newest tokens (54 bits) and, as the payload,
// hi = the oldest token, or ts.mark4 for an invalid window.
template <int NG>
__device__ __forceinline__ uint64_t ngram_key_lds(const int32_t* s, uint32_t j,
                                                  const TokSrc& ts) {
  uint64_t key = 0;
  bool ok = true;
#pragma unroll
  for (int q = 0; q < NG; ++q) {
    const int32_t t = s[j + q];
    ok = ok && t >= 0 && t < ts.vocab;
    key = (key << 18) | (uint64_t)(uint32_t)(t & 0x3FFFF);
  }
  return ok ? key : ts.mark;
}

template <int SRC, class K>
__device__ __forceinline__ K key_at_lds(const int32_t* s, uint32_t j, const TokSrc& ts) {
  if (SRC == kSrcNgram4) {
    uint64_t key = 0;
#pragma unroll
    for (int q = 1; q < 4; ++q) key = (key << 18) | (uint64_t)(uint32_t)(s[j + q] & 0x3FFFF);
    return (K)key;
  }
  return (K)ngram_key_lds<(SRC >= 1 && SRC <= 3) ? SRC : 1>(s, j, ts);
}

__device__ __forceinline__ uint64_t val4_at_lds(const int32_t* s, uint32_t j, const TokSrc& ts) {
  bool ok = true;
#pragma unroll
  for (int q = 0; q < 4; ++q) ok = ok && s[j + q] >= 0 && s[j + q] < ts.vocab;
  return ok ? (uint64_t)(uint32_t)s[j] : (uint64_t)ts.mark4;
}

// Number of sorted keys below the invalid-window mark (one thread: binary
// search).
__global__ void k_count_valid(const uint64_t* keys, uint64_t nwin, uint64_t mark,
                              unsigned long long* count) {
  uint64_t lo = 0, hi = nwin;
  while (lo < hi) {
    const uint64_t mid = lo + (hi - lo) / 2;
    if (keys[mid] < mark) lo = mid + 1;
    else hi = mid;
  }
  *count = lo;
}

__global__ void k_count_valid_hi(const uint32_t* hi, uint64_t nwin, uint32_t mark,
                                 unsigned long long* count) {
  uint64_t lo = 0, top = nwin;
  while (lo < top) {
    const uint64_t mid = lo + (top - lo) / 2;
    if (hi[mid] < mark) lo = mid + 1;
    else top = mid;
  }
  *count = lo;
}

// ---- device-wide exclusive scan of uint32 (totals below 2^32) ----------------

template <int NT>
__device__ uint32_t block_scan_excl(uint32_t v, uint32_t* s_wave, uint32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  if (lane == 63) s_wave[wave] = x;
  __syncthreads();
  uint32_t off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    off += w < wave ? s_wave[w] : 0u;
    tot += s_wave[w];
  }
  __syncthreads();
  *total = tot;
  return x - v + off;
}

// Pass 1: per-block sums.
__global__ __launch_bounds__(kScanThreads) void k_scan_reduce(const uint32_t* in, uint64_t n,
                                                              uint32_t* part) {
  __shared__ uint32_t s_wave[kScanThreads / 64];
  const uint64_t base = (uint64_t)blockIdx.x * kScanBlock;
  // All loads first (masked past n), then the sum: one round trip.
  uint32_t v[kScanItems];
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const uint64_t i = base + (uint64_t)k * kScanThreads + threadIdx.x;
    v[k] = i < n ? in[i] : 0u;
  }
  uint32_t s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) s += v[k];
  uint32_t tot;
  (void)block_scan_excl<kScanThreads>(s, s_wave, &tot);
  if (threadIdx.x == 0) part[blockIdx.x] = tot;
}

// Exclusive scan of the block sums in one block (nb <= kScanBlock), and
// their total: the run count places its starts with it.
__global__ __launch_bounds__(kScanThreads) void k_scan_partials(uint32_t* part, uint32_t nb,
                                                                uint32_t* total) {
  __shared__ uint32_t s_wave[kScanThreads / 64];
  uint32_t v[kScanItems];
  uint32_t s = 0;
  for (int k = 0; k < kScanItems; ++k) {
    const uint32_t i = threadIdx.x * kScanItems + k;
    v[k] = i < nb ? part[i] : 0u;
    s += v[k];
  }
  uint32_t tot;
  uint32_t run = block_scan_excl<kScanThreads>(s, s_wave, &tot);
  for (int k = 0; k < kScanItems; ++k) {
    const uint32_t i = threadIdx.x * kScanItems + k;
    if (i < nb) part[i] = run;
    run += v[k];
  }
  if (threadIdx.x == 0 && total) *total = tot;
}

// Inclusive sum over the lanes up to this one: DPP shifts within each
// 16-lane row, then the totals of the rows below (read out as scalars).
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t x) {
  const int lane = threadIdx.x & 63;
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xF, 0xF, false);  // row_shr:1
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xF, 0xF, false);  // row_shr:2
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xF, 0xF, false);  // row_shr:4
  x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xF, 0xF, false);  // row_shr:8
  const uint32_t r0 = (uint32_t)__builtin_amdgcn_readlane((int)x, 15);
  const uint32_t r1 = (uint32_t)__builtin_amdgcn_readlane((int)x, 31);
  const uint32_t r2 = (uint32_t)__builtin_amdgcn_readlane((int)x, 47);
  const int row = lane >> 4;
  return x + (row >= 1 ? r0 : 0u) + (row >= 2 ? r1 : 0u) + (row >= 3 ? r2 : 0u);
}

// Pass 3: scan within blocks plus the block offset.  Wave w of a block scans
// its contiguous kScanItems x 64 elements in rounds of 64 (coalesced), with
// a running carry; one exchange of wave totals places the waves.  part
// holds the blocks' sums as pass 1 left them: each block adds up those of
// the blocks before it itself (at most kScanItems per thread, from L2),
// which saves a one-block scan launch.
__global__ __launch_bounds__(kScanThreads) void k_scan_down(const uint32_t* in, uint64_t n,
                                                            const uint32_t* part, uint32_t* out) {
  __shared__ uint32_t s_tot[kScanThreads / 64];
  __shared__ uint32_t s_red[kScanThreads / 64];
  uint32_t off = 0;
  {
    uint32_t b = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
      const uint32_t j = (uint32_t)k * kScanThreads + threadIdx.x;
      b += j < blockIdx.x ? part[j] : 0u;
    }
    (void)block_scan_excl<kScanThreads>(b, s_red, &off);
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t base = (uint64_t)blockIdx.x * kScanBlock + (uint64_t)wave * (64 * kScanItems);
  uint32_t v[kScanItems];
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const uint64_t i = base + (uint64_t)k * 64 + lane;
    v[k] = i < n ? in[i] : 0u;
  }
  uint32_t carry = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const uint32_t inc = wave_incl_scan(v[k]);
    const uint32_t ex = carry + inc - v[k];
    carry += (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
    v[k] = ex;
  }
  if (lane == 0) s_tot[wave] = carry;
  __syncthreads();
  for (int w = 0; w < wave; ++w) off += s_tot[w];
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const uint64_t i = base + (uint64_t)k * 64 + lane;
    if (i < n) out[i] = off + v[k];
  }
}

// ---- 2. stable LSD radix sort (9-bit digits) --------------------------------

template <class K>
__device__ __forceinline__ uint32_t digit_of(K k, int shift) {
  return (uint32_t)(k >> shift) & (kBins - 1u);
}

// Radix tile of this block.  Workgroups are dispatched round-robin over the
// 8 XCDs (each with its own L2); giving every XCD a contiguous range of
// tiles keeps the 32 tiles that share a 128-byte line of the digit-major
// histogram matrix on one XCD, so each line is written and read through
// one L2 instead of eight.  A bijection of [0, G) for any G.
__device__ __forceinline__ uint32_t xcd_tile(uint32_t b, uint32_t G) {
  const uint32_t q = G >> 3, r = G & 7u, x = b & 7u;
  return x * q + min(x, r) + (b >> 3);
}

// Lanes of the wave whose digit equals this lane's (active lanes only).
__device__ __forceinline__ uint64_t match_digit(uint32_t d, bool active) {
  uint64_t m = __builtin_amdgcn_ballot_w64(active);
#pragma unroll
  for (int b = 0; b < kDigitBits; ++b) {
    const uint64_t bb = __builtin_amdgcn_ballot_w64(active && ((d >> b) & 1u));
    m &= ((d >> b) & 1u) ? bb : ~bb;
  }
  return m;
}

// Digit histogram of one tile of TILE keys (kHistThreads threads; the keys
// are loaded first).  Per round, the lanes holding the first lane's digit
// add their number with one atomic and the others add 1 each: Zipf-skewed
// digits (high bits of frequent tokens are mostly 0) would otherwise pile
// same-address LDS atomics onto one bin; measured on MI355X this beats both
// plain atomics and counting every group of equal digits once.
template <class K, int TILE, int SRC>
__global__ __launch_bounds__(kHistThreads) void k_rs_hist(const K* keys, TokSrc ts, uint64_t n,
                                                          int shift, uint32_t* hist,
                                                          uint32_t ntiles) {
  constexpr int ITEMS = TILE / kHistThreads;
  constexpr bool kTok = SRC != kSrcKeys;
  __shared__ uint32_t h[kBins];
  __shared__ int32_t s_tok[kTok ? TILE + 3 : 1];
  for (int e = threadIdx.x; e < (int)kBins; e += kHistThreads) h[e] = 0u;
  const uint32_t tile = xcd_tile(blockIdx.x, gridDim.x);
  const uint64_t base = (uint64_t)tile * TILE;
  if (kTok) {
    stage_tokens<TILE, kHistThreads>(ts, n, base, s_tok);
    __syncthreads();
  }
  K kk[ITEMS];
#pragma unroll
  for (int k = 0; k < ITEMS; ++k) {
    const uint64_t i = base + (uint64_t)k * kHistThreads + threadIdx.x;
    if (kTok)
      kk[k] = i < n ? key_at_lds<SRC, K>(s_tok, (uint32_t)(i - base), ts) : (K)0;
    else
      kk[k] = i < n ? keys[i] : (K)0;
  }
  __syncthreads();
  const uint64_t lt = (1ull << (threadIdx.x & 63)) - 1ull;
#pragma unroll
  for (int k = 0; k < ITEMS; ++k) {
    const bool act = base + (uint64_t)k * kHistThreads + threadIdx.x < n;
    const uint32_t d = digit_of(kk[k], shift);
    const uint32_t d0 = __builtin_amdgcn_readfirstlane(d);
    const uint64_t m = __builtin_amdgcn_ballot_w64(act && d == d0);
    if (act && d == d0) {
      if ((m & lt) == 0) atomicAdd(&h[d0], (uint32_t)__builtin_popcountll(m));
    } else if (act) {
      atomicAdd(&h[d], 1u);
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < (int)kBins; e += kHistThreads)
    hist[(size_t)e * ntiles + tile] = h[e];
}

// Scatter of one tile.  Wave w ranks the keys [w 64 ITEMS, (w+1) 64 ITEMS)
// of the tile in ITEMS rounds of 64 consecutive keys: the rank of a key
// among the wave's earlier keys of its digit is the wave's running count
// plus the matching lanes below it; the first lane of each digit group
// advances the count.  Tile positions follow (digit, wave, rank), i.e. the
// stable order; the tile is reordered in LDS and written in digit runs.
template <class K, class V, bool PAIRS, int ITEMS, int SRC>
__global__ __launch_bounds__(kTileThreads) void k_rs_scatter(const K* keys, const V* vals,
                                                             TokSrc ts, uint64_t n, int shift,
                                                             const uint32_t* offs,
                                                             uint32_t ntiles, K* keys_out,
                                                             V* vals_out) {
  constexpr int TILE = kTileThreads * ITEMS;
  __shared__ uint32_t wcnt[kTileWaves][kBins];
  __shared__ uint32_t s_loc[kBins];   // tile-local start of each digit
  __shared__ uint32_t s_glob[kBins];  // global start of each digit's run of this tile
  __shared__ uint32_t s_wave[kTileWaves];
  __shared__ K s_keys[TILE];
  __shared__ V s_vals[PAIRS ? TILE : 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int e = threadIdx.x; e < kTileWaves * (int)kBins; e += kTileThreads) (&wcnt[0][0])[e] = 0u;
  const uint32_t tile = xcd_tile(blockIdx.x, gridDim.x);
  const uint64_t base = (uint64_t)tile * TILE + (uint64_t)wave * (64 * ITEMS);
  const uint64_t lt = (1ull << lane) - 1ull;
  // Token-sourced keys: the tile's tokens are staged in the reorder buffer,
  // which is free until the keys are placed (two barriers later).
  constexpr bool kTok = SRC != kSrcKeys;
  static_assert(!kTok || (TILE + 3) * 4 <= TILE * (int)sizeof(K), "token staging fits");
  int32_t* s_tok = (int32_t*)s_keys;
  if (kTok) {
    stage_tokens<TILE, kTileThreads>(ts, n, (uint64_t)tile * TILE, s_tok);
    __syncthreads();
  }
  K kk[ITEMS];
  V vv[PAIRS ? ITEMS : 1];
  uint32_t rank[ITEMS];
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    const uint64_t i = base + (uint64_t)r * 64 + lane;
    const uint32_t j = (uint32_t)(i - (uint64_t)tile * TILE);
    if (kTok) {
      kk[r] = i < n ? key_at_lds<SRC, K>(s_tok, j, ts) : (K)0;
      if (PAIRS) vv[PAIRS ? r : 0] = i < n ? (V)val4_at_lds(s_tok, j, ts) : (V)0;
    } else {
      kk[r] = i < n ? keys[i] : (K)0;
      if (PAIRS) vv[PAIRS ? r : 0] = i < n ? vals[i] : (V)0;
    }
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    const bool act = base + (uint64_t)r * 64 + lane < n;
    const uint32_t d = digit_of(kk[r], shift);
    const uint64_t m = match_digit(d, act);
    const uint32_t before = wcnt[wave][d];
    rank[r] = before + (uint32_t)__builtin_popcountll(m & lt);
    // The lowest matching lane advances the wave's count of this digit.
    if (act && (m & lt) == 0) wcnt[wave][d] = before + (uint32_t)__builtin_popcountll(m);
  }
  __syncthreads();
  // Per digit (one thread each): counts of earlier waves, the tile's digit
  // starts.
  const uint32_t d = threadIdx.x;
  uint32_t tot = 0;
  if (d < kBins) {
    for (int w = 0; w < kTileWaves; ++w) {
      const uint32_t c = wcnt[w][d];
      wcnt[w][d] = tot;  // becomes the offset of wave w within the digit
      tot += c;
    }
  }
  uint32_t all;
  const uint32_t loc = block_scan_excl<kTileThreads>(tot, s_wave, &all);
  if (d < kBins) {
    s_loc[d] = loc;
    s_glob[d] = offs[(size_t)d * ntiles + tile];
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < ITEMS; ++r) {
    const uint64_t i = base + (uint64_t)r * 64 + lane;
    if (i < n) {
      const uint32_t dd = digit_of(kk[r], shift);
      const uint32_t pos = s_loc[dd] + wcnt[wave][dd] + rank[r];
      s_keys[pos] = kk[r];
      if (PAIRS) s_vals[PAIRS ? pos : 0] = vv[PAIRS ? r : 0];
    }
  }
  __syncthreads();
  const uint64_t tile0 = (uint64_t)tile * TILE;
  const uint32_t cnt = (uint32_t)min((uint64_t)TILE, n - tile0);
  for (uint32_t p = threadIdx.x; p < cnt; p += kTileThreads) {
    const K k = s_keys[p];
    const uint32_t dd = digit_of(k, shift);
    const uint64_t dst = (uint64_t)s_glob[dd] + (p - s_loc[dd]);
    keys_out[dst] = k;
    if (PAIRS) vals_out[dst] = s_vals[PAIRS ? p : 0];
  }
}

// ---- 3. run-length count ----------------------------------------------------

// Runs of equal keys in the sorted valid keys (hi: the high key word of
// 4-grams, or null), in two passes shaped like the scan: the number of run
// starts per block, then (after the scan of those counts) each start's key
// and position at its rank.  A start is a key that differs from the one
// before it.  Wave w of a block covers kScanItems rounds of 64 keys.

// Run starts among the kScanItems rounds of 64 keys of this wave from base:
// the keys (and high words) are loaded first, at clamped indices, so that
// all loads are in flight at once; each key's predecessor comes from the
// lane below (lane 0: lane 63 of the round before, or one load for the
// wave's first key); then one ballot per round.  cur keeps the keys (and
// hcur the high words).
__device__ __forceinline__ uint64_t from_lane_below(uint64_t x, uint64_t carry) {
  const int lane = threadIdx.x & 63;
  const uint32_t lo = (uint32_t)__shfl_up((int)(uint32_t)x, 1, 64);
  const uint32_t hi = (uint32_t)__shfl_up((int)(uint32_t)(x >> 32), 1, 64);
  return lane == 0 ? carry : ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t lane63(uint64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, 63);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), 63);
  return ((uint64_t)hi << 32) | lo;
}

template <bool WIDE>
__device__ __forceinline__ void run_starts(const uint64_t* keys, const uint32_t* hi, uint64_t base,
                                           uint64_t n, uint64_t (&m)[kScanItems],
                                           uint64_t (&cur)[kScanItems],
                                           uint32_t (&hcur)[WIDE ? kScanItems : 1]) {
  const int lane = threadIdx.x & 63;
  const uint64_t i0 = base > 0 ? (base - 1 < n ? base - 1 : n - 1) : 0;
  const uint64_t first = keys[i0];
  const uint32_t hfirst = WIDE ? hi[i0] : 0u;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const uint64_t i = base + (uint64_t)k * 64 + lane;
    const uint64_t ic = i < n ? i : n - 1;
    cur[k] = keys[ic];
    if (WIDE) hcur[WIDE ? k : 0] = hi[ic];
  }
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const uint64_t i = base + (uint64_t)k * 64 + lane;
    const uint64_t prv = from_lane_below(cur[k], k == 0 ? first : lane63(cur[k > 0 ? k - 1 : 0]));
    bool differs = cur[k] != prv;
    if (WIDE) {
      const uint32_t hc = hcur[WIDE ? k : 0];
      const uint32_t hcarry =
          k == 0 ? hfirst
                 : (uint32_t)__builtin_amdgcn_readlane((int)hcur[WIDE ? (k > 0 ? k - 1 : 0) : 0], 63);
      // Shuffled in every lane before the select: a lane that reads an
      // inactive one gets 0.
      const uint32_t below = (uint32_t)__shfl_up((int)hc, 1, 64);
      const uint32_t hp = lane == 0 ? hcarry : below;
      differs = differs || hc != hp;
    }
    m[k] = __builtin_amdgcn_ballot_w64(i < n && (i == 0 || differs));
  }
}

template <bool WIDE>
__global__ __launch_bounds__(kScanThreads) void k_runs_reduce(const uint64_t* keys,
                                                              const uint32_t* hi, uint64_t n,
                                                              uint32_t* part) {
  __shared__ uint32_t s_tot[kScanThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t base = (uint64_t)blockIdx.x * kScanBlock + (uint64_t)wave * (64 * kScanItems);
  uint64_t m[kScanItems], cur[kScanItems];
  uint32_t hcur[WIDE ? kScanItems : 1];
  run_starts<WIDE>(keys, hi, base, n, m, cur, hcur);
  uint32_t c = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) c += (uint32_t)__builtin_popcountll(m[k]);
  if (lane == 0) s_tot[wave] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = 0;
    for (int w = 0; w < kScanThreads / 64; ++w) t += s_tot[w];
    part[blockIdx.x] = t;
  }
}

template <bool WIDE>
__global__ __launch_bounds__(kScanThreads) void k_runs_write(const uint64_t* keys,
                                                             const uint32_t* hi, uint64_t n,
                                                             const uint32_t* part, uint64_t* ukey,
                                                             uint32_t* uhi, uint32_t* ustart) {
  __shared__ uint32_t s_tot[kScanThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint64_t base = (uint64_t)blockIdx.x * kScanBlock + (uint64_t)wave * (64 * kScanItems);
  uint64_t m[kScanItems], cur[kScanItems];
  uint32_t hcur[WIDE ? kScanItems : 1];
  run_starts<WIDE>(keys, hi, base, n, m, cur, hcur);
  uint32_t c = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) c += (uint32_t)__builtin_popcountll(m[k]);
  if (lane == 0) s_tot[wave] = c;
  __syncthreads();
  uint32_t r = part[blockIdx.x];
  for (int w = 0; w < wave; ++w) r += s_tot[w];
  const uint64_t lt = (1ull << lane) - 1ull;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const uint64_t i = base + (uint64_t)k * 64 + lane;
    if ((m[k] >> lane) & 1ull) {
      const uint32_t idx = r + (uint32_t)__builtin_popcountll(m[k] & lt);
      ukey[idx] = cur[k];
      if (WIDE) uhi[idx] = hcur[WIDE ? k : 0];
      ustart[idx] = (uint32_t)i;
    }
    r += (uint32_t)__builtin_popcountll(m[k]);
  }
}

// Run lengths, and the histogram of min(count, kSelBins - 1) for the
// selection (per-block LDS bins added to the global ones).
constexpr int kSelBins = 4096;

__global__ __launch_bounds__(1024) void k_run_counts(const uint32_t* ustart, uint32_t u,
                                                     uint32_t n, uint32_t* ucount,
                                                     uint32_t* bins) {
  __shared__ uint32_t h[kSelBins];
  for (int e = threadIdx.x; e < kSelBins; e += 1024) h[e] = 0u;
  __syncthreads();
  const uint32_t base = blockIdx.x * (1024u * 16u);
  for (int k = 0; k < 16; ++k) {
    const uint32_t i = base + (uint32_t)k * 1024u + threadIdx.x;
    const bool in = i < u;
    uint32_t bin = 0;
    if (in) {
      const uint32_t c = (i + 1 < u ? ustart[i + 1] : n) - ustart[i];
      ucount[i] = c;
      bin = c < (uint32_t)kSelBins ? c : (uint32_t)kSelBins - 1u;
    }
    // Most runs are short, so most lanes share a bin: the lanes holding the
    // first lane's bin add their number with one atomic (one atomic per
    // lane put 64-way same-address atomics on the few small-count bins).
    if (__builtin_amdgcn_ballot_w64(in)) {
      const uint32_t b0 = __builtin_amdgcn_readfirstlane(bin);
      const uint64_t m = __builtin_amdgcn_ballot_w64(in && bin == b0);
      if (in && bin != b0)
        atomicAdd(&h[bin], 1u);
      else if (in && (m & ((1ull << (threadIdx.x & 63)) - 1ull)) == 0)
        atomicAdd(&h[b0], (uint32_t)__builtin_popcountll(m));
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < kSelBins; e += 1024)
    if (h[e]) atomicAdd(&bins[e], h[e]);
}

// ---- 4. selection -----------------------------------------------------------

// The selection state: {prefix, mask, need, above, done}.  After the
// selection, prefix = c* (the R-th largest count), need = how many runs of
// count c* belong to ranks [0, R), above = the runs with larger counts.

// From the histogram of min(count, kSelBins - 1) (one block, 1024 threads,
// 4 bins each from the top): if c* < kSelBins - 1 the selection is done;
// otherwise the radix passes below find it.
__global__ __launch_bounds__(1024) void k_sel_small(const uint32_t* bins, uint32_t* state) {
  __shared__ uint32_t s_wave[16];
  const uint32_t t = threadIdx.x;
  const uint32_t need = state[2];
  uint32_t v[4], sum = 0;
  for (int k = 0; k < 4; ++k) {
    v[k] = bins[kSelBins - 1 - (4 * t + k)];  // bins in descending count order
    sum += v[k];
  }
  uint32_t tot;
  uint32_t ex = block_scan_excl<1024>(sum, s_wave, &tot);
  for (int k = 0; k < 4; ++k) {
    const uint32_t c = kSelBins - 1 - (4 * t + k);
    if (ex < need && need <= ex + v[k] && c < (uint32_t)kSelBins - 1) {
      state[0] = c;
      state[1] = 0xFFFFFFFFu;
      state[2] = need - ex;
      state[3] = ex;
      state[4] = 1u;
    }
    ex += v[k];
  }
}

// Histogram of digit `shift` of the counts whose higher digits equal
// `prefix` (under `mask`): one pass of a radix select on a 32-bit value.
__global__ __launch_bounds__(256) void k_sel_hist(const uint32_t* cnt, uint32_t u,
                                                  const uint32_t* state, int shift,
                                                  uint32_t* hist) {
  __shared__ uint32_t h[256];
  if (state[4]) return;  // done from the small-count histogram
  h[threadIdx.x] = 0u;
  __syncthreads();
  const uint32_t prefix = state[0], mask = state[1];
  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < u; i += gridDim.x * 256) {
    const uint32_t c = cnt[i];
    if ((c & mask) == prefix) atomicAdd(&h[(c >> shift) & 255u], 1u);
  }
  __syncthreads();
  if (h[threadIdx.x]) atomicAdd(&hist[threadIdx.x], h[threadIdx.x]);
}

// One block: pick the digit bin holding the need-th largest, update the
// state {prefix, mask, need, above} and clear the histogram.
__global__ __launch_bounds__(256) void k_sel_pick(uint32_t* hist, uint32_t* state, int shift) {
  __shared__ uint32_t s_wave[4];
  const uint32_t t = threadIdx.x;
  // Every thread reads the state before the scan's barriers, so the one
  // update below cannot be seen by a late reader.
  if (state[4]) return;
  const uint32_t need = state[2];
  const uint32_t v = hist[255 - t];  // thread t looks at bin 255 - t
  uint32_t tot;
  const uint32_t ex = block_scan_excl<256>(v, s_wave, &tot);
  if (ex < need && need <= ex + v) {
    state[0] |= (255u - t) << shift;
    state[1] |= 255u << shift;
    state[2] = need - ex;
    state[3] += ex;
  }
  hist[255 - t] = 0u;
}

// keep[i]: count > c*, or count == c* and among the first `need` such runs.
// The runs that make ranks [0, R): with c* = state[0] and need = state[2],
// run i is kept when its count exceeds c*, or equals c* and fewer than
// `need` runs of count c* come before it.  Kept runs keep their order
// (rkey = ~count, rval = the run index): the stable sort that ranks them
// then leaves equal counts in tuple order.  Two launches over the counts:
// per-block numbers above and at c*, then each block places its kept runs.

// Per block of kScanBlock runs: how many counts exceed c* and how many
// equal it.
__global__ __launch_bounds__(kScanThreads) void k_sel_count(const uint32_t* cnt, uint32_t u,
                                                            const uint32_t* state,
                                                            uint32_t* part_gt, uint32_t* part_eq) {
  __shared__ uint32_t s_gt[kScanThreads / 64], s_eq[kScanThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t cstar = state[0];  // >= 1: the R-th largest count
  const uint64_t base = (uint64_t)blockIdx.x * kScanBlock + (uint64_t)wave * (64 * kScanItems);
  uint32_t c[kScanItems];
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const uint64_t i = base + (uint64_t)k * 64 + lane;
    c[k] = i < u ? cnt[i] : 0u;  // 0: no run
  }
  uint32_t g = 0, e = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    g += (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(c[k] > cstar));
    e += (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(c[k] == cstar));
  }
  if (lane == 0) {
    s_gt[wave] = g;
    s_eq[wave] = e;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t tg = 0, te = 0;
    for (int w = 0; w < kScanThreads / 64; ++w) {
      tg += s_gt[w];
      te += s_eq[w];
    }
    part_gt[blockIdx.x] = tg;
    part_eq[blockIdx.x] = te;
  }
}

// Places the block's kept runs.  The runs above c* before the block, and
// the kept ones at c* (the first `need` of them, in order), are added up
// from the per-block numbers of the earlier blocks (at most kScanItems per
// thread, from L2); within the block each wave takes its contiguous
// kScanItems x 64 runs, ranks the ones at c* and then the kept ones with
// ballots, and one exchange of wave totals places the waves.  Positions at
// or past R (none when the selection state is consistent) are not written.
__global__ __launch_bounds__(kScanThreads) void k_sel_place(const uint32_t* cnt, uint32_t u,
                                                            const uint32_t* state,
                                                            const uint32_t* part_gt,
                                                            const uint32_t* part_eq, uint32_t R,
                                                            uint32_t* rkey, uint64_t* rval) {
  __shared__ uint64_t s_sum[kScanThreads / 64];
  __shared__ uint32_t s_eq[kScanThreads / 64], s_keep[kScanThreads / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const uint32_t cstar = state[0], need = state[2];
  const uint64_t base = (uint64_t)blockIdx.x * kScanBlock + (uint64_t)wave * (64 * kScanItems);
  uint32_t c[kScanItems];
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const uint64_t i = base + (uint64_t)k * 64 + lane;
    c[k] = i < u ? cnt[i] : 0u;
  }
  // Earlier blocks: above c* in the high word, at c* in the low word (each
  // total is below 2^32).
  uint64_t b = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const uint32_t j = (uint32_t)k * kScanThreads + threadIdx.x;
    if (j < blockIdx.x) b += ((uint64_t)part_gt[j] << 32) | part_eq[j];
  }
  for (int d = 32; d >= 1; d >>= 1) b += __shfl_xor(b, d, 64);
  if (lane == 0) s_sum[wave] = b;
  const uint64_t lt = (1ull << lane) - 1ull;
  uint64_t em[kScanItems];
  uint32_t e = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    em[k] = __builtin_amdgcn_ballot_w64(c[k] == cstar);
    e += (uint32_t)__builtin_popcountll(em[k]);
  }
  if (lane == 0) s_eq[wave] = e;
  __syncthreads();
  uint64_t before = 0;
  for (int w = 0; w < kScanThreads / 64; ++w) before += s_sum[w];
  const uint32_t gt_before = (uint32_t)(before >> 32), eq_before = (uint32_t)before;
  uint32_t erun = eq_before;
  for (int w = 0; w < wave; ++w) erun += s_eq[w];
  uint64_t km[kScanItems];
  uint32_t kc = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    const uint32_t er = erun + (uint32_t)__builtin_popcountll(em[k] & lt);
    const bool keep = c[k] > cstar || (((em[k] >> lane) & 1ull) && er < need);
    km[k] = __builtin_amdgcn_ballot_w64(keep);
    kc += (uint32_t)__builtin_popcountll(km[k]);
    erun += (uint32_t)__builtin_popcountll(em[k]);
  }
  if (lane == 0) s_keep[wave] = kc;
  __syncthreads();
  uint32_t krun = gt_before + min(need, eq_before);
  for (int w = 0; w < wave; ++w) krun += s_keep[w];
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    if ((km[k] >> lane) & 1ull) {
      const uint32_t pos = krun + (uint32_t)__builtin_popcountll(km[k] & lt);
      if (pos < R) {
        rkey[pos] = ~c[k];  // ascending ~count = descending count
        rval[pos] = base + (uint64_t)k * 64 + lane;
      }
    }
    krun += (uint32_t)__builtin_popcountll(km[k]);
  }
}

// ---- 6. output ----------------------------------------------------------------

__global__ __launch_bounds__(256) void k_unpack(const uint32_t* rkey, const uint64_t* rval,
                                                const uint64_t* ukey, const uint32_t* uhi,
                                                uint64_t skip, uint64_t m, int n,
                                                int32_t* tuples, int64_t* counts) {
  const uint64_t i = (uint64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < m) {
    const uint64_t run = rval[skip + i];
    const uint64_t k = ukey[run];
    const int nlo = uhi ? 3 : n;  // tokens held in the low word
    int32_t* t = tuples + i * n;
    if (uhi) t[0] = (int32_t)uhi[run];
    for (int j = 0; j < nlo; ++j)
      t[n - nlo + j] = (int32_t)((k >> (18 * (nlo - 1 - j))) & 0x3FFFFu);
    counts[i] = (int64_t)(uint32_t)~rkey[skip + i];
  }
}

uint32_t blocks_for(uint64_t n, uint64_t per) { return (uint32_t)((n + per - 1) / per); }

// Exclusive scan of n uint32 values (in may equal out); total to *total (device).
hipError_t scan_u32(const uint32_t* in, uint32_t* out, uint64_t n, uint32_t* part,
                    hipStream_t s) {
  const uint32_t nb = blocks_for(n, kScanBlock);
  if (nb == 0) return hipSuccess;
  if (nb > (uint32_t)kScanBlock) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_scan_reduce, dim3(nb), dim3(kScanThreads), 0, s, in, n, part);
  hipLaunchKernelGGL(k_scan_down, dim3(nb), dim3(kScanThreads), 0, s, in, n, part, out);
  return hipGetLastError();
}

template <class K, class V, bool PAIRS, int SRC>
hipError_t radix_pass(K* keys, K* keys_alt, V* vals, V* vals_alt, const TokSrc& ts,
                      uint64_t n, int shift, uint32_t ntiles, uint32_t* hist, uint32_t* part,
                      hipStream_t s) {
  constexpr int ITEMS = tile_items<K, PAIRS, V>();
  hipLaunchKernelGGL((k_rs_hist<K, tile_keys<K, PAIRS, V>(), SRC>), dim3(ntiles), dim3(kHistThreads),
                     0, s, keys, ts, n, shift, hist, ntiles);
  hipError_t e = scan_u32(hist, hist, (uint64_t)kBins * ntiles, part, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_rs_scatter<K, V, PAIRS, ITEMS, SRC>), dim3(ntiles), dim3(kTileThreads), 0, s,
                     keys, vals, ts, n, shift, hist, ntiles, keys_alt, vals_alt);
  return hipGetLastError();
}

// Stable LSD sort of n keys (and payloads) by their low `bits` bits; the
// first pass reads its keys (and payloads) from SRC.  hist holds
// kBins x ceil(n / kMinTile) entries.
template <class K, bool PAIRS, int SRC = kSrcKeys, class V = uint64_t>
hipError_t radix_sort(K*& keys, K*& keys_alt, V*& vals, V*& vals_alt, uint64_t n,
                      int bits, uint32_t* hist, uint32_t* part, hipStream_t s,
                      const TokSrc& ts = TokSrc{nullptr, 0, 0, 0, 0}) {
  const uint32_t ntiles = blocks_for(n, tile_keys<K, PAIRS, V>());
  if (ntiles == 0) return hipSuccess;
  for (int shift = 0; shift < bits; shift += kDigitBits) {
    const hipError_t e =
        shift == 0
            ? radix_pass<K, V, PAIRS, SRC>(keys, keys_alt, vals, vals_alt, ts, n, shift, ntiles,
                                        hist, part, s)
            : radix_pass<K, V, PAIRS, kSrcKeys>(keys, keys_alt, vals, vals_alt, ts, n, shift,
                                             ntiles, hist, part, s);
    if (e != hipSuccess) return e;
    std::swap(keys, keys_alt);
    if (PAIRS) std::swap(vals, vals_alt);
  }
  return hipGetLastError();
}

// Scratch of the construction: device buffers kept for reuse by later calls
// (a hipMalloc / hipFree pair costs about 25 / 150 us per buffer and
// synchronises the device; a construction takes a dozen buffers) until
// tfe_ngram_release.  A request takes the smallest idle buffer of the device
// that holds it without wasting more than half; on a miss the device's idle
// buffers are returned first, so the cache never holds more than the calls
// in flight plus the buffers of one call.
struct CachedBuf {
  void* p;
  size_t bytes;
  int device;
  bool used;
};
std::mutex g_cache_mu;
std::vector<CachedBuf> g_cache;

void* cache_get(int device, size_t bytes) {
  constexpr size_t kGrain = (size_t)2 << 20;
  std::lock_guard<std::mutex> lock(g_cache_mu);
  int best = -1;
  for (size_t i = 0; i < g_cache.size(); ++i) {
    const CachedBuf& c = g_cache[i];
    if (!c.used && c.device == device && c.bytes >= bytes && c.bytes <= 2 * bytes + kGrain &&
        (best < 0 || c.bytes < g_cache[(size_t)best].bytes))
      best = (int)i;
  }
  if (best >= 0) {
    g_cache[(size_t)best].used = true;
    return g_cache[(size_t)best].p;
  }
  for (size_t i = 0; i < g_cache.size();) {
    if (!g_cache[i].used && g_cache[i].device == device) {
      dev_free(g_cache[i].p);
      g_cache[i] = g_cache.back();
      g_cache.pop_back();
    } else {
      ++i;
    }
  }
  const size_t rounded = (bytes + kGrain - 1) / kGrain * kGrain;
  void* p = nullptr;
  if (dev_malloc(&p, rounded) != hipSuccess) return nullptr;
  g_cache.push_back(CachedBuf{p, rounded, device, true});
  return p;
}

void cache_put(void* p) {
  std::lock_guard<std::mutex> lock(g_cache_mu);
  for (CachedBuf& c : g_cache)
    if (c.p == p) c.used = false;
}

struct Scratch {
  hipStream_t s;
  int device = 0;
  std::vector<void*> bufs;
  explicit Scratch(hipStream_t stream) : s(stream) { (void)hipGetDevice(&device); }
  ~Scratch() {
    // Idle only once the stream is done with them (error paths return early).
    (void)hipStreamSynchronize(s);
    for (void* p : bufs) cache_put(p);
  }
  template <class T>
  T* get(uint64_t count) {
    void* p = cache_get(device, std::max<uint64_t>(count, 1) * sizeof(T));
    if (p) bufs.push_back(p);
    return (T*)p;
  }
};

#define BUILD_HIP(call, what)                                                        \
  do {                                                                               \
    hipError_t e_ = (call);                                                          \
    if (e_ != hipSuccess) return fail(TFE_ERR_HIP, "%s: %s", what, hipGetErrorString(e_)); \
  } while (0)

tfe_status ngram_top(const int32_t* tokens, int64_t N, int32_t vocab, int32_t n, int64_t skip,
                     int64_t top, int32_t* out_tuples, int64_t* out_counts, int64_t* written,
                     hipStream_t s) {
  if (!written) return fail(TFE_ERR_INVALID_ARG, "null written");
  *written = 0;
  // The two-level scans cover up to 2^28 elements.
  if (N < 0 || N > (1ll << 28)) return fail(TFE_ERR_INVALID_ARG, "N outside [0, 2^28]");
  if (vocab < 1 || vocab > (1 << 18)) return fail(TFE_ERR_INVALID_ARG, "vocab outside [1, 2^18]");
  if (n < 1 || n > 4) return fail(TFE_ERR_UNSUPPORTED, "n = %d (1..4 supported)", n);
  if (skip < 0 || top < 0) return fail(TFE_ERR_INVALID_ARG, "negative skip or top");
  if (N < n || top == 0) return TFE_OK;
  if (!tokens || !out_tuples || !out_counts)
    return fail(TFE_ERR_INVALID_ARG, "null tokens or outputs");
  // Allocates scratch and waits for the stream: not capturable.
  {
    const tfe_status st = refuse_capture(s, "tfe_ngram_top");
    if (st != TFE_OK) return st;
  }
  const uint64_t nwin = (uint64_t)(N - n + 1);
  const bool wide = n == 4;
  Scratch sc(s);
  uint64_t* keys = sc.get<uint64_t>(nwin);
  uint64_t* keys_alt = sc.get<uint64_t>(nwin);
  // 4-grams: the high word, payload of the low-word sort, then keys.
  uint32_t* wv = wide ? sc.get<uint32_t>(nwin) : nullptr;
  uint32_t* wv_alt = wide ? sc.get<uint32_t>(nwin) : nullptr;
  uint32_t* hi = nullptr;
  uint32_t* hi_alt = nullptr;
  const uint32_t ntiles = blocks_for(nwin, kMinTile);
  uint32_t* hist = sc.get<uint32_t>((uint64_t)kBins * ntiles);
  uint32_t* part = sc.get<uint32_t>(kScanBlock);
  unsigned long long* d_count = sc.get<unsigned long long>(1);
  uint32_t* d_small = sc.get<uint32_t>(8);
  uint32_t* sel_bins = sc.get<uint32_t>(kSelBins);
  if (!keys || !keys_alt || !hist || !part || !d_count || !d_small || !sel_bins ||
      (wide && (!wv || !wv_alt)))
    return fail(TFE_ERR_OOM, "n-gram scratch for %llu windows", (unsigned long long)nwin);
  // 1-2. keys of all windows, formed by the first radix pass, sorted (one
  // bit above the key fields carries the invalid-window mark); the valid
  // keys are the first M.  4-grams sort by the low word, then stably by the
  // high word (LSD over both words).
  uint64_t* no_vals = nullptr;
  uint64_t* no_vals2 = nullptr;
  // Invalid windows: with vocab < 2^18 the oldest-token field holds vocab
  // (above every valid token), so the keys keep 18 n bits; with vocab =
  // 2^18 one more bit above the fields.
  const bool narrow = vocab < (1 << 18);
  const uint64_t mark = narrow ? (uint64_t)vocab << (18 * (n - 1)) : 1ull << (18 * n);
  const uint32_t mark4 = narrow ? (uint32_t)vocab : (1u << 18);
  const TokSrc ts{tokens, n, vocab, mark, mark4};
  if (!wide) {
    const int bits = 18 * n + (narrow ? 0 : 1);
    hipError_t e = n == 1   ? radix_sort<uint64_t, false, 1>(keys, keys_alt, no_vals, no_vals2,
                                                             nwin, bits, hist, part, s, ts)
                   : n == 2 ? radix_sort<uint64_t, false, 2>(keys, keys_alt, no_vals, no_vals2,
                                                             nwin, bits, hist, part, s, ts)
                            : radix_sort<uint64_t, false, 3>(keys, keys_alt, no_vals, no_vals2,
                                                             nwin, bits, hist, part, s, ts);
    BUILD_HIP(e, "key sort");
    hipLaunchKernelGGL(k_count_valid, dim3(1), dim3(1), 0, s, keys, nwin, mark, d_count);
  } else {
    BUILD_HIP((radix_sort<uint64_t, true, kSrcNgram4, uint32_t>(keys, keys_alt, wv, wv_alt, nwin,
                                                                54, hist, part, s, ts)),
              "low-word sort");
    hi = wv;  // the high words, now in low-word order, become the keys
    hi_alt = wv_alt;
    BUILD_HIP((radix_sort<uint32_t, true>(hi, hi_alt, keys, keys_alt, nwin, narrow ? 18 : 19,
                                          hist, part, s)),
              "high-word sort");
    hipLaunchKernelGGL(k_count_valid_hi, dim3(1), dim3(1), 0, s, hi, nwin, mark4, d_count);
  }
  BUILD_HIP(hipGetLastError(), "count launch");
  unsigned long long m_host = 0;
  BUILD_HIP(hipMemcpyAsync(&m_host, d_count, sizeof m_host, hipMemcpyDeviceToHost, s), "copy");
  BUILD_HIP(hipStreamSynchronize(s), "sync");
  const uint64_t M = m_host;
  if (M == 0) return TFE_OK;
  // 3. runs.
  const uint32_t nbr = blocks_for(M, kScanBlock);
  if (wide)
    hipLaunchKernelGGL(k_runs_reduce<true>, dim3(nbr), dim3(kScanThreads), 0, s, keys, hi, M, part);
  else
    hipLaunchKernelGGL(k_runs_reduce<false>, dim3(nbr), dim3(kScanThreads), 0, s, keys, hi, M,
                       part);
  hipLaunchKernelGGL(k_scan_partials, dim3(1), dim3(kScanThreads), 0, s, part, nbr, d_small);
  BUILD_HIP(hipGetLastError(), "run count launches");
  uint32_t U = 0;
  BUILD_HIP(hipMemcpyAsync(&U, d_small, sizeof U, hipMemcpyDeviceToHost, s), "copy");
  BUILD_HIP(hipStreamSynchronize(s), "sync");
  uint64_t* ukey = sc.get<uint64_t>(U);
  uint32_t* uhi = wide ? sc.get<uint32_t>(U) : nullptr;
  uint32_t* ustart = sc.get<uint32_t>(U);
  uint32_t* ucnt = sc.get<uint32_t>(U);
  if (!ukey || !ustart || !ucnt || (wide && !uhi)) return fail(TFE_ERR_OOM, "run arrays");
  if (wide)
    hipLaunchKernelGGL(k_runs_write<true>, dim3(nbr), dim3(kScanThreads), 0, s, keys, hi, M, part,
                       ukey, uhi, ustart);
  else
    hipLaunchKernelGGL(k_runs_write<false>, dim3(nbr), dim3(kScanThreads), 0, s, keys, hi, M, part,
                       ukey, uhi, ustart);
  BUILD_HIP(hipMemsetAsync(sel_bins, 0, kSelBins * sizeof(uint32_t), s), "memset");
  hipLaunchKernelGGL(k_run_counts, dim3(blocks_for(U, 16384)), dim3(1024), 0, s, ustart, U,
                     (uint32_t)M, ucnt, sel_bins);
  BUILD_HIP(hipGetLastError(), "run launches");
  const uint64_t R = std::min<uint64_t>((uint64_t)skip + (uint64_t)top, U);
  if (R <= (uint64_t)skip) return TFE_OK;
  // 4. the R-th largest count and the runs that make ranks [0, R): from the
  // small-count histogram when it lies below kSelBins - 1, else by a radix
  // select over the counts (its passes return at once when done).
  uint32_t* selh = hist;  // 256 bins, cleared by each pick
  const uint32_t state0[5] = {0u, 0u, (uint32_t)R, 0u, 0u};
  BUILD_HIP(hipMemsetAsync(selh, 0, 256 * sizeof(uint32_t), s), "memset");
  BUILD_HIP(hipMemcpyAsync(d_small, state0, sizeof state0, hipMemcpyHostToDevice, s), "copy");
  hipLaunchKernelGGL(k_sel_small, dim3(1), dim3(1024), 0, s, sel_bins, d_small);
  // The R largest counts add up to at most M, so the R-th largest is at
  // most M / R: below kSelBins - 1 the small-count histogram has found it
  // for certain, and the radix passes (which would return at once, at
  // about 5 us per launch) are not launched.
  if (M / R >= (uint64_t)kSelBins - 1) {
    // Few blocks: each adds its LDS histogram to the 256 global bins once.
    const uint32_t sel_blocks = std::min<uint32_t>(blocks_for(U, 256), 512);
    for (int shift = 24; shift >= 0; shift -= 8) {
      hipLaunchKernelGGL(k_sel_hist, dim3(sel_blocks), dim3(256), 0, s, ucnt, U, d_small, shift,
                         selh);
      hipLaunchKernelGGL(k_sel_pick, dim3(1), dim3(256), 0, s, selh, d_small, shift);
    }
  }
  BUILD_HIP(hipGetLastError(), "select launches");
  // state = {c*, ~0, needed runs with count c*, runs above c*}.
  uint32_t* rkey = sc.get<uint32_t>(R);
  uint32_t* rkey_alt = sc.get<uint32_t>(R);
  uint64_t* rval = sc.get<uint64_t>(R);
  uint64_t* rval_alt = sc.get<uint64_t>(R);
  if (!rkey || !rkey_alt || !rval || !rval_alt) return fail(TFE_ERR_OOM, "rank arrays");
  // Per-block numbers in the radix histogram buffer (idle until the rank
  // sort; it holds kBins x ntiles >= 2 x blocks entries).
  const uint32_t nbs = blocks_for(U, kScanBlock);
  uint32_t* part_gt = hist;
  uint32_t* part_eq = hist + nbs;
  hipLaunchKernelGGL(k_sel_count, dim3(nbs), dim3(kScanThreads), 0, s, ucnt, U, d_small, part_gt,
                     part_eq);
  hipLaunchKernelGGL(k_sel_place, dim3(nbs), dim3(kScanThreads), 0, s, ucnt, U, d_small, part_gt,
                     part_eq, (uint32_t)R, rkey, rval);
  BUILD_HIP(hipGetLastError(), "selection launches");
  // 5. rank by count (stable: tuple order among equal counts).
  BUILD_HIP((radix_sort<uint32_t, true>(rkey, rkey_alt, rval, rval_alt, R, 32, hist, part, s)),
            "rank sort");
  // 6. ranks [skip, R).
  const uint64_t m = R - (uint64_t)skip;
  hipLaunchKernelGGL(k_unpack, dim3(blocks_for(m, 256)), dim3(256), 0, s, rkey, rval, ukey, uhi,
                     (uint64_t)skip, m, n, out_tuples, out_counts);
  BUILD_HIP(hipGetLastError(), "unpack launch");
  BUILD_HIP(hipStreamSynchronize(s), "sync");
  *written = (int64_t)m;
  return TFE_OK;
}

}  // namespace
}  // namespace tfe

extern "C" tfe_status tfe_ngram_release(void) {
  tfe::begin_call();
  std::lock_guard<std::mutex> lock(tfe::g_cache_mu);
  int cur = 0;
  (void)hipGetDevice(&cur);
  for (size_t i = 0; i < tfe::g_cache.size();) {
    if (!tfe::g_cache[i].used) {
      (void)hipSetDevice(tfe::g_cache[i].device);
      tfe::dev_free(tfe::g_cache[i].p);
      tfe::g_cache[i] = tfe::g_cache.back();
      tfe::g_cache.pop_back();
    } else {
      ++i;
    }
  }
  (void)hipSetDevice(cur);
  return TFE_OK;
}

extern "C" tfe_status tfe_ngram_top(const int32_t* tokens, int64_t n_tokens, int32_t vocab,
                                    int32_t n, int64_t skip, int64_t top, int32_t* out_tuples,
                                    int64_t* out_counts, int64_t* written, void* stream) {
  tfe::begin_call();
  return tfe::ngram_top(tokens, n_tokens, vocab, n, skip, top, out_tuples, out_counts, written,
                        (hipStream_t)stream);
}
