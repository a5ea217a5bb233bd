// Internal declarations of the early-exit prefetch head (not part of the C ABI).
#pragma once
#include <stdint.h>

#include <hip/hip_runtime_api.h>

namespace tfe {

// Limits of the top-K selection.
constexpr int kHeadMaxK = 256;
constexpr int kHeadMaxTiles = 16384;  // 16-token tiles per row: vocab <= 2^18

struct HeadArgs {
  const void* w;        // [V x D] bf16, row-major
  const void* hidden;   // [B x D] bf16
  // Scratch: groups of 64 rows (B rounded up), tpitch 16-token tiles per
  // group (V rounded up to 32, over 16), tblocks = tpitch / 16 rounded up.
  float* logits;        // [groups x tpitch x 64 x 16], tile-major
  uint64_t* tkey;       // [groups x tblocks x 64 x 16]: largest (logit, id) key per tile
  float* tsum;          // [groups x tblocks x 64 x 16]: sum of exp(logit - tile max)
  uint64_t* bmax;       // [groups x nblk x 64]: largest tile key per (logits block, row)
  int32_t* top_ids;     // [B x K]
  float* top_prob;      // [B x K]
  uint32_t V, tpitch, tblocks, D, B, K;
  uint32_t nblk;        // logits blocks per 64-row group (one per compute unit)
  // One-launch path (B <= 64; see launch_head_fused): per (row, logits
  // block) the high word of the block's largest key (0: no logits) and its
  // sum of exp(logit - that logit); per (row, block) a segment of ccap
  // words: the number of the block's logit keys that reach the row's bound,
  // then the keys; the grid barrier's counters and flags and a fault word.
  uint32_t* bhi;        // [64 x nblk]
  uint32_t* bsum;       // [64 x nblk], float bits
  uint64_t* cand;       // [64 x nblk x ccap]
  unsigned long long* bar;
  unsigned long long* fault;  // the last faulted call's epoch + 1
  uint32_t ccap;        // 1 + 16 x the most tiles a block owns, rounded up to 16
  unsigned long long* ectl;  // [16 i], i < 16: blocks of earlier one-launch calls
                             // on this scratch that have left (block b adds to b mod 16)
  uint32_t wait_limit;  // polls before a barrier wait gives up (kHeadWaitLimit)
};

// Polls of a one-launch barrier before it gives up (about a second).  The
// environment variable TFE_HEAD_WAIT_LIMIT overrides it per call, so that
// tests can force the give-up path from the host.
constexpr uint32_t kHeadWaitLimit = 1u << 20;

// True if D has a logits kernel.
bool head_dim_supported(int D);
// Bytes of static LDS the logits kernel uses for D (checked against the device).
uint32_t head_lds_bytes(int D);

hipError_t launch_head_logits(const HeadArgs& a, hipStream_t s);
hipError_t launch_head_rows(const HeadArgs& a, hipStream_t s);

// The one-launch head: true if a call of this shape can take it (B <= 64,
// B and K at most nblk, nblk a power of two <= 256, at most 48 tiles per
// block).
bool head_fused_fits(const HeadArgs& a);
// Words per (row, block) segment of the candidate scratch for this vocabulary.
uint32_t head_fused_ccap(uint32_t V, uint32_t nblk);
// True if a block of the one-launch kernel for D fits a compute unit of the
// current device.
bool head_fused_resident(int D);
// Launch of nblk blocks, one per compute unit, all resident at once.
hipError_t launch_head_fused(const HeadArgs& a, hipStream_t s);

}  // namespace tfe
