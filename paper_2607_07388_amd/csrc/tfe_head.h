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
};

// True if D has a logits kernel.
bool head_dim_supported(int D);
// Bytes of static LDS the logits kernel uses for D (checked against the device).
uint32_t head_lds_bytes(int D);

hipError_t launch_head_logits(const HeadArgs& a, hipStream_t s);
hipError_t launch_head_rows(const HeadArgs& a, hipStream_t s);

}  // namespace tfe
