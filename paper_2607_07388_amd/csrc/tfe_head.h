// Internal declarations of the early-exit prefetch head (not part of the C ABI).
#pragma once
#include <stdint.h>

#include <hip/hip_runtime_api.h>

namespace tfe {

// Chunks per batch row of the top-K selection and its limits.
constexpr int kHeadMaxK = 256;
constexpr int kHeadMaxChunks = 16;
constexpr int kHeadChunkMax = 16384;  // logits per chunk (keys held in registers)

struct HeadArgs {
  const void* w;        // [V x D] bf16, row-major
  const void* hidden;   // [B x D] bf16
  float* logits;        // [B x V] scratch
  uint64_t* cand;       // [B x C x K] scratch: selected (logit, id) keys per chunk
  uint32_t* cnt;        // [B x C] keys selected per chunk
  float* part;          // [B x C x 2] chunk max logit and sum of exp(logit - max)
  int32_t* top_ids;     // [B x K]
  float* top_prob;      // [B x K]
  uint32_t V, D, B, K, C;
};

// Chunks per row for a vocabulary of V tokens.
uint32_t head_chunks(uint32_t V);
// True if D has a logits kernel.
bool head_dim_supported(int D);
// Bytes of static LDS the logits kernel uses for D (checked against the device).
uint32_t head_lds_bytes(int D);

hipError_t launch_head_logits(const HeadArgs& a, uint32_t blocks, hipStream_t s);
hipError_t launch_head_select(const HeadArgs& a, hipStream_t s);
hipError_t launch_head_merge(const HeadArgs& a, hipStream_t s);

}  // namespace tfe
