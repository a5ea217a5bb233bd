// Internal declarations of libtfe (not part of the C ABI).
#pragma once
#include <stdarg.h>
#include <stdint.h>

#include "../../include/tfe.h"
#include "tfe_index.h"

#if defined(__HIPCC__) || defined(__HIP_PLATFORM_AMD__)
#include <hip/hip_runtime_api.h>
#endif

namespace tfe {

// Thread-local error message; fail() formats it and returns the status.
tfe_status fail(tfe_status st, const char* fmt, ...);
void clear_error();

int64_t index_capacity(int64_t n, double lf);
tfe_status validate_phrases(const int32_t* tokens, const uint8_t* lens, int64_t P, int n_min,
                            int n_max, int vocab);
tfe_status build_index(const int32_t* tokens, const uint8_t* lens, int64_t P, int n_max,
                       tfe_slot* slots, int64_t cap);

#if defined(__HIPCC__) || defined(__HIP_PLATFORM_AMD__)

// Per-call arguments of the lookup + inject kernels.
struct LookupArgs {
  const tfe_slot* slots;
  uint64_t bucket_mask;       // buckets - 1
  const void* values;         // resident value rows [P x dim]
  const int32_t* tokens;      // [B x W]
  uint32_t T;                 // B * S (< 2^31)
  int32_t S, ctx, W;          // W = ctx + S
  int32_t n_min, n_max, vocab;
  const void* hin;
  void* hout;
  int32_t inplace;
  uint8_t* hit;
  int32_t* slot_out;
  uint8_t* len_out;           // may be null
  int32_t gate;
  float scale;
  float inv_d;                // 1 / dim
  float inv_sqrt_d;           // 1 / sqrt(dim)
};

// Launches the fused resident-table kernel; returns the launch error.
hipError_t launch_lookup_inject(const LookupArgs& a, int dtype, int dim, hipStream_t stream);

// True if (dtype, dim) has a kernel instantiation.
bool dim_supported(int dtype, int dim);

#endif

}  // namespace tfe

#if defined(__HIPCC__) || defined(__HIP_PLATFORM_AMD__)
struct tfe_table {
  int device = 0;
  int cus = 256;                 // compute units of `device`
  int64_t n_phrases = 0;
  int32_t n_min = 2, n_max = 3, vocab = 0, dim = 0, dtype = 0;
  int64_t capacity = 0;          // index slots
  tfe_slot* d_slots = nullptr;   // [capacity]
  void* d_values = nullptr;      // resident: [P x dim]
  int64_t cache_rows = 0;        // tiered mode when > 0
  tfe_stats stats = {};
};
#endif
