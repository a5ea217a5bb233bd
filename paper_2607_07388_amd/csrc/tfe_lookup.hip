// Fused lookup + inject kernel for tables resident in HBM (gfx950, wave64).
//
// One wavefront owns one position and runs the whole path for it:
//   1. key formation: the n-grams ending at the position (n = n_max..n_min)
//      are packed into 64-bit keys (+ a 32-bit extension for 4-grams)
//      (Eq. 3, first level of Eq. 10);
//   2. probe: 8 lanes per key read the key's home bucket (8 slots = 128 bytes)
//      with one 16-byte load each and compare full keys; ballots give match
//      and empty masks, so an exact answer normally costs one bucket read per
//      key; all lengths are probed at once and the longest match is the
//      lowest matching lane group (Sec. 4.2);
//   3. gather: the matched value row is streamed with 16-byte loads, 1 KiB
//      per wave instruction (Eq. 3);
//   4. gate + residual: three fp32 wave reductions (h.h, m.m, h.m) give the
//      gate, then h' = h + g m is formed with fmaf and rounded to nearest
//      even (Eq. 5).
// The hidden row is requested first, so its transfer overlaps the dependent
// token -> bucket -> value chain.  Hidden rows are read and written with
// non-temporal hints (touched once); value rows use the normal cached path
// because Zipf-distributed queries hit the same rows repeatedly.  Nothing is
// staged through LDS: each lane keeps its own 16 bf16 of the row in
// registers, and the only cross-lane traffic is the three reductions (DPP).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tfe_device.h"
#include "tfe_internal.h"

// Launch-shape defaults (tuning knobs of the launchers below).
#ifndef TFE_BIG_WPB
#define TFE_BIG_WPB 4
#endif
#ifndef TFE_SMALL_WPB
#define TFE_SMALL_WPB 1
#endif
#ifndef TFE_SMALL_T
#define TFE_SMALL_T 4096
#endif

namespace tfe {
namespace {

using dev::u32x4;

template <int DT, int NCH, int WPB>
__global__ __launch_bounds__(WPB * 64) void k_lookup_inject(const LookupArgs a) {
  constexpr int ROW_VECS = NCH * 64;  // 16-byte vectors per row
  const int lane = threadIdx.x & 63;
  const uint32_t p = blockIdx.x * WPB + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (p >= a.T) return;

  u32x4 hv[NCH];
  const u32x4* hin = (const u32x4*)a.hin + (size_t)p * ROW_VECS;
#pragma unroll
  for (int k = 0; k < NCH; ++k) hv[k] = dev::load_hidden(hin + k * 64 + lane);

  int32_t tw[4];
  dev::window_tokens(a, p, tw);
  const dev::Probe pr = dev::probe_begin(a, tw, lane);
  int len;
  const int32_t row = dev::probe_finish(a, pr, lane, &len);
  if (lane == 0) {
    dev::write_result(a, p, row, len);
    dev::count_hit(a, row >= 0);
  }

  u32x4* out = (u32x4*)a.hout + (size_t)p * ROW_VECS;
  if (row < 0) {
    if (!a.inplace) {
#pragma unroll
      for (int k = 0; k < NCH; ++k) dev::store_out(hv[k], out + k * 64 + lane);
    }
    return;
  }
  u32x4 mv[NCH];
  const u32x4* mrow = (const u32x4*)a.values + (size_t)row * ROW_VECS;
#pragma unroll
  for (int k = 0; k < NCH; ++k) mv[k] = dev::load_value(mrow + k * 64 + lane);
  const float g = dev::gate_of<DT, NCH>(a, hv, mv);
  dev::store_injected<DT, NCH>(out, hv, mv, g, lane);
}

template <int DT, int NCH, int WPB>
hipError_t launch_shape(const LookupArgs& a, hipStream_t stream) {
  const uint32_t blocks = (a.T + WPB - 1) / WPB;
  hipLaunchKernelGGL((k_lookup_inject<DT, NCH, WPB>), dim3(blocks), dim3(WPB * 64), 0, stream,
                     a);
  return hipGetLastError();
}

// Small batches (decode steps) put one wave in each block, spreading the rows
// over as many compute units as possible; large batches use 4-wave blocks.  A
// launch of 16384 rows is two generations of resident waves, so the second
// generation's reads overlap the first generation's writes.  (Measured
// alternatives that were slower on MI355X: two rows per wave, and a
// software-pipelined walk that probes the next row while streaming the
// current one.)
template <int DT, int NCH>
hipError_t launch_t(const LookupArgs& a, hipStream_t stream) {
  if (a.T < TFE_SMALL_T) return launch_shape<DT, NCH, TFE_SMALL_WPB>(a, stream);
  return launch_shape<DT, NCH, TFE_BIG_WPB>(a, stream);
}

}  // namespace

bool dim_supported(int dtype, int dim) {
  const int per_chunk = dtype == TFE_F32 ? 256 : 512;
  if (dim <= 0 || dim % per_chunk) return false;
  const int nch = dim / per_chunk;
  return nch == 1 || nch == 2 || nch == 4 || nch == 8;
}

hipError_t launch_lookup_inject(const LookupArgs& a, int dtype, int dim, hipStream_t stream) {
  if (a.T == 0) return hipSuccess;
  const int nch = dim / (dtype == TFE_F32 ? 256 : 512);
  if (dtype == TFE_F32) {
    switch (nch) {
      case 1: return launch_t<0, 1>(a, stream);
      case 2: return launch_t<0, 2>(a, stream);
      case 4: return launch_t<0, 4>(a, stream);
      case 8: return launch_t<0, 8>(a, stream);
    }
  } else {
    switch (nch) {
      case 1: return launch_t<1, 1>(a, stream);
      case 2: return launch_t<1, 2>(a, stream);
      case 4: return launch_t<1, 4>(a, stream);
      case 8: return launch_t<1, 8>(a, stream);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace tfe
