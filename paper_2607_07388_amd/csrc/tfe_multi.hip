// Multi-match lookup + inject for tables resident in HBM (gfx950, wave64).
//
// Every phrase that ends at the position and is in the table is retained,
// and their value rows are combined as m = sum_j alpha_j v_j with weights
// that add up to 1 (Eq. 4, Eq. 11): proportional to the phrase length, or
// uniform.  The aggregate goes through the same gate and residual as the
// longest-match kernel (Eq. 5).
//
// One wavefront per position, as in the longest-match kernel: the probe
// already resolves every length at once (lane group j holds the n-gram of
// length n_max - j), so the only differences are that every matching group's
// row is kept and that up to three value rows are streamed.  All row loads
// are issued before the first is consumed; the aggregate stays in fp32
// registers (never rounded) and feeds the gate sums directly.  With a single
// retained row alpha = 1 and the arithmetic is the longest-match kernel's,
// so both kernels give identical bytes there.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/tfe.h"
#include "tfe_device.h"
#include "tfe_internal.h"

namespace tfe {
namespace {

using dev::u32x4;

template <int DT, int NCH, int WPB>
__global__ __launch_bounds__(WPB * 64) void k_lookup_inject_multi(const LookupArgs a) {
  constexpr int ROW_VECS = NCH * 64;
  constexpr int VN = dev::Vec<DT>::N;
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
  const dev::Walk w = dev::probe_walk(a, pr, lane);

  // Row of lane group j (length n_max - j), wave-uniform; -1 if absent.
  int32_t rows[3];
  float wt[3];
  float wsum = 0.f;
  uint32_t mask = 0;
  const int span = a.n_max - a.n_min;  // column of length n is n - n_min
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    const uint32_t bits = (uint32_t)(w.found >> (8 * j)) & 0xFFu;
    rows[j] = bits ? __builtin_amdgcn_readlane(w.myrow, 8 * j + __builtin_ctz(bits)) : -1;
    wt[j] = rows[j] < 0 ? 0.f : (a.weighting == TFE_WEIGHT_LENGTH ? (float)(a.n_max - j) : 1.f);
    wsum += wt[j];
    if (rows[j] >= 0) mask |= 1u << (span - j);
  }
  if (lane <= span) {
    const int j = span - lane;
    a.slot_out[(size_t)p * (span + 1) + lane] = j == 0 ? rows[0] : (j == 1 ? rows[1] : rows[2]);
  }
  if (lane == 0) {
    a.hit[p] = (uint8_t)mask;
    dev::count_hit(a, mask != 0);
  }

  u32x4* out = (u32x4*)a.hout + (size_t)p * ROW_VECS;
  if (mask == 0) {
    if (!a.inplace) {
#pragma unroll
      for (int k = 0; k < NCH; ++k) dev::store_out(hv[k], out + k * 64 + lane);
    }
    return;
  }
  u32x4 mv[3][NCH];
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    if (rows[j] < 0) continue;
    const u32x4* mrow = (const u32x4*)a.values + (size_t)rows[j] * ROW_VECS;
#pragma unroll
    for (int k = 0; k < NCH; ++k) mv[j][k] = dev::load_value(mrow + k * 64 + lane);
  }
  // m = sum_j alpha_j v_j, in group order (longest first); the first term
  // is a plain product so that alpha = 1 reproduces the row exactly.
  float m[NCH][VN];
  bool first = true;
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    if (rows[j] < 0) continue;
    const float alpha = wt[j] / wsum;
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      float v[VN];
      dev::unpack<DT>(mv[j][k], v);
#pragma unroll
      for (int i = 0; i < VN; ++i) m[k][i] = first ? alpha * v[i] : fmaf(alpha, v[i], m[k][i]);
    }
    first = false;
  }
  float g = a.scale;
  if (a.gate == TFE_GATE_SIGMOID) {
    float shh = 0.f, smm = 0.f, shm = 0.f;
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      float h[VN];
      dev::unpack<DT>(hv[k], h);
#pragma unroll
      for (int i = 0; i < VN; ++i) {
        shh = fmaf(h[i], h[i], shh);
        smm = fmaf(m[k][i], m[k][i], smm);
        shm = fmaf(h[i], m[k][i], shm);
      }
    }
    g = dev::gate_finish(a, shh, smm, shm);
  }
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    float h[VN], o[VN];
    dev::unpack<DT>(hv[k], h);
#pragma unroll
    for (int i = 0; i < VN; ++i) o[i] = fmaf(g, m[k][i], h[i]);
    dev::store_out(dev::pack<DT>(o), out + k * 64 + lane);
  }
}

template <int DT, int NCH, int WPB>
hipError_t launch_shape(const LookupArgs& a, hipStream_t stream) {
  const uint32_t blocks = (a.T + WPB - 1) / WPB;
  hipLaunchKernelGGL((k_lookup_inject_multi<DT, NCH, WPB>), dim3(blocks), dim3(WPB * 64), 0,
                     stream, a);
  return hipGetLastError();
}

// Same launch shapes as the longest-match kernel: one wave per block for
// decode-sized calls, four for large ones.
template <int DT, int NCH>
hipError_t launch_t(const LookupArgs& a, hipStream_t stream) {
  if (a.T < 4096) return launch_shape<DT, NCH, 1>(a, stream);
  return launch_shape<DT, NCH, 4>(a, stream);
}

}  // namespace

hipError_t launch_lookup_inject_multi(const LookupArgs& a, int dtype, int dim,
                                      hipStream_t stream) {
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
