// Fused lookup + inject kernel for tables resident in HBM (gfx950, wave64).
//
// One wavefront owns one position at a time and runs the whole path for it:
//   1. key formation: the n-grams ending at the position (n = n_max..n_min)
//      are packed into 64-bit keys (+ a 32-bit extension for 4-grams)
//      (Eq. 3, Eq. 10 first level);
//   2. probe: 8 lanes per key read the key's home bucket (8 slots = 128 bytes)
//      with one 16-byte load each and compare full keys; a ballot gives
//      match and empty masks, so an exact answer normally costs one bucket
//      read per key; all lengths are probed at once and the longest match is
//      the lowest matching lane group (Sec. 4.2);
//   3. gather: the matched value row is streamed with 16-byte loads, 1 KiB
//      per wave instruction (Eq. 3);
//   4. gate + residual: three fp32 wave reductions (h.h, m.m, h.m) give the
//      gate, then h' = h + g m is formed with fmaf and rounded to nearest
//      even (Eq. 5).
// The hidden row is requested before the probe so its load overlaps the
// dependent bucket and value loads.  Hidden rows are read and written with
// non-temporal hints (touched once); value rows use the normal cached path
// because Zipf-distributed queries hit the same rows repeatedly.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "tfe_internal.h"

namespace tfe {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Elements of type DT held by one 16-byte vector.
template <int DT> struct Vec;
template <> struct Vec<0> { static constexpr int N = 4; };  // float32
template <> struct Vec<1> { static constexpr int N = 8; };  // bfloat16

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// float32 -> bfloat16 bits, nearest even; NaN stays NaN.
__device__ __forceinline__ uint32_t to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

template <int DT>
__device__ __forceinline__ void unpack(const u32x4 v, float* f) {
  if (DT == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(v[i]);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) { f[2 * i] = bf16_lo(v[i]); f[2 * i + 1] = bf16_hi(v[i]); }
  }
}

template <int DT>
__device__ __forceinline__ u32x4 pack(const float* f) {
  u32x4 v;
  if (DT == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = __float_as_uint(f[i]);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = to_bf16(f[2 * i]) | (to_bf16(f[2 * i + 1]) << 16);
  }
  return v;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

__device__ __forceinline__ bool tok_ok(int32_t t, int32_t vocab) {
  return t >= 0 && t < vocab;
}

// Longest-match probe for the position at column c of `row` (wave-uniform).
// Returns the matched phrase row id (-1 on a miss) in every lane and its
// length in *len.
__device__ __forceinline__ int32_t probe_longest(const LookupArgs& a, const int32_t* row, int c,
                                                 int lane, int* len) {
  // Newest-first window tokens; columns before 0 do not exist.
  const int32_t t0 = row[c];
  const int32_t t1 = c >= 1 ? row[c - 1] : -1;
  const int32_t t2 = c >= 2 ? row[c - 2] : -1;
  const int32_t t3 = c >= 3 ? row[c - 3] : -1;
  const bool ok0 = tok_ok(t0, a.vocab), ok1 = tok_ok(t1, a.vocab);
  const bool ok2 = tok_ok(t2, a.vocab), ok3 = tok_ok(t3, a.vocab);

  const int j = lane >> 3;            // key group: n = n_max - j
  const int q = lane & 7;             // slot within the bucket
  const int n = a.n_max - j;
  bool active = j < 3 && n >= a.n_min && ok0 && ok1 && (n < 3 || ok2) && (n < 4 || ok3);
  const uint64_t key = tfe_key(n, (uint32_t)t0, (uint32_t)t1, n >= 3 ? (uint32_t)t2 : 0u);
  const uint32_t ext = n == 4 ? (uint32_t)t3 : 0u;
  uint64_t b = tfe_hash(key, ext) & a.bucket_mask;
  bool matched = false;
  int32_t myrow = -1;
  // Every bucket read by an active group either ends its probe or moves it
  // to the next bucket; a load factor below 1 leaves an empty slot, and the
  // bucket count bounds the walk in any case.
  for (uint64_t it = 0; it <= a.bucket_mask; ++it) {
    bool match = false, empty = false;
    if (active) {
      const u32x4 s = *(const u32x4*)(a.slots + b * TFE_SLOTS_PER_BUCKET + q);
      const uint64_t sk = (uint64_t)s[0] | ((uint64_t)s[1] << 32);
      match = sk == key && s[2] == ext;
      empty = sk == TFE_EMPTY_KEY;
      if (match) { matched = true; myrow = (int32_t)s[3]; }
    }
    const uint64_t mm = __builtin_amdgcn_ballot_w64(match);
    const uint64_t me = __builtin_amdgcn_ballot_w64(empty);
    const uint64_t grp = 0xFFull << (8 * j);
    if (active && ((mm | me) & grp)) active = false;
    if (active) b = (b + 1) & a.bucket_mask;
    if (__builtin_amdgcn_ballot_w64(active) == 0) break;
  }
  const uint64_t found = __builtin_amdgcn_ballot_w64(matched);
  if (found == 0) { *len = 0; return -1; }
  const int sel = __builtin_amdgcn_readfirstlane(__builtin_ctzll(found));
  *len = a.n_max - (sel >> 3);
  return __builtin_amdgcn_readlane(myrow, sel);
}

template <int DT, int NCH, int WPB>
__global__ __launch_bounds__(WPB * 64) void k_lookup_inject(const LookupArgs a) {
  constexpr int VN = Vec<DT>::N;
  constexpr int ROW_VECS = NCH * 64;  // 16-byte vectors per row
  const int lane = threadIdx.x & 63;
  const int64_t p = (int64_t)blockIdx.x * WPB + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (p >= a.T) return;
  const int32_t bseq = (int32_t)(p / a.S);
  const int32_t c = a.ctx + (int32_t)(p - (int64_t)bseq * a.S);

  const u32x4* hin = (const u32x4*)a.hin + p * ROW_VECS;
  u32x4 hv[NCH];
#pragma unroll
  for (int k = 0; k < NCH; ++k) hv[k] = __builtin_nontemporal_load(hin + k * 64 + lane);

  int len;
  const int32_t row = probe_longest(a, a.tokens + (int64_t)bseq * a.W, c, lane, &len);
  if (lane == 0) {
    a.hit[p] = row >= 0 ? 1 : 0;
    a.slot_out[p] = row;
    if (a.len_out) a.len_out[p] = (uint8_t)len;
  }
  u32x4* hout = (u32x4*)a.hout + p * ROW_VECS;
  if (row < 0) {
    if (!a.inplace) {
#pragma unroll
      for (int k = 0; k < NCH; ++k) __builtin_nontemporal_store(hv[k], hout + k * 64 + lane);
    }
    return;
  }
  const u32x4* mrow = (const u32x4*)a.values + (int64_t)row * ROW_VECS;
  u32x4 mv[NCH];
#pragma unroll
  for (int k = 0; k < NCH; ++k) mv[k] = mrow[k * 64 + lane];

  float shh = 0.f, smm = 0.f, shm = 0.f;
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    float h[VN], m[VN];
    unpack<DT>(hv[k], h);
    unpack<DT>(mv[k], m);
#pragma unroll
    for (int i = 0; i < VN; ++i) {
      shh = fmaf(h[i], h[i], shh);
      smm = fmaf(m[i], m[i], smm);
      shm = fmaf(h[i], m[i], shm);
    }
  }
  float g = a.scale;
  if (a.gate == TFE_GATE_SIGMOID) {
    shh = wave_sum(shh);
    smm = wave_sum(smm);
    shm = wave_sum(shm);
    const float rh = sqrtf(fmaf(shh, a.inv_d, 1e-6f));
    const float rm = sqrtf(fmaf(smm, a.inv_d, 1e-6f));
    const float z = shm / (rh * rm) * a.inv_sqrt_d;
    g = a.scale / (1.0f + expf(-z));
  }
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    float h[VN], m[VN], o[VN];
    unpack<DT>(hv[k], h);
    unpack<DT>(mv[k], m);
#pragma unroll
    for (int i = 0; i < VN; ++i) o[i] = fmaf(g, m[i], h[i]);
    __builtin_nontemporal_store(pack<DT>(o), hout + k * 64 + lane);
  }
}

constexpr int kWavesPerBlock = 4;

template <int DT, int NCH>
hipError_t launch_t(const LookupArgs& a, hipStream_t stream) {
  const int64_t blocks = (a.T + kWavesPerBlock - 1) / kWavesPerBlock;
  hipLaunchKernelGGL((k_lookup_inject<DT, NCH, kWavesPerBlock>), dim3((unsigned)blocks),
                     dim3(kWavesPerBlock * 64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

bool dim_supported(int dtype, int dim) {
  const int per_chunk = dtype == TFE_F32 ? 256 : 512;
  if (dim % per_chunk) return false;
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
