// Device building blocks shared by the lookup + inject kernels (gfx950,
// wave64): key formation and the wave-cooperative bucket probe, the fp32
// wave reductions of the gate, and the gated residual of one row.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tfe_internal.h"

// Cache hints of the streamed rows (tuning knobs): hidden rows in and out
// are touched once (non-temporal); value rows default to the cached path.
#ifndef TFE_NT_HIDDEN_LOAD
#define TFE_NT_HIDDEN_LOAD 1
#endif
#ifndef TFE_NT_OUT_STORE
#define TFE_NT_OUT_STORE 1
#endif
#ifndef TFE_NT_VALUE_LOAD
#define TFE_NT_VALUE_LOAD 0
#endif

namespace tfe {
namespace dev {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ u32x4 load_hidden(const u32x4* p) {
#if TFE_NT_HIDDEN_LOAD
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

__device__ __forceinline__ u32x4 load_value(const u32x4* p) {
#if TFE_NT_VALUE_LOAD
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}

__device__ __forceinline__ void store_out(u32x4 v, u32x4* p) {
#if TFE_NT_OUT_STORE
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

// Elements of type DT held by one 16-byte vector.
template <int DT> struct Vec;
template <> struct Vec<0> { static constexpr int N = 4; };  // float32
template <> struct Vec<1> { static constexpr int N = 8; };  // bfloat16

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two float32 -> two bfloat16 (low half = a), nearest even: one
// v_cvt_pk_bf16_f32 on gfx950.
__device__ __forceinline__ uint32_t to_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
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
    for (int i = 0; i < 4; ++i) v[i] = to_bf16x2(f[2 * i], f[2 * i + 1]);
  }
  return v;
}

// Sum over the 64 lanes of a wavefront, returned as a wave-uniform value.
// DPP row operations reduce each 16-lane row (quad swaps, then half-row and
// row mirrors); the four row sums are read out and added in a fixed order,
// so the result is deterministic.
template <int CTRL>
__device__ __forceinline__ float dpp_add(float x) {
  return x + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF,
                                                        false));
}

__device__ __forceinline__ float wave_sum(float x) {
  x = dpp_add<0xB1>(x);   // quad_perm [1,0,3,2]
  x = dpp_add<0x4E>(x);   // quad_perm [2,3,0,1]
  x = dpp_add<0x141>(x);  // row_half_mirror
  x = dpp_add<0x140>(x);  // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return (r0 + r1) + (r2 + r3);
}

__device__ __forceinline__ bool tok_ok(int32_t t, int32_t vocab) {
  return t >= 0 && t < vocab;
}

// Window tokens of position p (wave-uniform), newest first (t[0] = column
// c); columns before 0 and positions beyond T read as -1 (invalid).
__device__ __forceinline__ void window_tokens(const LookupArgs& a, uint32_t p, int32_t* t) {
  t[0] = t[1] = t[2] = t[3] = -1;
  if (p >= a.T) return;
  const uint32_t b = p / (uint32_t)a.S;
  const int32_t c = a.ctx + (int32_t)(p - b * (uint32_t)a.S);
  // The token ids are never written during a launch: reading them through the
  // constant address space lets wave-uniform reads use scalar loads, whose
  // wait counter is separate from the vector loads in flight.
  const __attribute__((address_space(4))) int32_t* row =
      (const __attribute__((address_space(4))) int32_t*)(a.tokens + (size_t)b * (uint32_t)a.W);
  t[0] = row[c];
  if (c >= 1) t[1] = row[c - 1];
  if (c >= 2) t[2] = row[c - 2];
  if (c >= 3) t[3] = row[c - 3];
}

// Longest-match probe of one position.  Lane group j = lane >> 3 (j < 3)
// holds the key of the n-gram of length n_max - j ending at the position, and
// lane q = lane & 7 reads slot q of the key's current bucket (8 slots = 128
// bytes, one 16-byte load per lane).
struct Probe {
  uint64_t key;
  uint32_t ext;
  uint64_t bucket;
  bool active;
  u32x4 slot;  // the slot this lane read
};

// Forms the keys from the window tokens t (newest first) and issues the
// first bucket read.  Lanes without a key read bucket 0 (one shared, cached
// line), which keeps the read unconditional.
__device__ __forceinline__ Probe probe_begin(const LookupArgs& a, const int32_t* t, int lane) {
  const int j = lane >> 3;
  const int n = a.n_max - j;
  Probe pr;
  pr.active = j < 3 && n >= a.n_min && tok_ok(t[0], a.vocab) && tok_ok(t[1], a.vocab) &&
              (n < 3 || tok_ok(t[2], a.vocab)) && (n < 4 || tok_ok(t[3], a.vocab));
  pr.key = tfe_key(n, (uint32_t)t[0], (uint32_t)t[1], n >= 3 ? (uint32_t)t[2] : 0u);
  pr.ext = n == 4 ? (uint32_t)t[3] : 0u;
  pr.bucket = pr.active ? (tfe_hash(pr.key, pr.ext) & a.bucket_mask) : 0;
  pr.slot = *(const u32x4*)(a.slots + pr.bucket * TFE_SLOTS_PER_BUCKET + (lane & 7));
  return pr;
}

// Outcome of a probe: bit l of `found` is set where lane l read the slot of
// its group's key (at most one lane per group), and `myrow` is the row id in
// that slot (meaningful in the lanes whose bit is set).
struct Walk {
  uint64_t found;
  int32_t myrow;
};

// Consumes the bucket reads: a key group stops at its key (a match) or at an
// empty slot (absent), and otherwise walks on to the next bucket.
__device__ __forceinline__ Walk probe_walk(const LookupArgs& a, const Probe& pr, int lane) {
  bool matched = false;
  bool active = pr.active;
  int32_t myrow = -1;
  const uint64_t grp = 0xFFull << (lane & ~7);
  auto round = [&](const u32x4 sl) {
    const uint64_t sk = (uint64_t)sl[0] | ((uint64_t)sl[1] << 32);
    const bool match = active && sk == pr.key && sl[2] == pr.ext;
    const bool empty = active && sk == TFE_EMPTY_KEY;
    matched = matched || match;
    myrow = match ? (int32_t)sl[3] : myrow;
    const uint64_t done = __builtin_amdgcn_ballot_w64(match) | __builtin_amdgcn_ballot_w64(empty);
    active = active && (done & grp) == 0;
  };
  round(pr.slot);
  // Walks past a full bucket (rare at load factor 1/2): each round advances
  // every unfinished group by one bucket; a load factor below 1 leaves empty
  // slots, and the bucket count bounds the walk in any case.
  uint64_t bucket = pr.bucket;
  for (uint64_t it = 0; it < a.bucket_mask && __builtin_amdgcn_ballot_w64(active); ++it) {
    bucket = (bucket + 1) & a.bucket_mask;
    round(*(const u32x4*)(a.slots + bucket * TFE_SLOTS_PER_BUCKET + (lane & 7)));
  }
  return Walk{__builtin_amdgcn_ballot_w64(matched), myrow};
}

// Longest match: the phrase row (-1 on a miss) in every lane and its length
// in *len; the longest match is the lowest matching lane group.
__device__ __forceinline__ int32_t probe_finish(const LookupArgs& a, const Probe& pr, int lane,
                                                int* len) {
  const Walk w = probe_walk(a, pr, lane);
  if (w.found == 0) {
    *len = 0;
    return -1;
  }
  const int sel = __builtin_amdgcn_readfirstlane(__builtin_ctzll(w.found));
  *len = a.n_max - (sel >> 3);
  return __builtin_amdgcn_readlane(w.myrow, sel);
}

// Exact-match probe of one key by one thread (no cross-lane work): the
// key's home bucket is read whole (8 slots of 16 bytes, all in flight), then
// the following buckets while the key is neither found nor ruled out by an
// empty slot.  Returns the row, or -1 when the key is absent.  Used where one
// thread handles a whole window (the single-block prefetch).
__device__ __forceinline__ int32_t probe_key_thread(const LookupArgs& a, uint64_t key,
                                                    uint32_t ext) {
  uint64_t b = tfe_hash(key, ext) & a.bucket_mask;
  for (uint64_t it = 0; it <= a.bucket_mask; ++it) {
    u32x4 sl[TFE_SLOTS_PER_BUCKET];
    const u32x4* bp = (const u32x4*)(a.slots + b * TFE_SLOTS_PER_BUCKET);
#pragma unroll
    for (int i = 0; i < TFE_SLOTS_PER_BUCKET; ++i) sl[i] = bp[i];
    bool empty = false;
    int32_t row = -1;
#pragma unroll
    for (int i = 0; i < TFE_SLOTS_PER_BUCKET; ++i) {
      const uint64_t sk = (uint64_t)sl[i][0] | ((uint64_t)sl[i][1] << 32);
      if (sk == key && sl[i][2] == ext) row = (int32_t)sl[i][3];
      empty = empty || sk == TFE_EMPTY_KEY;
    }
    if (row >= 0 || empty) return row;
    b = (b + 1) & a.bucket_mask;
  }
  return -1;
}

// The key and extension word of the n-gram of window t (newest first) and
// whether the window holds n valid tokens.
__device__ __forceinline__ bool window_key(const LookupArgs& a, const int32_t* t, int n,
                                           uint64_t* key, uint32_t* ext) {
  const bool ok = tok_ok(t[0], a.vocab) && tok_ok(t[1], a.vocab) &&
                  (n < 3 || tok_ok(t[2], a.vocab)) && (n < 4 || tok_ok(t[3], a.vocab));
  *key = tfe_key(n, (uint32_t)t[0], (uint32_t)t[1], n >= 3 ? (uint32_t)t[2] : 0u);
  *ext = n == 4 ? (uint32_t)t[3] : 0u;
  return ok;
}

// Gate of Eq. 5 from this lane's partial sums of h.h, m.m and h.m.
__device__ __forceinline__ float gate_finish(const LookupArgs& a, float shh, float smm,
                                             float shm) {
  shh = wave_sum(shh);
  smm = wave_sum(smm);
  shm = wave_sum(shm);
  const float inv_rh = __builtin_amdgcn_rsqf(fmaf(shh, a.inv_d, 1e-6f));
  const float inv_rm = __builtin_amdgcn_rsqf(fmaf(smm, a.inv_d, 1e-6f));
  const float z = shm * inv_rh * inv_rm * a.inv_sqrt_d;
  return a.scale * __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

// Gate of Eq. 5 for one row held across the wave (hv, mv: NCH 16-byte
// vectors per lane).  Sigmoid gate: scale * sigmoid(<h/rms_h, m/rms_m> /
// sqrt(D)), rms_x = sqrt(mean(x^2) + 1e-6), from three fp32 wave sums; the
// reciprocal square roots, exponential and reciprocal use the hardware
// approximations (about 1 ulp each).
template <int DT, int NCH>
__device__ __forceinline__ float gate_of(const LookupArgs& a, const u32x4* hv, const u32x4* mv) {
  if (a.gate != TFE_GATE_SIGMOID) return a.scale;
  constexpr int VN = Vec<DT>::N;
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
  return gate_finish(a, shh, smm, shm);
}

// h' = h + g m for one row, rounded to nearest even, stored non-temporally.
template <int DT, int NCH>
__device__ __forceinline__ void store_injected(u32x4* out, const u32x4* hv, const u32x4* mv,
                                               float g, int lane) {
  constexpr int VN = Vec<DT>::N;
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    float h[VN], m[VN], o[VN];
    unpack<DT>(hv[k], h);
    unpack<DT>(mv[k], m);
#pragma unroll
    for (int i = 0; i < VN; ++i) o[i] = fmaf(g, m[i], h[i]);
    store_out(pack<DT>(o), out + k * 64 + lane);
  }
}

__device__ __forceinline__ void write_result(const LookupArgs& a, uint32_t p, int32_t row,
                                             int len) {
  a.hit[p] = row >= 0 ? 1 : 0;
  a.slot_out[p] = row;
  if (a.len_out) a.len_out[p] = (uint8_t)len;
}

// Resident tables: one matched position added to the table's hit count
// (called by one lane of the position's wave, right after the probe; an
// addition after the value row's loads, or after the stores, measured
// slower).  The counter is picked by block, spreading a launch's additions.
__device__ __forceinline__ void count_hit(const LookupArgs& a, bool matched) {
  if (a.hit_ctr && matched)
    __hip_atomic_fetch_add(a.hit_ctr + (blockIdx.x & (kHitCounters - 1)) * kHitStride, 1ull,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace dev
}  // namespace tfe
