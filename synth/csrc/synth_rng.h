// Counter-based random numbers for the seeded synthetic workloads.
//
// This header belongs to the input generator only.  It holds no part of the
// phrase-memory method: it turns (seed, stream tag, element index) into bits,
// and both the host build (synth_host.cpp) and the device build
// (synth_dev.hip) of the generator include it so that a value drawn on the GPU
// has exactly the same bits as the same value drawn on the CPU.
//
// Definitions (all arithmetic modulo 2^64):
//   mix(x)      SplitMix64 output function (S. Vigna, "SplitMix64", public
//               domain): x ^= x>>30; x *= 0xBF58476D1CE4E5B9;
//               x ^= x>>27; x *= 0x94D049BB133111EB; x ^= x>>31.
//   draw(k, i)  i-th output of a SplitMix64 generator whose state starts at k:
//               mix(k + (i+1) * 0x9E3779B97F4A7C15).
//   key(s, t)   stream key for seed s and tag t: draw(s, t).
//   normal(k,e) Irwin-Hall(12) approximation of N(0,1) for element e: the
//               twelve 16-bit fields of draw(k,3e), draw(k,3e+1), draw(k,3e+2)
//               are summed as integers, giving N = sum - 393210, which equals
//               65536 * (sum_j (u_j + 1/2)/65536 - 6).  The float result is
//               float(N) * scale with scale = float32(sigma / 65536): one exact
//               int->float conversion and one IEEE multiply, so it is
//               bit-identical on every IEEE machine.
#pragma once
#include <stdint.h>

#if defined(__HIPCC__)
#define SYNTH_FN __host__ __device__ static inline
#else
#define SYNTH_FN static inline
#endif

#define SYNTH_GAMMA 0x9E3779B97F4A7C15ull

SYNTH_FN uint64_t synth_mix(uint64_t x) {
  x ^= x >> 30;
  x *= 0xBF58476D1CE4E5B9ull;
  x ^= x >> 27;
  x *= 0x94D049BB133111EBull;
  x ^= x >> 31;
  return x;
}

SYNTH_FN uint64_t synth_draw(uint64_t k, uint64_t i) {
  return synth_mix(k + (i + 1) * SYNTH_GAMMA);
}

SYNTH_FN uint64_t synth_key(uint64_t seed, uint64_t tag) { return synth_draw(seed, tag); }

SYNTH_FN int32_t synth_irwin_hall_n(uint64_t k, uint64_t e) {
  int32_t s = 0;
  for (int d = 0; d < 3; ++d) {
    uint64_t w = synth_draw(k, 3 * e + (uint64_t)d);
    s += (int32_t)(w & 0xFFFF) + (int32_t)((w >> 16) & 0xFFFF) +
         (int32_t)((w >> 32) & 0xFFFF) + (int32_t)(w >> 48);
  }
  return s - 393210;
}

// Round a float to bfloat16, nearest-even (inputs here are finite).
SYNTH_FN uint16_t synth_f32_to_bf16(float f) {
  union { float f; uint32_t u; } v;
  v.f = f;
  uint32_t u = v.u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
