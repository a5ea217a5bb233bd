// Phrase index layout shared by the host index builder and the device probe.
//
// An exact-match phrase index (first level of the paper's two-level index,
// Eq. 10): each stored phrase owns one 16-byte slot holding its full key and
// its row id, so distinct phrases never share a slot (Sec. 4.1, 4.2) and a
// lookup compares full keys, never hashes.
//
// Slots are grouped in buckets of 8 (128 bytes, one L2 line on gfx950); a
// bucket is read by 8 lanes of a wavefront with one 16-byte load each.
#pragma once
#include <stdint.h>

#if defined(__HIPCC__)
#define TFE_HD __host__ __device__ static inline
#else
#define TFE_HD static inline
#endif

#define TFE_SLOTS_PER_BUCKET 8
#define TFE_EMPTY_KEY 0xFFFFFFFFFFFFFFFFull
#define TFE_TOKEN_BITS 18

struct alignas(16) tfe_slot {
  uint64_t key;     // n << 61 | up to three newest tokens, 18 bits each
  uint32_t key_ext; // oldest token of a 4-gram, 0 otherwise
  int32_t row;      // phrase row id
};

// Key of the n-gram x[0..n-1] (oldest first) given as its newest tokens:
// t0 = x[n-1] (newest), t1 = x[n-2], t2 = x[n-3], t3 = x[n-4] (absent = 0).
TFE_HD uint64_t tfe_key(int n, uint32_t t0, uint32_t t1, uint32_t t2) {
  return ((uint64_t)n << 61) | ((uint64_t)t2 << (2 * TFE_TOKEN_BITS)) |
         ((uint64_t)t1 << TFE_TOKEN_BITS) | (uint64_t)t0;
}

// murmur3 fmix64 finalizer (A. Appleby, public domain) of the key pair.
TFE_HD uint64_t tfe_hash(uint64_t key, uint32_t ext) {
  uint64_t h = key ^ ((uint64_t)ext * 0x9E3779B97F4A7C15ull);
  h ^= h >> 33;
  h *= 0xFF51AFD7ED558CCDull;
  h ^= h >> 33;
  h *= 0xC4CEB9FE1A85EC53ull;
  h ^= h >> 33;
  return h;
}
