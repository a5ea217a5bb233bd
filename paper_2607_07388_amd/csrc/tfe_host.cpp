// Host side of the phrase index: validation, capacity, build and a host probe.
#include <stdint.h>
#include <string.h>

#include "../../include/tfe.h"
#include "tfe_index.h"
#include "tfe_internal.h"

namespace tfe {

int64_t index_capacity(int64_t n, double lf) {
  if (lf <= 0.0) lf = 0.5;
  const double need = (double)n / lf;
  int64_t cap = TFE_SLOTS_PER_BUCKET;
  while ((double)cap < need) cap <<= 1;
  return cap;
}

// Key of phrase tokens w[0..n-1] (oldest first).
static inline void phrase_key(const int32_t* w, int n, uint64_t* key, uint32_t* ext) {
  const uint32_t t0 = (uint32_t)w[n - 1];
  const uint32_t t1 = (uint32_t)w[n - 2];
  const uint32_t t2 = n >= 3 ? (uint32_t)w[n - 3] : 0u;
  *key = tfe_key(n, t0, t1, t2);
  *ext = n == 4 ? (uint32_t)w[0] : 0u;
}

tfe_status validate_phrases(const int32_t* tokens, const uint8_t* lens, int64_t P, int n_min,
                            int n_max, int vocab) {
  if (P < 0) return fail(TFE_ERR_INVALID_ARG, "n_phrases < 0");
  if (n_min < 2 || n_max > 4 || n_min > n_max)
    return fail(TFE_ERR_INVALID_ARG, "need 2 <= n_min <= n_max <= 4");
  if (vocab <= 0 || vocab > (1 << TFE_TOKEN_BITS))
    return fail(TFE_ERR_INVALID_ARG, "vocab must be in [1, 2^18]");
  if (P > 0x7FFFFFFFll) return fail(TFE_ERR_UNSUPPORTED, "more than 2^31-1 phrases");
  if (P > 0 && (!tokens || !lens)) return fail(TFE_ERR_INVALID_ARG, "null phrase arrays");
  for (int64_t i = 0; i < P; ++i) {
    const int n = lens[i];
    if (n < n_min || n > n_max)
      return fail(TFE_ERR_INVALID_ARG, "phrase %lld has length %d outside [%d, %d]",
                  (long long)i, n, n_min, n_max);
    const int32_t* w = tokens + i * n_max;
    for (int j = 0; j < n; ++j)
      if (w[j] < 0 || w[j] >= vocab)
        return fail(TFE_ERR_INVALID_ARG, "phrase %lld token %d = %d outside [0, %d)",
                    (long long)i, j, w[j], vocab);
  }
  return TFE_OK;
}

tfe_status build_index(const int32_t* tokens, const uint8_t* lens, int64_t P, int n_max,
                       tfe_slot* slots, int64_t cap) {
  if (cap < TFE_SLOTS_PER_BUCKET || (cap & (cap - 1)) != 0)
    return fail(TFE_ERR_INVALID_ARG, "capacity must be a power of two >= 8");
  if (P >= cap) return fail(TFE_ERR_INVALID_ARG, "capacity %lld too small for %lld phrases",
                            (long long)cap, (long long)P);
  for (int64_t s = 0; s < cap; ++s) {
    slots[s].key = TFE_EMPTY_KEY;
    slots[s].key_ext = 0;
    slots[s].row = -1;
  }
  const int64_t nb = cap / TFE_SLOTS_PER_BUCKET;
  for (int64_t i = 0; i < P; ++i) {
    uint64_t key;
    uint32_t ext;
    phrase_key(tokens + i * n_max, lens[i], &key, &ext);
    int64_t b = (int64_t)(tfe_hash(key, ext) & (uint64_t)(nb - 1));
    for (;;) {
      tfe_slot* bk = slots + b * TFE_SLOTS_PER_BUCKET;
      int free_at = -1;
      for (int q = 0; q < TFE_SLOTS_PER_BUCKET; ++q) {
        if (bk[q].key == TFE_EMPTY_KEY) { free_at = q; break; }
        if (bk[q].key == key && bk[q].key_ext == ext)
          return fail(TFE_ERR_DUPLICATE_KEY, "phrase %lld repeats phrase %d", (long long)i,
                      bk[q].row);
      }
      if (free_at >= 0) {
        bk[free_at].key = key;
        bk[free_at].key_ext = ext;
        bk[free_at].row = (int32_t)i;
        break;
      }
      b = (b + 1) & (nb - 1);
    }
  }
  return TFE_OK;
}

}  // namespace tfe

extern "C" {

int64_t tfe_index_capacity(int64_t n_phrases, double max_load_factor) {
  if (n_phrases < 0 || max_load_factor < 0.0 || max_load_factor > 0.9) return -1;
  return tfe::index_capacity(n_phrases, max_load_factor);
}

tfe_status tfe_index_build_host(const int32_t* phrase_tokens, const uint8_t* phrase_len,
                                int64_t n_phrases, int32_t n_min, int32_t n_max, int32_t vocab,
                                void* slots, int64_t capacity) {
  tfe::clear_error();
  tfe_status st = tfe::validate_phrases(phrase_tokens, phrase_len, n_phrases, n_min, n_max, vocab);
  if (st != TFE_OK) return st;
  if (!slots) return tfe::fail(TFE_ERR_INVALID_ARG, "null slots");
  return tfe::build_index(phrase_tokens, phrase_len, n_phrases, n_max, (tfe_slot*)slots, capacity);
}

tfe_status tfe_index_probe_host(const void* slots, int64_t capacity, const int32_t* tokens,
                                int32_t n, int32_t* row, int32_t* buckets_read, int64_t* home) {
  tfe::clear_error();
  if (!slots || !tokens || !row || n < 2 || n > 4 || capacity < TFE_SLOTS_PER_BUCKET ||
      (capacity & (capacity - 1)) != 0)
    return tfe::fail(TFE_ERR_INVALID_ARG, "bad probe arguments");
  uint64_t key;
  uint32_t ext;
  tfe::phrase_key(tokens, n, &key, &ext);
  const int64_t nb = capacity / TFE_SLOTS_PER_BUCKET;
  int64_t b = (int64_t)(tfe_hash(key, ext) & (uint64_t)(nb - 1));
  if (home) *home = b;
  const tfe_slot* s = (const tfe_slot*)slots;
  *row = -1;
  int32_t nread = 0;
  for (int64_t it = 0; it < nb; ++it) {
    const tfe_slot* bk = s + b * TFE_SLOTS_PER_BUCKET;
    ++nread;
    bool empty = false;
    for (int q = 0; q < TFE_SLOTS_PER_BUCKET; ++q) {
      if (bk[q].key == key && bk[q].key_ext == ext) *row = bk[q].row;
      if (bk[q].key == TFE_EMPTY_KEY) empty = true;
    }
    if (*row >= 0 || empty) break;
    b = (b + 1) & (nb - 1);
  }
  if (buckets_read) *buckets_read = nread;
  return TFE_OK;
}

}  // extern "C"
