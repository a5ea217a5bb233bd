// Host side of libtfe: the error message, the allocation-failure hook and
// the held-memory count, and the phrase index (validation, capacity, build
// and a host probe).  Nothing here calls the HIP runtime.
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <chrono>
#include <mutex>
#include <thread>
#include <unordered_map>
#include <vector>

#include "../../include/tfe.h"
#include "tfe_index.h"
#include "tfe_internal.h"

namespace tfe {

static thread_local char g_err[512] = "";
// Allocations made so far by the current library call on this thread.
static thread_local int64_t g_allocs_in_call = 0;

tfe_status fail(tfe_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return st;
}

void clear_error() {
  g_err[0] = 0;
  g_allocs_in_call = 0;
}

const char* last_error() { return g_err; }

bool alloc_fails() {
  const int64_t k = ++g_allocs_in_call;
  const char* s = getenv("TFE_FAIL_ALLOC");
  if (!s || !*s) return false;
  return strtoll(s, nullptr, 10) == k;
}

namespace {
struct Held {
  std::mutex mu;
  std::unordered_map<const void*, std::pair<size_t, bool>> live;  // size, pinned
  int64_t bytes[2] = {0, 0};                                      // device, pinned
};
Held& held() {
  static Held* h = new Held;  // never destroyed: tables may outlive static teardown
  return *h;
}
}  // namespace

void note_alloc(const void* p, size_t n, bool pinned) {
  if (!p) return;
  Held& h = held();
  std::lock_guard<std::mutex> g(h.mu);
  h.live[p] = {n, pinned};
  h.bytes[pinned] += (int64_t)n;
}

void note_free(const void* p) {
  if (!p) return;
  Held& h = held();
  std::lock_guard<std::mutex> g(h.mu);
  auto it = h.live.find(p);
  if (it == h.live.end()) return;
  h.bytes[it->second.second] -= (int64_t)it->second.first;
  h.live.erase(it);
}

// A thread spins while requests keep coming and sleeps briefly once it has
// been idle for a while; the first request after a quiet period therefore
// waits up to about a tenth of a millisecond.
void stage_serve(StageSlot* q, char* rows, const char* pageable, int64_t first_row,
                 int64_t n_rows, size_t row_bytes, uint64_t first, uint64_t step,
                 const volatile bool* stop) {
  using clock = std::chrono::steady_clock;
  constexpr auto kSpin = std::chrono::milliseconds(2);
  uint64_t tk = first;
  auto last = clock::now();
  while (!__atomic_load_n(stop, __ATOMIC_ACQUIRE)) {
    StageSlot& slot = q[tk % kStageSlots];
    const unsigned long long r = __atomic_load_n(&slot.req, __ATOMIC_ACQUIRE);
    if ((r >> 32) != ((tk + 1) & 0xFFFFFFFFull)) {
      if (clock::now() - last < kSpin)
        __builtin_ia32_pause();
      else
        std::this_thread::sleep_for(std::chrono::microseconds(20));
      continue;
    }
    const int64_t i = (int64_t)(int32_t)(uint32_t)r - first_row;
    char* dst = rows + (tk % kStageSlots) * row_bytes;
    if (i >= 0 && i < n_rows)
      memcpy(dst, pageable + i * (int64_t)row_bytes, row_bytes);
    else
      memset(dst, 0, row_bytes);
    // The row's stores (memcpy may use non-temporal ones) are visible
    // before the slot is marked done.
    std::atomic_thread_fence(std::memory_order_seq_cst);
    __atomic_store_n(&slot.done, tk + 1, __ATOMIC_RELEASE);
    tk += step;
    last = clock::now();
  }
}

void memory_held(int64_t* device_bytes, int64_t* pinned_bytes) {
  Held& h = held();
  std::lock_guard<std::mutex> g(h.mu);
  if (device_bytes) *device_bytes = h.bytes[0];
  if (pinned_bytes) *pinned_bytes = h.bytes[1];
}

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

// Runs fn(begin, end) over [0, n) on up to `threads` host threads.
template <class F>
static void parallel_ranges(int64_t n, F fn) {
  unsigned hw = std::thread::hardware_concurrency();
  int64_t threads = hw ? (int64_t)hw : 1;
  if (threads > 32) threads = 32;
  const int64_t min_per_thread = 1 << 16;
  if (threads > n / min_per_thread) threads = n / min_per_thread;
  if (threads <= 1) {
    fn((int64_t)0, n);
    return;
  }
  std::vector<std::thread> pool;
  for (int64_t i = 0; i < threads; ++i)
    pool.emplace_back(fn, n * i / threads, n * (i + 1) / threads);
  for (auto& th : pool) th.join();
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
  // First bad phrase (lowest index) wins, so the message does not depend on
  // the thread schedule.
  std::atomic<int64_t> first_bad(P);
  parallel_ranges(P, [&](int64_t a, int64_t b) {
    for (int64_t i = a; i < b && i < first_bad.load(std::memory_order_relaxed); ++i) {
      const int n = lens[i];
      bool bad = n < n_min || n > n_max;
      for (int j = 0; j < n && !bad; ++j) {
        const int32_t x = tokens[i * n_max + j];
        bad = x < 0 || x >= vocab;
      }
      if (bad) {
        int64_t cur = first_bad.load();
        while (i < cur && !first_bad.compare_exchange_weak(cur, i)) {
        }
        return;
      }
    }
  });
  const int64_t i = first_bad.load();
  if (i < P) {
    const int n = lens[i];
    if (n < n_min || n > n_max)
      return fail(TFE_ERR_INVALID_ARG, "phrase %lld has length %d outside [%d, %d]",
                  (long long)i, n, n_min, n_max);
    return fail(TFE_ERR_INVALID_ARG, "phrase %lld has a token outside [0, %d)", (long long)i,
                vocab);
  }
  return TFE_OK;
}

// Inserts the phrases from several host threads.  A slot is claimed by a
// compare-and-swap of its key from empty; its extension word and row follow,
// the row last (release), so a thread that meets an equal key waits for the
// row before it compares the extension.  Within a bucket the claimed slots
// stay a prefix, so a lookup may still stop at the first empty slot.  Which
// slot a phrase lands in depends on the schedule; what a lookup returns does
// not.
tfe_status build_index(const int32_t* tokens, const uint8_t* lens, int64_t P, int n_max,
                       tfe_slot* slots, int64_t cap) {
  if (cap < TFE_SLOTS_PER_BUCKET || (cap & (cap - 1)) != 0)
    return fail(TFE_ERR_INVALID_ARG, "capacity must be a power of two >= 8");
  if (P >= cap) return fail(TFE_ERR_INVALID_ARG, "capacity %lld too small for %lld phrases",
                            (long long)cap, (long long)P);
  parallel_ranges(cap, [&](int64_t a, int64_t b) {
    for (int64_t s = a; s < b; ++s) {
      slots[s].key = TFE_EMPTY_KEY;
      slots[s].key_ext = 0;
      slots[s].row = -1;
    }
  });
  const int64_t nb = cap / TFE_SLOTS_PER_BUCKET;
  std::atomic<int64_t> dup_row(-1), dup_of(-1);
  parallel_ranges(P, [&](int64_t a, int64_t b) {
    for (int64_t i = a; i < b && dup_row.load(std::memory_order_relaxed) < 0; ++i) {
      uint64_t key;
      uint32_t ext;
      phrase_key(tokens + i * n_max, lens[i], &key, &ext);
      int64_t bk = (int64_t)(tfe_hash(key, ext) & (uint64_t)(nb - 1));
      bool placed = false;
      while (!placed) {
        tfe_slot* s = slots + bk * TFE_SLOTS_PER_BUCKET;
        for (int q = 0; q < TFE_SLOTS_PER_BUCKET && !placed; ++q) {
          uint64_t k = __atomic_load_n(&s[q].key, __ATOMIC_ACQUIRE);
          if (k == TFE_EMPTY_KEY) {
            uint64_t expected = TFE_EMPTY_KEY;
            if (__atomic_compare_exchange_n(&s[q].key, &expected, key, false, __ATOMIC_ACQ_REL,
                                            __ATOMIC_ACQUIRE)) {
              __atomic_store_n(&s[q].key_ext, ext, __ATOMIC_RELAXED);
              __atomic_store_n(&s[q].row, (int32_t)i, __ATOMIC_RELEASE);
              placed = true;
              break;
            }
            k = expected;
          }
          if (k == key) {
            int32_t other;
            while ((other = __atomic_load_n(&s[q].row, __ATOMIC_ACQUIRE)) < 0) {
            }
            if (__atomic_load_n(&s[q].key_ext, __ATOMIC_RELAXED) == ext) {
              int64_t none = -1;
              if (dup_row.compare_exchange_strong(none, i)) dup_of.store(other);
              return;
            }
          }
        }
        bk = (bk + 1) & (nb - 1);
      }
    }
  });
  if (dup_row.load() >= 0) {
    const int64_t x = dup_row.load(), y = dup_of.load();
    return fail(TFE_ERR_DUPLICATE_KEY, "phrases %lld and %lld are the same", (long long)(x < y ? x : y),
                (long long)(x < y ? y : x));
  }
  return TFE_OK;
}

}  // namespace tfe

extern "C" {

const char* tfe_last_error(void) { return tfe::last_error(); }

tfe_status tfe_memory_held(int64_t* device_bytes, int64_t* pinned_bytes) {
  tfe::clear_error();
  if (!device_bytes && !pinned_bytes) return tfe::fail(TFE_ERR_INVALID_ARG, "no output");
  tfe::memory_held(device_bytes, pinned_bytes);
  return TFE_OK;
}

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
