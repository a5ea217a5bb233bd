// Drives the host half of libtfe (tfe_host.cpp: error messages, the
// allocation-failure hook, the held-memory count, phrase validation and the
// multi-threaded index build) so that it can run under AddressSanitizer,
// UndefinedBehaviorSanitizer and ThreadSanitizer without a GPU.
//
// Exit status 0 and a final "ok" line when every check holds; otherwise the
// first failed check is printed and the status is 1.  A sanitizer report
// ends the process on its own (the test builds with -fno-sanitize-recover).
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <string>
#include <thread>
#include <vector>

#include "tfe.h"
#include "tfe_internal.h"

#define CHECK(c)                                                     \
  do {                                                               \
    if (!(c)) {                                                      \
      fprintf(stderr, "check failed at line %d: %s (last error: %s)\n", \
              __LINE__, #c, tfe_last_error());                       \
      exit(1);                                                       \
    }                                                                \
  } while (0)

static const int V = 1 << 18;
static const int NMAX = 4;

// Phrase i of a set of distinct phrases: length 2 + i % 3, newest token
// i % V, the one before it i / V (so the pair, with the length, names i),
// the rest from a mixing function of i.
static void make_phrase(int64_t i, int32_t* w, uint8_t* len) {
  const int n = 2 + (int)(i % 3);
  uint64_t x = (uint64_t)i * 0x9E3779B97F4A7C15ull + 1;
  for (int j = 0; j < NMAX; ++j) {
    x ^= x >> 29;
    x *= 0xBF58476D1CE4E5B9ull;
    w[j] = j < n ? (int32_t)(x % V) : -1;
  }
  w[n - 1] = (int32_t)(i % V);
  w[n - 2] = (int32_t)(i / V);
  *len = (uint8_t)n;
}

struct Phrases {
  std::vector<int32_t> tok;
  std::vector<uint8_t> len;
  explicit Phrases(int64_t P) : tok((size_t)P * NMAX), len((size_t)P) {
    for (int64_t i = 0; i < P; ++i) make_phrase(i, &tok[(size_t)i * NMAX], &len[(size_t)i]);
  }
};

static void build_and_probe_all(int64_t P) {
  Phrases ph(P);
  const int64_t cap = tfe_index_capacity(P, 0.5);
  CHECK(cap >= 2 * P && (cap & (cap - 1)) == 0);
  std::vector<tfe_slot> slots((size_t)cap);
  CHECK(tfe_index_build_host(ph.tok.data(), ph.len.data(), P, 2, 4, V, slots.data(), cap) ==
        TFE_OK);
  int64_t used = 0;
  for (const tfe_slot& s : slots) used += s.key != TFE_EMPTY_KEY;
  CHECK(used == P);
  for (int64_t i = 0; i < P; ++i) {
    int32_t row = -2, nread = 0;
    int64_t home = -1;
    CHECK(tfe_index_probe_host(slots.data(), cap, &ph.tok[(size_t)i * NMAX], ph.len[(size_t)i],
                               &row, &nread, &home) == TFE_OK);
    CHECK(row == i && nread >= 1 && home >= 0 && home < cap / 8);
  }
  // Absent: the same newest pair under another length names no phrase.
  for (int64_t i = 0; i < 1000; ++i) {
    int32_t w[4];
    uint8_t n;
    make_phrase(i, w, &n);
    const int n2 = n == 4 ? 2 : n + 1;
    int32_t x[4] = {7, 7, 7, 7};
    x[n2 - 1] = w[n - 1];
    x[n2 - 2] = w[n - 2];
    int32_t row = -2, nread = 0;
    CHECK(tfe_index_probe_host(slots.data(), cap, x, n2, &row, &nread, nullptr) == TFE_OK);
    CHECK(row == -1 || (row % 3) + 2 == n2);
  }
}

static void validation_errors() {
  Phrases ph(1 << 18);
  const int64_t P = 1 << 18;
  const int64_t cap = tfe_index_capacity(P, 0.5);
  std::vector<tfe_slot> slots((size_t)cap);
  CHECK(tfe_index_build_host(ph.tok.data(), ph.len.data(), -1, 2, 4, V, slots.data(), cap) ==
        TFE_ERR_INVALID_ARG);
  CHECK(tfe_index_build_host(ph.tok.data(), ph.len.data(), P, 1, 4, V, slots.data(), cap) ==
        TFE_ERR_INVALID_ARG);
  CHECK(tfe_index_build_host(ph.tok.data(), ph.len.data(), P, 3, 2, V, slots.data(), cap) ==
        TFE_ERR_INVALID_ARG);
  CHECK(tfe_index_build_host(ph.tok.data(), ph.len.data(), P, 2, 4, V + 1, slots.data(), cap) ==
        TFE_ERR_INVALID_ARG);
  CHECK(tfe_index_build_host(nullptr, ph.len.data(), P, 2, 4, V, slots.data(), cap) ==
        TFE_ERR_INVALID_ARG);
  CHECK(tfe_index_build_host(ph.tok.data(), ph.len.data(), P, 2, 4, V, nullptr, cap) ==
        TFE_ERR_INVALID_ARG);
  CHECK(tfe_index_build_host(ph.tok.data(), ph.len.data(), P, 2, 4, V, slots.data(), cap / 2 + 3) ==
        TFE_ERR_INVALID_ARG);
  CHECK(tfe_index_build_host(ph.tok.data(), ph.len.data(), P, 2, 4, V, slots.data(), 8) ==
        TFE_ERR_INVALID_ARG);
  // Bad phrases in several threads' ranges: the lowest index is reported,
  // whatever the schedule.
  std::vector<int32_t> tok = ph.tok;
  std::vector<uint8_t> len = ph.len;
  len[(size_t)P - 5] = 7;
  tok[(size_t)(P / 2) * NMAX] = V;
  tok[(size_t)(P / 3) * NMAX] = -3;
  for (int rep = 0; rep < 4; ++rep) {
    CHECK(tfe_index_build_host(tok.data(), len.data(), P, 2, 4, V, slots.data(), cap) ==
          TFE_ERR_INVALID_ARG);
    const std::string msg = tfe_last_error();
    CHECK(msg.find("phrase " + std::to_string(P / 3) + " ") != std::string::npos);
  }
  len[(size_t)P / 5] = 1;
  CHECK(tfe_index_build_host(tok.data(), len.data(), P, 2, 4, V, slots.data(), cap) ==
        TFE_ERR_INVALID_ARG);
  CHECK(std::string(tfe_last_error()).find("length 1") != std::string::npos);
  // Probe argument errors.
  int32_t row;
  CHECK(tfe_index_probe_host(slots.data(), 12, ph.tok.data(), 2, &row, nullptr, nullptr) ==
        TFE_ERR_INVALID_ARG);
  CHECK(tfe_index_probe_host(slots.data(), cap, ph.tok.data(), 5, &row, nullptr, nullptr) ==
        TFE_ERR_INVALID_ARG);
  CHECK(tfe_index_capacity(10, 0.95) == -1 && tfe_index_capacity(-1, 0.5) == -1);
}

static void duplicates() {
  const int64_t P = 1 << 19;
  // One duplicate pair, far apart.
  Phrases ph(P);
  memcpy(&ph.tok[(size_t)(P - 2) * NMAX], &ph.tok[(size_t)17 * NMAX], NMAX * sizeof(int32_t));
  ph.len[(size_t)P - 2] = ph.len[17];
  const int64_t cap = tfe_index_capacity(P, 0.5);
  std::vector<tfe_slot> slots((size_t)cap);
  CHECK(tfe_index_build_host(ph.tok.data(), ph.len.data(), P, 2, 4, V, slots.data(), cap) ==
        TFE_ERR_DUPLICATE_KEY);
  CHECK(std::string(tfe_last_error()) ==
        "phrases 17 and " + std::to_string(P - 2) + " are the same");
  // Every phrase twice (second half repeats the first): threads meet equal
  // keys concurrently and wait for each other's row publish.
  Phrases half(P / 2);
  std::vector<int32_t> tok((size_t)P * NMAX);
  std::vector<uint8_t> len((size_t)P);
  for (int64_t i = 0; i < P; ++i) {
    const int64_t j = i % (P / 2);
    memcpy(&tok[(size_t)i * NMAX], &half.tok[(size_t)j * NMAX], NMAX * sizeof(int32_t));
    len[(size_t)i] = half.len[(size_t)j];
  }
  for (int rep = 0; rep < 3; ++rep)
    CHECK(tfe_index_build_host(tok.data(), len.data(), P, 2, 4, V, slots.data(), cap) ==
          TFE_ERR_DUPLICATE_KEY);
  // 4-grams that differ only in their oldest token are distinct.
  int32_t t4[3 * NMAX] = {1, 7, 8, 9, 2, 7, 8, 9, 0, 7, 8, 9};
  uint8_t l4[3] = {4, 4, 4};
  std::vector<tfe_slot> s4(8);
  CHECK(tfe_index_build_host(t4, l4, 3, 2, 4, V, s4.data(), 8) == TFE_OK);
}

static void hook_and_held_memory() {
  // The k-th allocation of a call fails; the count restarts with each call.
  setenv("TFE_FAIL_ALLOC", "2", 1);
  tfe::clear_error();
  CHECK(!tfe::alloc_fails());
  CHECK(tfe::alloc_fails());
  CHECK(!tfe::alloc_fails());
  tfe::clear_error();
  CHECK(!tfe::alloc_fails() && tfe::alloc_fails());
  unsetenv("TFE_FAIL_ALLOC");
  tfe::clear_error();
  CHECK(!tfe::alloc_fails() && !tfe::alloc_fails());
  // Held bytes from many threads at once, with the error message of each
  // thread its own.
  int64_t d0 = -1, p0 = -1;
  CHECK(tfe_memory_held(&d0, &p0) == TFE_OK && d0 == 0 && p0 == 0);
  CHECK(tfe_memory_held(nullptr, nullptr) == TFE_ERR_INVALID_ARG);
  std::vector<std::vector<char>> bufs(8, std::vector<char>(4096));
  std::vector<std::thread> pool;
  for (int th = 0; th < 8; ++th)
    pool.emplace_back([th, &bufs] {
      bool live[64] = {};
      for (int r = 0; r < 2000; ++r) {
        const int k = (r * 7) % 64;  // a live address is freed before it is handed out again
        const char* p = bufs[(size_t)th].data() + k;
        if (live[k]) tfe::note_free(p);
        tfe::note_alloc(p, 100 + th, (r & 1) != 0);
        live[k] = true;
        tfe::fail(TFE_ERR_OOM, "thread %d round %d", th, r);
        if (r % 3 == 0) {
          tfe::note_free(p);
          live[k] = false;
        }
        char want[64];
        snprintf(want, sizeof want, "thread %d round %d", th, r);
        if (strcmp(tfe_last_error(), want) != 0) abort();
      }
      for (int k = 0; k < 64; ++k)
        if (live[k]) tfe::note_free(bufs[(size_t)th].data() + k);
    });
  for (auto& t : pool) t.join();
  int64_t d1 = -1, p1 = -1;
  CHECK(tfe_memory_held(&d1, &p1) == TFE_OK && d1 == 0 && p1 == 0);
  tfe::note_free(nullptr);
  tfe::note_free(bufs[0].data());  // unknown pointer: ignored
  CHECK(tfe_memory_held(&d1, nullptr) == TFE_OK && d1 == 0);
}

// The staging queue of pageable rows (StageSlot, stage_serve) with emulated
// requesters following the kernels' protocol: take a ticket, wait until the
// slot's previous ticket is acknowledged, post the row and then the ticket,
// wait for done, check the staged row against the pageable one, acknowledge.
// More requests than slots, several requesters and two serving threads.
static void staging_protocol() {
  const int64_t first_row = 1000, n_rows = 20000;
  const size_t row_bytes = 256;
  std::vector<char> pageable((size_t)n_rows * row_bytes);
  for (size_t i = 0; i < pageable.size(); ++i) pageable[i] = (char)((i * 131u) >> 3);
  std::vector<tfe::StageSlot> q(tfe::kStageSlots);
  memset(q.data(), 0, q.size() * sizeof(tfe::StageSlot));
  std::vector<char> rows((size_t)tfe::kStageSlots * row_bytes);
  volatile bool stop = false;
  const int servers = 2;
  std::vector<std::thread> serve;
  for (int i = 0; i < servers; ++i)
    serve.emplace_back(tfe::stage_serve, q.data(), rows.data(), pageable.data(), first_row,
                       n_rows, row_bytes, (uint64_t)i, (uint64_t)servers, &stop);
  std::vector<unsigned long long> ack(tfe::kStageSlots, 0);  // device memory on the GPU
  unsigned long long ticket = 0;
  const int requesters = 8, per = 7500;  // 60000 requests: the queue wraps 14 times
  std::vector<int> bad(requesters, 0);
  std::vector<std::thread> req;
  for (int w = 0; w < requesters; ++w)
    req.emplace_back([&, w] {
      uint64_t x = 0x9E3779B97F4A7C15ull * (w + 1);
      for (int r = 0; r < per; ++r) {
        x ^= x << 13;
        x ^= x >> 7;
        x ^= x << 17;
        const int32_t row = (int32_t)(first_row + (int64_t)(x % (uint64_t)n_rows));
        const unsigned long long tk = __atomic_fetch_add(&ticket, 1ull, __ATOMIC_RELAXED);
        const size_t k = tk % tfe::kStageSlots;
        tfe::StageSlot& sl = q[k];
        const unsigned long long prev = tk >= tfe::kStageSlots ? tk + 1 - tfe::kStageSlots : 0;
        while (__atomic_load_n(&ack[k], __ATOMIC_ACQUIRE) != prev) std::this_thread::yield();
        __atomic_store_n(&sl.req, tfe::stage_request(tk, row), __ATOMIC_RELEASE);
        while (__atomic_load_n(&sl.done, __ATOMIC_ACQUIRE) != tk + 1) std::this_thread::yield();
        const char* got = rows.data() + k * row_bytes;
        const char* want = pageable.data() + (size_t)(row - first_row) * row_bytes;
        if (memcmp(got, want, row_bytes) != 0) ++bad[(size_t)w];
        __atomic_store_n(&ack[k], tk + 1, __ATOMIC_RELEASE);
      }
    });
  for (auto& t : req) t.join();
  __atomic_store_n(&stop, true, __ATOMIC_RELEASE);
  for (auto& t : serve) t.join();
  for (int w = 0; w < requesters; ++w) CHECK(bad[(size_t)w] == 0);
  CHECK(ticket == (unsigned long long)requesters * per);
  // A row id outside the pageable range (never asked for by the kernels)
  // is staged as zeros.
  memset(q.data(), 0, q.size() * sizeof(tfe::StageSlot));
  memset(rows.data(), 0x5A, row_bytes);
  stop = false;
  std::thread one(tfe::stage_serve, q.data(), rows.data(), pageable.data(), first_row, n_rows,
                  row_bytes, (uint64_t)0, (uint64_t)1, &stop);
  __atomic_store_n(&q[0].req, tfe::stage_request(0, (int32_t)(first_row - 1)), __ATOMIC_RELEASE);
  while (__atomic_load_n(&q[0].done, __ATOMIC_ACQUIRE) != 1ull) std::this_thread::yield();
  for (size_t i = 0; i < row_bytes; ++i) CHECK(rows[i] == 0);
  __atomic_store_n(&stop, true, __ATOMIC_RELEASE);
  one.join();
}

int main() {
  validation_errors();
  build_and_probe_all(1 << 20);
  build_and_probe_all(5);
  duplicates();
  hook_and_held_memory();
  staging_protocol();
  printf("ok\n");
  return 0;
}
