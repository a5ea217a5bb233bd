// Seeded synthetic workload generator, host part (C ABI, OpenMP).
//
// Test and benchmark infrastructure only: it produces token streams, phrase
// tables and normal-distributed rows.  It contains none of the phrase-memory
// method's arithmetic (no key packing of the method, no hashing of the method,
// no lookup, no gate), and it is the only code shared by the oracle side and
// the GPU side of the tests.
//
// Results never depend on the number of OpenMP threads.
#include <stdint.h>
#include <string.h>

#include <sys/mman.h>

#include <algorithm>
#include <cstdlib>
#include <new>
#include <cmath>
#include <vector>

#include "synth_rng.h"

namespace {

// Vose's alias method (M. D. Vose, IEEE TSE 1991) for the truncated Zipf law
// p(r) ~ r^-s over ranks r = 1..V; token id = r - 1.
void build_alias(int V, double s, double* prob, int32_t* alias) {
  std::vector<double> q(V);
  double z = 0.0;
  for (int i = 0; i < V; ++i) z += std::pow((double)(i + 1), -s);
  for (int i = 0; i < V; ++i) q[i] = std::pow((double)(i + 1), -s) / z * V;
  std::vector<int32_t> small, large;
  small.reserve(V);
  large.reserve(V);
  for (int i = V - 1; i >= 0; --i) (q[i] < 1.0 ? small : large).push_back(i);
  while (!small.empty() && !large.empty()) {
    int32_t l = small.back(); small.pop_back();
    int32_t g = large.back(); large.pop_back();
    prob[l] = q[l];
    alias[l] = g;
    q[g] = (q[g] + q[l]) - 1.0;
    (q[g] < 1.0 ? small : large).push_back(g);
  }
  for (int32_t g : large) { prob[g] = 1.0; alias[g] = g; }
  for (int32_t l : small) { prob[l] = 1.0; alias[l] = l; }
}

template <class K>
inline K pack_tuple(const int32_t* t, int n, int V) {
  K k = 0;
  for (int j = 0; j < n; ++j) k = k * (K)V + (K)(uint32_t)t[j];
  return k;
}

template <class K>
inline void unpack_tuple(K k, int n, int V, int32_t* t) {
  for (int j = n - 1; j >= 0; --j) { t[j] = (int32_t)(k % (K)V); k /= (K)V; }
}

template <class K>
inline uint32_t part_of(K k) {
  uint64_t lo = (uint64_t)k, hi = (uint64_t)(k >> 32 >> 32);
  return (uint32_t)(synth_mix(lo ^ synth_mix(hi)) >> 56);
}


// Uninitialised array whose pages are first touched by the parallel loops
// that fill it (value-initialising a multi-GB vector would zero it serially),
// backed by transparent huge pages where the kernel allows them: a
// multi-GB scratch array otherwise costs millions of 4 KiB page faults.
template <class T>
struct RawArray {
  T* p = nullptr;
  size_t bytes = 0;
  explicit RawArray(int64_t n) {
    const size_t huge = (size_t)2 << 20;
    bytes = (sizeof(T) * (size_t)(n > 0 ? n : 1) + huge - 1) / huge * huge;
    p = static_cast<T*>(std::aligned_alloc(huge, bytes));
    if (!p) throw std::bad_alloc();
    madvise(p, bytes, MADV_HUGEPAGE);
  }
  ~RawArray() { std::free(p); }
  RawArray(const RawArray&) = delete;
  RawArray& operator=(const RawArray&) = delete;
  T& operator[](int64_t i) { return p[i]; }
};

template <class K>
int64_t ngram_top(const int32_t* tok, int64_t ntok, int n, int V, int64_t skip,
                  int64_t want, int32_t* out_tuples, int64_t* out_counts) {
  const int64_t nk = ntok - n + 1;
  if (nk <= 0 || want <= 0) return 0;
  const int NP = 1024;
  // Fixed chunking: the scatter order never depends on the thread count.
  const int NCH = 128;
  std::vector<int64_t> hist((size_t)NCH * NP, 0);
#pragma omp parallel for schedule(static)
  for (int c = 0; c < NCH; ++c) {
    int64_t a = nk * c / NCH, b = nk * (c + 1) / NCH;
    int64_t* h = &hist[(size_t)c * NP];
    for (int64_t i = a; i < b; ++i) h[part_of(pack_tuple<K>(tok + i, n, V)) % NP]++;
  }
  std::vector<int64_t> off((size_t)NCH * NP + 1, 0), pstart(NP + 1, 0);
  {
    int64_t acc = 0;
    for (int p = 0; p < NP; ++p) {
      pstart[p] = acc;
      for (int c = 0; c < NCH; ++c) { off[(size_t)c * NP + p] = acc; acc += hist[(size_t)c * NP + p]; }
    }
    pstart[NP] = acc;
  }
  RawArray<K> part(nk);
#pragma omp parallel for schedule(static)
  for (int c = 0; c < NCH; ++c) {
    int64_t a = nk * c / NCH, b = nk * (c + 1) / NCH;
    int64_t* o = &off[(size_t)c * NP];
    for (int64_t i = a; i < b; ++i) {
      K k = pack_tuple<K>(tok + i, n, V);
      part[o[part_of(k) % NP]++] = k;
    }
  }
  // Per partition: sort and run-length count in place (distinct keys are
  // compacted to the front of the partition; counts go to a parallel array).
  RawArray<int64_t> cnt(nk);
  std::vector<int64_t> ndist(NP, 0);
#pragma omp parallel for schedule(dynamic, 1)
  for (int p = 0; p < NP; ++p) {
    K* a = part.p + pstart[p];
    int64_t* c = cnt.p + pstart[p];
    int64_t m = pstart[p + 1] - pstart[p];
    std::sort(a, a + m);
    int64_t d = 0;
    for (int64_t i = 0; i < m;) {
      int64_t j = i + 1;
      while (j < m && a[j] == a[i]) ++j;
      a[d] = a[i];
      c[d] = j - i;
      ++d;
      i = j;
    }
    ndist[p] = d;
  }
  int64_t total = 0;
  for (int p = 0; p < NP; ++p) total += ndist[p];
  const int64_t K_ = std::min<int64_t>(skip + want, total);
  if (K_ <= skip) return 0;
  // Threshold count: the K_-th largest count.
  std::vector<int64_t> allc;
  allc.reserve(total);
  for (int p = 0; p < NP; ++p) allc.insert(allc.end(), cnt.p + pstart[p], cnt.p + pstart[p] + ndist[p]);
  std::nth_element(allc.begin(), allc.begin() + (K_ - 1), allc.end(), std::greater<int64_t>());
  const int64_t cstar = allc[K_ - 1];
  std::vector<int64_t>().swap(allc);
  std::vector<std::pair<int64_t, K>> sel;  // (-count, key)
  std::vector<K> ties;
  for (int p = 0; p < NP; ++p) {
    const K* a = part.p + pstart[p];
    const int64_t* c = cnt.p + pstart[p];
    for (int64_t i = 0; i < ndist[p]; ++i) {
      if (c[i] > cstar) sel.push_back({-c[i], a[i]});
      else if (c[i] == cstar) ties.push_back(a[i]);
    }
  }
  std::sort(ties.begin(), ties.end());
  for (int64_t i = 0; (int64_t)sel.size() < K_; ++i) sel.push_back({-cstar, ties[i]});
  std::sort(sel.begin(), sel.end());
  int64_t got = K_ - skip;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < got; ++i) {
    unpack_tuple<K>(sel[skip + i].second, n, V, out_tuples + i * n);
    out_counts[i] = -sel[skip + i].first;
  }
  return got;
}

}  // namespace

extern "C" {

// Alias tables for truncated Zipf(s) over V ids.  prob: double[V], alias: int32[V].
int synth_zipf_alias(int V, double s, double* prob, int32_t* alias) {
  if (V <= 0 || !(s > 0.0)) return -1;
  build_alias(V, s, prob, alias);
  return 0;
}

// n i.i.d. Zipf tokens: token i uses draw(key, i) (upper 32 bits pick a column
// by multiply-shift, lower 32 bits are the acceptance fraction).
void synth_zipf_tokens(uint64_t key, int64_t i0, int64_t n, const double* prob,
                       const int32_t* alias, int V, int32_t* out) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    uint64_t h = synth_draw(key, (uint64_t)(i0 + i));
    uint32_t col = (uint32_t)(((h >> 32) * (uint64_t)(uint32_t)V) >> 32);
    double frac = (double)(uint32_t)h * (1.0 / 4294967296.0);
    out[i] = frac < prob[col] ? (int32_t)col : alias[col];
  }
}

// Most frequent distinct n-grams (2 <= n <= 4) of one token stream, ranked by
// count descending then by tuple ascending; ranks [skip, skip+want) are
// written as tuples (oldest token first) with their counts.  Returns how many
// were written.
int64_t synth_ngram_top(const int32_t* tok, int64_t ntok, int n, int V, int64_t skip,
                        int64_t want, int32_t* out_tuples, int64_t* out_counts) {
  if (n < 1 || n > 4 || V <= 0) return -1;
  if (n <= 3) return ngram_top<uint64_t>(tok, ntok, n, V, skip, want, out_tuples, out_counts);
  return ngram_top<unsigned __int128>(tok, ntok, n, V, skip, want, out_tuples, out_counts);
}

// Normal rows: element (row, col) of a table with `cols` columns is
// normal(key, row*cols + col) * scale.  rows: int64[nrows] (row ids to draw).
// dtype 0 = float32, 1 = bfloat16 (nearest-even).  out: [nrows x cols].
void synth_normal_rows(uint64_t key, const int64_t* rows, int64_t nrows, int64_t cols,
                       float scale, int dtype, void* out) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < nrows; ++r) {
    uint64_t base = (uint64_t)rows[r] * (uint64_t)cols;
    for (int64_t c = 0; c < cols; ++c) {
      float x = (float)synth_irwin_hall_n(key, base + (uint64_t)c) * scale;
      if (dtype == 0) ((float*)out)[r * cols + c] = x;
      else ((uint16_t*)out)[r * cols + c] = synth_f32_to_bf16(x);
    }
  }
}

// Same as synth_normal_rows for the contiguous row range [row0, row0+nrows).
void synth_normal_range(uint64_t key, int64_t row0, int64_t nrows, int64_t cols, float scale,
                        int dtype, void* out) {
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < nrows; ++r) {
    uint64_t base = (uint64_t)(row0 + r) * (uint64_t)cols;
    for (int64_t c = 0; c < cols; ++c) {
      float x = (float)synth_irwin_hall_n(key, base + (uint64_t)c) * scale;
      if (dtype == 0) ((float*)out)[r * cols + c] = x;
      else ((uint16_t*)out)[r * cols + c] = synth_f32_to_bf16(x);
    }
  }
}

uint64_t synth_stream_key(uint64_t seed, uint64_t tag) { return synth_key(seed, tag); }

}  // extern "C"
