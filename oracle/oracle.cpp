// CPU oracle of the TF-Engram phrase-memory lookup + gated residual injection.
//
// TEST INFRASTRUCTURE ONLY.  This is a plain, slow, obviously correct CPU
// statement of what the GPU path computes.  Only the tests, the smoke check
// and the benchmark's CPU-baseline leg may load it; the product library never
// does.  It shares no code with the GPU path (no headers, no helpers, no key
// packing, no hashing): phrases are looked up by their token tuples in a
// std::map.
//
// What it follows (paper sections and equations):
//  * the memory is a key -> value table (Eq. 2); every stored phrase has its
//    own entry and its own value row, so two phrases never share an entry
//    (Sec. 1, Sec. 4.1, Sec. 4.2: each phrase gets its own vector);
//  * the query at position t is formed from the recent tokens: the n-gram
//    windows that end at t, n = n_min..n_max (Eq. 3, Sec. 4.2 first index
//    level, read as "phrases ending at t");
//  * among matching phrases the longest one is selected (Sec. 4.2); a
//    position has one window per length and stored phrases are distinct, so
//    no two matches have the same length and no tie-breaker is needed;
//  * the retrieved row is injected as h' = h + g * m (Eq. 5) with the
//    parameter-free gate g = lambda * sigmoid(<h/rms(h), m/rms(m)> / sqrt(D)),
//    rms(x) = sqrt(mean(x^2) + eps): a train-free reading of "a learned
//    function of the current hidden state and retrieved memory" (Sec. 2.2,
//    Sec. 4.2: nothing is trained), or the constant gate g = lambda;
//  * a position without a match is left unchanged;
//  * the multi-match variant retains every matched phrase and injects their
//    weighted sum (Eq. 4, Eq. 11), with weights proportional to the phrase
//    length or uniform, normalised to add up to 1.
// All arithmetic is in double; the result is rounded once, to nearest-even,
// to the output type.
#include <stdint.h>
#include <string.h>

#include <cmath>
#include <map>
#include <vector>

namespace {

struct Table {
  std::map<std::vector<int32_t>, int64_t> phrase_to_row;
  int n_min = 0, n_max = 0, vocab = 0;
};

// Round a double to the nearest bfloat16 (8 significant bits, exponent range
// of float32), ties to even; returns the bfloat16 bit pattern.
uint16_t round_to_bf16(double x) {
  if (x == 0.0 || !std::isfinite(x)) {
    float f = (float)x;
    uint32_t u;
    memcpy(&u, &f, 4);
    if (std::isnan(x)) return 0x7FC0;
    return (uint16_t)(u >> 16);
  }
  int e;
  std::frexp(x, &e);                      // 2^(e-1) <= |x| < 2^e
  int q = e - 8;                          // spacing of 8-bit significands there
  if (q < -133) q = -133;                 // subnormal spacing
  double r = std::nearbyint(std::ldexp(x, -q));   // ties to even
  double y = std::ldexp(r, q);
  float f = (float)y;                     // exact unless it overflows
  if (std::fabs(y) > 3.3895313892515355e38) f = (float)(y > 0 ? INFINITY : -INFINITY);
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16);
}

double load_elem(const void* base, int64_t i, int dtype) {
  if (dtype == 0) return (double)((const float*)base)[i];
  uint32_t u = (uint32_t)((const uint16_t*)base)[i] << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

void store_elem(void* base, int64_t i, int dtype, double x) {
  if (dtype == 0) ((float*)base)[i] = (float)x;
  else ((uint16_t*)base)[i] = round_to_bf16(x);
}

}  // namespace

extern "C" {

// Status codes (same meaning as the library's, defined separately here).
enum { OR_OK = 0, OR_INVALID = -1, OR_DUPLICATE = -2 };

// Builds the phrase -> row map.  phrase_tokens: [P x n_max], oldest token
// first; row i is phrase_tokens[i, 0:lens[i]].  Rejects lengths outside
// [n_min, n_max], tokens outside [0, vocab) and repeated phrases.
void* oracle_table_new(const int32_t* phrase_tokens, const uint8_t* lens, int64_t P, int n_min,
                       int n_max, int vocab, int* status) {
  *status = OR_INVALID;
  if (P < 0 || n_min < 2 || n_max > 4 || n_min > n_max || vocab <= 0) return nullptr;
  Table* t = new Table;
  t->n_min = n_min;
  t->n_max = n_max;
  t->vocab = vocab;
  for (int64_t i = 0; i < P; ++i) {
    int n = lens[i];
    if (n < n_min || n > n_max) { delete t; return nullptr; }
    std::vector<int32_t> w(phrase_tokens + i * n_max, phrase_tokens + i * n_max + n);
    for (int32_t x : w)
      if (x < 0 || x >= vocab) { delete t; return nullptr; }
    if (!t->phrase_to_row.emplace(w, i).second) {
      delete t;
      *status = OR_DUPLICATE;
      return nullptr;
    }
  }
  *status = OR_OK;
  return t;
}

void oracle_table_free(void* t) { delete (Table*)t; }

// Longest-match lookup.  tokens: [B x (ctx + S)]; position (b, s) is column
// ctx + s of row b, and its n-gram window is columns ctx+s-n+1 .. ctx+s of
// the same row.  A window is formed only if it starts at column >= 0 and all
// its tokens lie in [0, vocab).  Outputs per position b*S + s: hit (0/1),
// row (-1 on a miss) and the matched length (0 on a miss).
int oracle_lookup(const void* table, const int32_t* tokens, int64_t B, int64_t ctx, int64_t S,
                  uint8_t* hit, int32_t* row, uint8_t* len) {
  const Table* t = (const Table*)table;
  if (!t || B < 0 || ctx < 0 || S < 0) return OR_INVALID;
  const int64_t W = ctx + S;
  for (int64_t b = 0; b < B; ++b) {
    for (int64_t s = 0; s < S; ++s) {
      const int64_t c = ctx + s;
      int64_t sel = -1;
      int sel_n = 0;
      for (int n = t->n_max; n >= t->n_min && sel < 0; --n) {
        const int64_t first = c - n + 1;
        if (first < 0) continue;
        std::vector<int32_t> w(tokens + b * W + first, tokens + b * W + c + 1);
        bool valid = true;
        for (int32_t x : w)
          if (x < 0 || x >= t->vocab) valid = false;
        if (!valid) continue;
        auto it = t->phrase_to_row.find(w);
        if (it != t->phrase_to_row.end()) { sel = it->second; sel_n = n; }
      }
      const int64_t p = b * S + s;
      hit[p] = sel >= 0 ? 1 : 0;
      row[p] = (int32_t)sel;
      len[p] = (uint8_t)sel_n;
    }
  }
  return OR_OK;
}

// All-matches lookup (Eq. 4, Eq. 11: every matched entry is retained).
// Same windows as oracle_lookup.  Outputs per position p = b*S + s:
// rows[p*L + j] is the row of the length-(n_min + j) window, or -1 when that
// window is absent or not in the table, L = n_max - n_min + 1; bit j of
// mask[p] is set where rows[p*L + j] >= 0.
int oracle_lookup_all(const void* table, const int32_t* tokens, int64_t B, int64_t ctx,
                      int64_t S, uint8_t* mask, int32_t* rows) {
  const Table* t = (const Table*)table;
  if (!t || B < 0 || ctx < 0 || S < 0) return OR_INVALID;
  const int64_t W = ctx + S;
  const int L = t->n_max - t->n_min + 1;
  for (int64_t b = 0; b < B; ++b) {
    for (int64_t s = 0; s < S; ++s) {
      const int64_t c = ctx + s, p = b * S + s;
      mask[p] = 0;
      for (int j = 0; j < L; ++j) {
        const int n = t->n_min + j;
        rows[p * L + j] = -1;
        const int64_t first = c - n + 1;
        if (first < 0) continue;
        std::vector<int32_t> w(tokens + b * W + first, tokens + b * W + c + 1);
        bool valid = true;
        for (int32_t x : w)
          if (x < 0 || x >= t->vocab) valid = false;
        if (!valid) continue;
        auto it = t->phrase_to_row.find(w);
        if (it == t->phrase_to_row.end()) continue;
        rows[p * L + j] = (int32_t)it->second;
        mask[p] |= (uint8_t)(1u << j);
      }
    }
  }
  return OR_OK;
}

// Gated residual injection (Eq. 5).  hidden, out: [T x D]; values: [R x D];
// index[p] is the row of `values` matched at position p, or -1 for a miss.
// dtype 0 = float32, 1 = bfloat16 (bit patterns); gate 0 = sigmoid of the
// scaled RMS-normalised dot product, 1 = constant.  eps = 1e-6.
int oracle_inject(const void* hidden, const void* values, int64_t R, const int64_t* index,
                  int64_t T, int64_t D, int dtype, int gate, double lambda, void* out) {
  if (T < 0 || D <= 0 || (dtype != 0 && dtype != 1) || (gate != 0 && gate != 1)) return OR_INVALID;
  const size_t esz = dtype == 0 ? 4 : 2;
  const double eps = 1e-6;
  for (int64_t p = 0; p < T; ++p) {
    const int64_t r = index[p];
    if (r < 0) {
      memcpy((char*)out + p * D * esz, (const char*)hidden + p * D * esz, D * esz);
      continue;
    }
    if (r >= R) return OR_INVALID;
    std::vector<double> h(D), m(D);
    for (int64_t j = 0; j < D; ++j) {
      h[j] = load_elem(hidden, p * D + j, dtype);
      m[j] = load_elem(values, r * D + j, dtype);
    }
    double g = lambda;
    if (gate == 0) {
      double shh = 0, smm = 0, shm = 0;
      for (int64_t j = 0; j < D; ++j) {
        shh += h[j] * h[j];
        smm += m[j] * m[j];
        shm += h[j] * m[j];
      }
      const double rms_h = std::sqrt(shh / (double)D + eps);
      const double rms_m = std::sqrt(smm / (double)D + eps);
      const double z = shm / (rms_h * rms_m) / std::sqrt((double)D);
      g = lambda / (1.0 + std::exp(-z));
    }
    for (int64_t j = 0; j < D; ++j) store_elem(out, p * D + j, dtype, h[j] + g * m[j]);
  }
  return OR_OK;
}

// Injection of an aggregated memory signal (Eq. 4 / Eq. 11, then Eq. 5).
// index: [T x L]; index[p*L + j] is the row of `values` retained at position
// p for the phrase of length n_min + j, or -1.  The retained rows are
// combined as m = sum_j alpha_j v_j with
//   weighting 0 (by length):  alpha_j = n_j / sum_k n_k,
//   weighting 1 (uniform):    alpha_j = 1 / |retained|,
// the sums running over the retained rows only, so the weights add up to 1.
// m then goes through the same gate and residual as oracle_inject; a
// position with no retained row is copied unchanged.
int oracle_inject_multi(const void* hidden, const void* values, int64_t R, const int64_t* index,
                        int64_t T, int L, int n_min, int64_t D, int dtype, int weighting,
                        int gate, double lambda, void* out) {
  if (T < 0 || D <= 0 || L < 1 || (dtype != 0 && dtype != 1) || (gate != 0 && gate != 1) ||
      (weighting != 0 && weighting != 1))
    return OR_INVALID;
  const size_t esz = dtype == 0 ? 4 : 2;
  const double eps = 1e-6;
  for (int64_t p = 0; p < T; ++p) {
    double wsum = 0;
    for (int j = 0; j < L; ++j) {
      const int64_t r = index[p * L + j];
      if (r >= R) return OR_INVALID;
      if (r >= 0) wsum += weighting == 0 ? (double)(n_min + j) : 1.0;
    }
    if (wsum == 0) {
      memcpy((char*)out + p * D * esz, (const char*)hidden + p * D * esz, D * esz);
      continue;
    }
    std::vector<double> h(D), m(D, 0.0);
    for (int64_t k = 0; k < D; ++k) h[k] = load_elem(hidden, p * D + k, dtype);
    for (int j = 0; j < L; ++j) {
      const int64_t r = index[p * L + j];
      if (r < 0) continue;
      const double alpha = (weighting == 0 ? (double)(n_min + j) : 1.0) / wsum;
      for (int64_t k = 0; k < D; ++k) m[k] += alpha * load_elem(values, r * D + k, dtype);
    }
    double g = lambda;
    if (gate == 0) {
      double shh = 0, smm = 0, shm = 0;
      for (int64_t k = 0; k < D; ++k) {
        shh += h[k] * h[k];
        smm += m[k] * m[k];
        shm += h[k] * m[k];
      }
      const double z = shm / (std::sqrt(shh / (double)D + eps) * std::sqrt(smm / (double)D + eps)) /
                       std::sqrt((double)D);
      g = lambda / (1.0 + std::exp(-z));
    }
    for (int64_t k = 0; k < D; ++k) store_elem(out, p * D + k, dtype, h[k] + g * m[k]);
  }
  return OR_OK;
}

// The gate value alone, for one (h, m) pair (used by the closed-form checks).
double oracle_gate(const void* h, const void* m, int64_t D, int dtype, int gate, double lambda) {
  if (gate == 1) return lambda;
  const double eps = 1e-6;
  double shh = 0, smm = 0, shm = 0;
  for (int64_t j = 0; j < D; ++j) {
    double a = load_elem(h, j, dtype), b = load_elem(m, j, dtype);
    shh += a * a;
    smm += b * b;
    shm += a * b;
  }
  const double z = shm / (std::sqrt(shh / (double)D + eps) * std::sqrt(smm / (double)D + eps)) /
                   std::sqrt((double)D);
  return lambda / (1.0 + std::exp(-z));
}

// Double -> bfloat16 rounding, exposed for its own pins.
uint16_t oracle_round_bf16(double x) { return round_to_bf16(x); }

}  // extern "C"
