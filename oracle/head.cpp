// CPU oracle of the early-exit prefetch head (TEST INFRASTRUCTURE ONLY; see
// oracle.cpp for who may load it).
//
// What it follows:
//  * the head maps an intermediate hidden state h (one row per sequence) to
//    an approximate next-token distribution p = softmax(W h), W being the
//    [V x D] projection of the head (Eq. 13);
//  * the candidates are the K most likely tokens of p (Eq. 14).  Ties in
//    probability (equal logits) are broken by the lower token id, which makes
//    the answer unique.
// Logits are exact-order double sums over d = 0..D-1; the softmax subtracts
// the maximum logit before exponentiating (the textbook stable form).
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

namespace {

double elem(const void* base, int64_t i, int dtype) {
  if (dtype == 0) return (double)((const float*)base)[i];
  uint32_t u = (uint32_t)((const uint16_t*)base)[i] << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

}  // namespace

extern "C" {

// w: [V x D], h: [B x D] (dtype 0 = float32, 1 = bfloat16 bit patterns).
// Outputs per row b: ids[b*K + i] and probs[b*K + i] for the i-th most likely
// token (probability descending, ties by lower id); logits, when not null,
// receives all [B x V] logits.  Returns 0, or -1 for bad sizes.
int oracle_head_topk(const void* w, const void* h, int64_t V, int64_t D, int64_t B, int64_t K,
                     int dtype, int32_t* ids, double* probs, double* logits) {
  if (V <= 0 || D <= 0 || B < 0 || K < 0 || K > V || (dtype != 0 && dtype != 1)) return -1;
  std::vector<double> l(V);
  std::vector<int64_t> order(V);
  for (int64_t b = 0; b < B; ++b) {
    for (int64_t v = 0; v < V; ++v) {
      double s = 0;
      for (int64_t d = 0; d < D; ++d) s += elem(w, v * D + d, dtype) * elem(h, b * D + d, dtype);
      l[v] = s;
      if (logits) logits[b * V + v] = s;
    }
    const double m = *std::max_element(l.begin(), l.end());
    double z = 0;
    for (int64_t v = 0; v < V; ++v) z += std::exp(l[v] - m);
    std::iota(order.begin(), order.end(), 0);
    std::partial_sort(order.begin(), order.begin() + K, order.end(), [&](int64_t a, int64_t c) {
      return l[a] > l[c] || (l[a] == l[c] && a < c);
    });
    for (int64_t i = 0; i < K; ++i) {
      ids[b * K + i] = (int32_t)order[i];
      probs[b * K + i] = std::exp(l[order[i]] - m) / z;
    }
  }
  return 0;
}

}  // extern "C"
