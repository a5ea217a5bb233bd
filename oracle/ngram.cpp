// CPU oracle of offline phrase-table construction by n-gram frequency
// (TEST INFRASTRUCTURE ONLY; see oracle.cpp for who may load it).
//
// What it follows: phrase mining selects candidate multi-token expressions
// by corpus frequency (Sec. 4.2, frequency thresholds; the construction-cost
// measurement counts this n-gram extraction step).  Here: every window of n
// consecutive tokens of the stream whose tokens all lie in [0, vocab) is one
// occurrence of its tuple; distinct tuples are ranked by occurrence count,
// most frequent first, equal counts by the tuple in lexicographic order
// (oldest token first); ranks [skip, skip + top) are the result.
// Plain steps: collect the tuples, sort them, count runs, sort by rank.
#include <stdint.h>

#include <algorithm>
#include <vector>

extern "C" {

// tokens: [N] int32 (HOST).  Writes up to `top` tuples (oldest token first,
// [top x n] int32) and their counts; returns how many were written, or -1
// for bad arguments.
int64_t oracle_ngram_top(const int32_t* tokens, int64_t N, int vocab, int n, int64_t skip,
                         int64_t top, int32_t* out_tuples, int64_t* out_counts) {
  if (N < 0 || vocab <= 0 || n < 1 || n > 4 || skip < 0 || top < 0) return -1;
  std::vector<std::vector<int32_t>> tuples;
  for (int64_t i = 0; i + n <= N; ++i) {
    bool ok = true;
    for (int j = 0; j < n; ++j)
      if (tokens[i + j] < 0 || tokens[i + j] >= vocab) ok = false;
    if (ok) tuples.emplace_back(tokens + i, tokens + i + n);
  }
  std::sort(tuples.begin(), tuples.end());
  std::vector<std::pair<int64_t, int64_t>> ranked;  // (-count, index of first occurrence)
  for (size_t i = 0; i < tuples.size();) {
    size_t j = i + 1;
    while (j < tuples.size() && tuples[j] == tuples[i]) ++j;
    ranked.push_back({-(int64_t)(j - i), (int64_t)i});
    i = j;
  }
  // Equal counts keep tuple order: the indices grow with the tuple.
  std::sort(ranked.begin(), ranked.end());
  int64_t w = 0;
  for (int64_t r = skip; r < (int64_t)ranked.size() && w < top; ++r, ++w) {
    const std::vector<int32_t>& t = tuples[ranked[r].second];
    for (int j = 0; j < n; ++j) out_tuples[w * n + j] = t[j];
    out_counts[w] = -ranked[r].first;
  }
  return w;
}

}  // extern "C"
