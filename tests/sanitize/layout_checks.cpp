// The host layout planner (relabel, dense prefix, capacities, regions; the
// all-host reference behind lda_describe_layout) under AddressSanitizer and
// UndefinedBehaviorSanitizer, CPU only: seeded corpora of many shapes, with
// the layout invariants checked.  Exit status 0 = every check held.
#include <algorithm>
#include <cstdio>
#include <numeric>
#include <random>
#include <vector>

#include "lda_internal.h"

#define CHECK(c)                                                      \
  do {                                                                \
    if (!(c)) {                                                       \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      return 1;                                                       \
    }                                                                 \
  } while (0)

static int one(std::mt19937 &g, int trial) {
  const int V = 1 + int(g() % 60), K = 2 + int(g() % 300), R = 1 + int(g() % 50);
  const int M = 1 + int(g() % 40), n = 1 + int(g() % 3000);
  const int cutoff = int(g() % 4) == 0 ? -1 : int(g() % 3) == 0 ? int(g() % 20) : 0;
  std::vector<int32_t> word(static_cast<size_t>(n)), doc(static_cast<size_t>(n));
  for (int i = 0; i < n; ++i) {
    word[size_t(i)] = int32_t(g() % uint32_t(V));
    doc[size_t(i)] = int32_t(g() % uint32_t(M));
  }
  if (trial % 2) std::sort(doc.begin(), doc.end());
  lda::Layout L;
  std::string msg;
  CHECK(lda::build_layout(word.data(), doc.data(), n, V, K, R, cutoff, L, msg) == LDA_OK);
  CHECK(L.word_off.size() == size_t(L.n_present) + 1 && L.word_off.back() == uint32_t(n));
  std::vector<int> seen(static_cast<size_t>(n), 0);
  for (uint32_t k : L.wt_key) seen[k]++;
  for (int s : seen) CHECK(s == 1);
  std::vector<int> covered(static_cast<size_t>(n), 0);
  for (size_t r = 0; r < L.region.size(); r += 3) {
    const uint32_t v = L.region[r], b = L.region[r + 1], e = L.region[r + 2];
    CHECK(int32_t(v) < L.n_present && b < e && L.word_off[v] <= b && e <= L.word_off[v + 1]);
    CHECK(e - b <= uint32_t(R) || int32_t(v) >= L.n_dense);
    for (uint32_t q = b; q < e; ++q) covered[q]++;
  }
  for (int c : covered) CHECK(c == 1);
  for (int32_t d = 0; d < L.M; ++d) CHECK(L.d_cap[size_t(d) + 1] > L.d_cap[size_t(d)]);
  // regions of a word-offset table with empty words, as an out-of-core chunk plans them
  std::vector<uint32_t> woff(static_cast<size_t>(V) + 1, 0);
  for (int v = 0; v < V; ++v) woff[size_t(v) + 1] = woff[size_t(v)] + (g() % 3 == 0 ? 0u : uint32_t(g() % 40));
  std::vector<uint8_t> split;
  std::vector<uint32_t> region;
  int64_t ndr = 0;
  lda::make_regions(woff, V, R, split, region, ndr);
  uint64_t tokens = 0;
  for (size_t r = 0; r < region.size(); r += 3) tokens += region[r + 2] - region[r + 1];
  CHECK(tokens == woff.back() && ndr == int64_t(region.size() / 3));
  return 0;
}

int main() {
  std::mt19937 g(20240);
  for (int trial = 0; trial < 300; ++trial)
    if (one(g, trial)) {
      std::fprintf(stderr, "trial %d\n", trial);
      return 1;
    }
  std::printf("layout checks passed\n");
  return 0;
}
