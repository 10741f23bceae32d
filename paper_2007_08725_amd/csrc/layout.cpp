// Token layout, host side (runs once inside lda_create).
//
//   Sec. 4.2: words are relabelled by descending token count so that the
//             dense words (count > K) form a prefix of the id space; a sparse
//             word's row capacity is its token count.
//   Sec. 4.3: the tokens are kept in two orders: by document (the order the
//             count rebuild of D walks) and by word (the order the sampler
//             walks); dt_wpos links each doc-ordered token to its word-order
//             slot, i.e. the inverted index between the two orders.
//   Sec. 5.1: every word is cut into regions of at most R consecutive
//             word-ordered tokens (large-word dissection); the regions are
//             the units the atomic scheduler hands out, in an order that
//             keeps the documents of concurrent regions close (see the end
//             of plan_from_counts).
//
// scan_tokens and plan_from_counts are shared by the device builder (the
// sorts run on the GPU, see layout_gpu.hip) and by build_layout, the
// all-host reference used by lda_describe_layout.
#include <algorithm>
#include <cmath>
#include <numeric>

#include "lda_internal.h"

namespace lda {

lda_status scan_tokens(const int32_t *word, const int32_t *doc, int64_t n, int32_t V, int32_t &M, bool &doc_sorted,
                       std::string &msg) {
  if (n <= 0 || V <= 0) {
    msg = "bad sizes";
    return LDA_E_ARG;
  }
  if (n >= (int64_t(1) << 32)) {
    msg = "n_tokens must be below 2^32 (32-bit token positions)";
    return LDA_E_RANGE;
  }
  int64_t maxdoc = -1;
  bool sorted = true;
  int32_t prev = 0;
  for (int64_t i = 0; i < n; i++) {
    const int32_t w = word[i], d = doc[i];
    if (w < 0 || w >= V) {
      msg = "word id out of range at token " + std::to_string(i);
      return LDA_E_ARG;
    }
    if (d < 0) {
      msg = "negative doc id at token " + std::to_string(i);
      return LDA_E_ARG;
    }
    if (d > maxdoc) maxdoc = d;
    if (d < prev) sorted = false;
    prev = d;
  }
  M = int32_t(maxdoc + 1);
  doc_sorted = sorted;
  return LDA_OK;
}

void make_regions(const std::vector<uint32_t> &word_off, int32_t nd, int32_t R, std::vector<uint8_t> &split,
                  std::vector<uint32_t> &region, int64_t &n_dense_regions) {
  const int32_t np = int32_t(word_off.size()) - 1;
  auto count = [&](uint32_t r) { return word_off[r + 1] - word_off[r]; };
  // regions (Sec. 5.1): a dense word with c tokens becomes ceil(c/R) regions
  // of near-equal size; a sparse word is always one region; a word without
  // tokens has none
  split.assign(size_t(std::max(nd, 0)), 0);
  region.clear();
  n_dense_regions = 0;
  for (int32_t r = 0; r < np; r++) {
    const uint32_t b = word_off[size_t(r)], c = count(uint32_t(r));
    if (c == 0) continue;
    uint64_t nreg = 1;
    if (r < nd) nreg = (uint64_t(c) + uint64_t(R) - 1) / uint64_t(R);
    if (r < nd && nreg > 1) split[size_t(r)] = 1;
    for (uint64_t q = 0; q < nreg; q++) {
      region.push_back(uint32_t(r));
      region.push_back(b + uint32_t(uint64_t(c) * q / nreg));
      region.push_back(b + uint32_t(uint64_t(c) * (q + 1) / nreg));
      if (r < nd) n_dense_regions++;
    }
  }
  // Hand-out order (a choice of this implementation, not the paper's): the
  // regions of split words by the middle of their span of the word's
  // document-sorted tokens, which tracks the document ids they touch, so the
  // regions that run at the same time read the D rows of nearby documents and
  // the device's last-level cache serves the repeated reads; then the
  // unsplit words in word order (the small regions last, filling the tail).
  const size_t nr = region.size() / 3;
  std::vector<size_t> split_idx, rest_idx;
  for (size_t i = 0; i < nr; ++i) {
    const uint32_t r = region[3 * i];
    (int32_t(r) < nd && split[r] ? split_idx : rest_idx).push_back(i);
  }
  // middle of region i as a fraction of its word: (b + e - 2 wb) / (2 c), compared exactly
  auto mid_num = [&](size_t i) {
    const uint32_t r = region[3 * i];
    return uint64_t(region[3 * i + 1] - word_off[r]) + uint64_t(region[3 * i + 2] - word_off[r]);
  };
  std::stable_sort(split_idx.begin(), split_idx.end(), [&](size_t x, size_t y) {
    const unsigned __int128 lhs = (unsigned __int128)mid_num(x) * count(region[3 * y]);
    const unsigned __int128 rhs = (unsigned __int128)mid_num(y) * count(region[3 * x]);
    return lhs < rhs;
  });
  std::vector<uint32_t> ordered;
  ordered.reserve(region.size());
  for (const std::vector<size_t> *part : {&split_idx, &rest_idx})
    for (size_t i : *part) ordered.insert(ordered.end(), region.begin() + 3 * i, region.begin() + 3 * i + 3);
  region.swap(ordered);
}

lda_status plan_from_counts(const std::vector<uint32_t> &cnt, int32_t K, int32_t R, int32_t dense_cutoff, Layout &L,
                            std::string &msg, bool rows) {
  const int32_t V = int32_t(cnt.size());
  const int32_t M = int32_t(L.doc_off.size()) - 1;
  for (int32_t d = 0; d < M; d++) {
    if (L.doc_off[size_t(d) + 1] - L.doc_off[size_t(d)] > uint32_t(LDA_MAX_DOC_LEN)) {
      msg = "document " + std::to_string(d) + " has more than 65535 tokens";
      return LDA_E_RANGE;
    }
  }
  // relabel: descending count, ties by ascending caller id (stable sort)
  std::vector<int32_t> order(static_cast<size_t>(V));
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return cnt[size_t(a)] > cnt[size_t(b)]; });
  L.relabel.assign(size_t(V), 0);
  for (int32_t r = 0; r < V; r++) L.relabel[size_t(order[size_t(r)])] = r;
  int32_t np = 0, nd = 0;
  const uint32_t cutoff = dense_cutoff == 0 ? uint32_t(K) : dense_cutoff < 0 ? 0u : uint32_t(dense_cutoff);
  for (int32_t r = 0; r < V; r++) {
    const uint32_t c = cnt[size_t(order[size_t(r)])];
    if (c > 0) np++;
    // dense iff the count exceeds the cutoff, K by default (Sec. 4.2); a
    // count above 65535 cannot be packed in a 16-bit sparse entry, so such a
    // word is dense as well
    if (c > 0 && (c > cutoff || c > 65535u)) nd++;
  }
  L.n_present = np;
  L.n_dense = nd;
  L.inv.assign(order.begin(), order.begin() + np);
  L.count.resize(size_t(np));
  for (int32_t r = 0; r < np; r++) L.count[size_t(r)] = cnt[size_t(order[size_t(r)])];
  L.word_off.assign(size_t(np) + 1, 0);
  for (int32_t r = 0; r < np; r++) L.word_off[size_t(r) + 1] = L.word_off[size_t(r)] + L.count[size_t(r)];

  if (!rows) return LDA_OK;
  // capacities: a D row is one header slot (len << 16 | nnz) followed by at
  // most min(len, K) packed entries (Sec. 4.2), padded to the sampler's
  // chunk (multiples of 32 slots); sparse W rows = token count
  L.d_cap.assign(size_t(M) + 1, 0);
  uint64_t total = 0;
  for (int32_t d = 0; d < M; d++) {
    const uint32_t len = L.doc_off[size_t(d) + 1] - L.doc_off[size_t(d)];
    total += d_row_slots(std::min<uint32_t>(len, uint32_t(K)));
    if (total + kRowPad >= (uint64_t(1) << 32)) {
      msg = "documents plus tokens exceed the 32-bit offsets of D";
      return LDA_E_RANGE;
    }
    L.d_cap[size_t(d) + 1] = uint32_t(total);
  }
  const int32_t ns = np - nd;
  L.ws_cap.assign(size_t(ns) + 1, 0);
  for (int32_t s = 0; s < ns; s++) L.ws_cap[size_t(s) + 1] = L.ws_cap[size_t(s)] + L.count[size_t(nd + s)];

  make_regions(L.word_off, nd, R, L.split, L.region, L.n_dense_regions);
  L.n_regions = int64_t(L.region.size() / 3);
  return LDA_OK;
}

lda_status build_layout(const int32_t *word, const int32_t *doc, int64_t n, int32_t V, int32_t K, int32_t R,
                        int32_t dense_cutoff, Layout &L, std::string &msg) {
  if (K < 2 || R <= 0) {
    msg = "build_layout: bad sizes";
    return LDA_E_ARG;
  }
  int32_t M = 0;
  bool identity = false;
  lda_status st = scan_tokens(word, doc, n, V, M, identity, msg);
  if (st != LDA_OK) return st;
  L = Layout();
  L.n = n;
  L.V = V;
  L.K = K;
  L.M = M;
  L.key_identity = identity;

  L.doc_off.assign(size_t(M) + 1, 0);
  for (int64_t i = 0; i < n; i++) L.doc_off[size_t(doc[i]) + 1]++;
  for (int32_t d = 0; d < M; d++) L.doc_off[size_t(d) + 1] += L.doc_off[size_t(d)];
  std::vector<uint32_t> cnt(static_cast<size_t>(V), 0u);
  for (int64_t i = 0; i < n; i++) cnt[size_t(word[i])]++;
  st = plan_from_counts(cnt, K, R, dense_cutoff, L, msg);
  if (st != LDA_OK) return st;

  // doc order: stable counting sort by document
  std::vector<uint32_t> dt_word(static_cast<size_t>(n)), dt_key;
  if (!identity) dt_key.resize(size_t(n));
  {
    std::vector<uint32_t> pos(L.doc_off.begin(), L.doc_off.end() - 1);
    for (int64_t i = 0; i < n; i++) {
      const uint32_t p = pos[size_t(doc[i])]++;
      dt_word[p] = uint32_t(L.relabel[size_t(word[i])]);
      if (!identity) dt_key[p] = uint32_t(i);
    }
  }
  // word order: stable counting sort of the doc-ordered tokens by new word id
  L.wt_key.resize(size_t(n));
  {
    std::vector<uint32_t> cur(L.word_off.begin(), L.word_off.end() - 1);
    for (int32_t d = 0; d < M; d++)
      for (uint32_t p = L.doc_off[size_t(d)]; p < L.doc_off[size_t(d) + 1]; p++)
        L.wt_key[cur[dt_word[p]]++] = identity ? p : dt_key[p];
  }
  return LDA_OK;
}

}  // namespace lda
