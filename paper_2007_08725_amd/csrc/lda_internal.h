// Internal declarations of liblda: host layout, device state and kernel
// launchers.  Device code targets gfx950 (CDNA4, wave64) only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "../../include/lda.h"

namespace lda {

// Slack entries after the last D row.
constexpr uint32_t kRowPad = 256;

// Slots a D row with nnz entries occupies: its header and entries, rounded
// up to the chunk the sampler reads it in (32 slots up to 128, 64 up to 256,
// then 128).  Every row starts at a multiple of 32 slots (128 bytes), so
// chunks are whole cache lines.  The slots past the entries hold count-0
// entries of topic K (K << 16), whose W^ is 0, so the sampler reads whole
// chunks without bounds checks.
__host__ __device__ inline uint32_t d_row_slots(uint32_t nnz) {
  const uint32_t n = nnz + 1u;
  return n <= 128u ? (n + 31u) & ~31u : n <= 256u ? (n + 63u) & ~63u : (n + 127u) & ~127u;
}
// Words of the per-iteration skip bitmap (one bit per token, a whole number
// of 64-word blocks).
__host__ __device__ inline int64_t skip_words(int64_t n) { return (n + 2047) / 2048 * 64; }
// LDS words (u32) per wave of the D rebuild: K 16-bit counts, a bitmap of K
// bits and a list of up to min(K, 2048) 16-bit topics
__host__ __device__ inline size_t d_rebuild_lds_words(int K) {
  const size_t half = size_t(K + 1) / 2;
  return half + size_t(K + 31) / 32 + (half < 1024 ? half : 1024);
}
constexpr int kDefaultRegionTokens = 10000;  // Sec. 5.1
constexpr int kBlock = 256;                  // threads per workgroup (4 wave64)
constexpr int kXcds = 8;                     // accelerator dies (XCDs), each with its own L2
// Documents longer than this many tokens are heavy: the doc pass and the D
// rebuild give each a whole workgroup instead of a wave (Sec. 5.1).
constexpr uint32_t kHeavyDocTokens = 4096;

// ----------------------------------------------------------------- layout --
// Host-side token layout (Sec. 4.2-4.3 and 5.1).
//   doc order : tokens stably sorted by document
//   word order: tokens stably sorted by relabelled word (within a word the
//               documents ascend, since the source is doc order)
struct Layout {
  int64_t n = 0;
  int32_t M = 0, V = 0, K = 0;
  int32_t n_present = 0;  // words with at least one token (relabelled ids 0..)
  int32_t n_dense = 0;    // relabelled ids [0, n_dense) have count > K
  std::vector<int32_t> relabel;   // [V] caller id -> new id
  std::vector<int32_t> inv;       // [n_present] new id -> caller id
  std::vector<uint32_t> count;    // [n_present] tokens per new id
  std::vector<uint32_t> doc_off;  // [M+1]
  std::vector<uint32_t> word_off; // [n_present+1]
  std::vector<uint32_t> wt_key;   // [n] input index of each word-ordered token (host reference only)
  std::vector<uint32_t> d_cap;    // [M+1] offsets of D rows: a header, then capacity min(len, K)
  std::vector<uint32_t> ws_cap;   // [n_present-n_dense+1] offsets of sparse W rows, capacity = count
  std::vector<uint32_t> region;   // [3*n_regions] (word, begin, end)
  std::vector<uint8_t> split;     // [n_dense] 1 if the dense word has more than one region
  int64_t n_regions = 0;
  int64_t n_dense_regions = 0;
  bool key_identity = false;      // input already doc-sorted: input index == doc-order position
};

// Validates ids (word in [0, V), doc >= 0, n < 2^32); M = max doc + 1 and
// whether the input is already sorted by document.
lda_status scan_tokens(const int32_t *word, const int32_t *doc, int64_t n, int32_t V, int32_t &M, bool &doc_sorted,
                       std::string &msg);
// From the per-word token counts (caller ids) and L.doc_off: relabel, dense
// prefix, relabelled word offsets, capacities and regions.  LDA_E_RANGE for a
// document longer than LDA_MAX_DOC_LEN.
// dense_cutoff as in lda_options (0 = K, negative = all words dense)
// rows = false: relabel, dense prefix and word offsets only (no D and sparse-W
// capacities, no regions: the out-of-core chunks plan their own).
lda_status plan_from_counts(const std::vector<uint32_t> &cnt, int32_t K, int32_t R, int32_t dense_cutoff, Layout &L,
                            std::string &msg, bool rows = true);
// Regions of the words with offsets word_off (Sec. 5.1): words below nd are
// cut into ceil(count / R) regions (split[word] = 1 when more than one), the
// others form one region each, words without tokens none; split words' regions
// first, by the middle of their span, then the rest in word order.
void make_regions(const std::vector<uint32_t> &word_off, int32_t nd, int32_t R, std::vector<uint8_t> &split,
                  std::vector<uint32_t> &region, int64_t &n_dense_regions);
// All-host reference of the layout (lda_describe_layout); fills L.wt_key.
lda_status build_layout(const int32_t *word, const int32_t *doc, int64_t n, int32_t V, int32_t K, int32_t R,
                        int32_t dense_cutoff, Layout &L, std::string &msg);

// Device layout steps (layout_gpu.hip).
unsigned bits_for(uint64_t max_value);
hipError_t sort_pairs_u32(void *tmp, size_t &tmp_bytes, const uint32_t *keys_in, uint32_t *keys_out,
                          const uint32_t *vals_in, uint32_t *vals_out, int64_t n, unsigned end_bit, hipStream_t s);
hipError_t launch_gather_u32(uint32_t *dst, const int32_t *src, const uint32_t *idx, int64_t n, hipStream_t s);
hipError_t launch_boundaries(const uint32_t *keys, int64_t n, uint32_t nbins, uint32_t *off, hipStream_t s);
hipError_t launch_word_order(const uint32_t *wkey, const uint32_t *wpos, int64_t n, const int32_t *relabel,
                             const uint32_t *woff_orig, const uint32_t *woff_new, const uint32_t *doc_sorted,
                             const int32_t *doc_in, const uint32_t *dt_key, uint32_t *dt_word, uint32_t *dt_wpos,
                             const uint32_t *d_cap, uint2 *wt_kr, hipStream_t s);
hipError_t launch_scatter_z(const uint16_t *z_w, const uint2 *wt_kr, int64_t n, int32_t *z_in, hipStream_t s);
hipError_t launch_gather_z(const int32_t *z_in, const uint2 *wt_kr, int64_t n, int32_t K, uint16_t *z_w,
                           unsigned long long *bad, hipStream_t s);
// Out-of-core chunks: the word-order slot of each doc-order position from the
// positions listed in word order; the per-token arrays derived from dt_wpos
// and the chunk's regions and document tables; topics between doc order
// (int32) and word order.
hipError_t launch_invert(const uint32_t *wpos, int64_t n, uint32_t *dt_wpos, hipStream_t s);
hipError_t launch_inflate(const uint32_t *region, int64_t n_regions, const uint32_t *doc_off, const uint32_t *d_cap,
                          int32_t M, const uint32_t *dt_wpos, uint32_t key_base, uint32_t *dt_word, uint2 *wt_kr,
                          hipStream_t s);
hipError_t launch_doc_gather_z(const uint32_t *dt_wpos, const uint16_t *z_w, int64_t n, int32_t *z_doc, hipStream_t s);
hipError_t launch_doc_scatter_z(const int32_t *z_doc, const uint32_t *dt_wpos, int64_t n, int32_t K, uint16_t *z_w,
                                unsigned long long *bad, hipStream_t s);

// ---------------------------------------------------------- device state --
struct WordRec {  // per relabelled word, refreshed every iteration (Sec. 3.2, steps 1 and 4)
  double a1, a2, a3;  // top-3 values of W^[v]
  double qp;          // Q' = sum_{k != K1} alpha * W^[v][k]
  double sumw;        // sum_k W^[v][k] (log-likelihood)
  uint32_t k1, k2;    // top-2 topic ids (lowest id on ties)
};

// Per-word record of the step-3 test in single precision (the test applies a
// margin that covers the rounding, so a skip is always exact).
struct SkipRec {
  uint32_t k12;          // K1 | K2 << 16
  float a1, a2, a3, qp;  // top-3 values of W^[v] and Q' (what the test needs at g <= 2)
  uint32_t k3;           // third top topic (>= K when K < 3)
  float a4;              // fourth top value (g = 3)
  uint32_t pad;
};

// A token whose draw the tiled sampler's last pass finishes: its place in
// the region, the recorded draw, C1 and row length, D-row offset, x and the
// start of Q'.
struct TiledRec {
  uint32_t q, code, cn, off;
  double x, keep;
};

struct DevState {
  // layout
  uint32_t *doc_off, *dt_word, *dt_key, *dt_wpos, *word_off;
  uint2 *wt_kr;       // per word-ordered token: (input index = RNG key, D-row offset of its document)
  uint32_t *region;   // 3 per region
  uint32_t *heavy_docs;  // documents longer than kHeavyDoc tokens (one workgroup each in the doc kernels)
  uint8_t *split;     // per dense word
  // assignment, word order
  uint16_t *z_w;
  uint32_t *skip_bits;  // one bit per word-ordered token: the step-3 test drew K1
  uint32_t *skip_doc;   // the same decisions in document order (null when not usable)
  unsigned long long *skip_hist;  // tokens skipped at step 3 by iteration parity: [t & 1]
  // counts
  uint32_t *d_cap, *d_ent;  // D row of doc d at d_cap[d]: header (len << 16 | nnz), then entries
  int32_t *w_dense;
  uint32_t *ws_cap, *ws_nnz, *ws_ent;
  uint32_t *T;
  double *den;
  double *bden;  // beta / den[k]: W^[v][k] where W[v][k] = 0
  WordRec *wrec;
  SkipRec *wskip;
  // scheduler counters and statistics
  uint32_t *counters;           // [8]
  unsigned long long *stats;    // [8]
  double *ll_part;              // [n_regions]
  double *ll_out;               // [1]
  // large K only (the tiled sampler): per-workgroup slices of max_region
  // entries carrying a token's S' part, C1 and split chunk between passes,
  // the records of the region's tokens whose draw finishes in the last pass,
  // and the LLPT kernel's W^' rows
  double *ts_s;
  uint32_t *ts_c1, *ts_code;
  TiledRec *ts_list;
  double *wscratch;
  // large K (p.sparse_pre): topics by ascending T (descending beta/den[k]),
  // their sort buffers, and the sum of beta/den[k] over all topics
  uint32_t *topic_order, *topic_keys, *topic_iota;
  void *topic_tmp;
  size_t topic_tmp_bytes;
  double *beta_sum;
};

struct Params {
  int64_t n;
  int64_t n_all;  // tokens of the whole corpus (n is a chunk's share in the out-of-core mode)
  int32_t M, V, K, n_present, n_dense;
  int64_t n_regions;
  double alpha, beta, vbeta;
  float alpha_f;
  uint64_t seed;
  int32_t g;
  int32_t no_skip;
  int32_t two_branch;  // Sec. 2.2 sampling over [S | Q]: no max-topic branch, no skip test
  int32_t key_identity;
  int32_t grid_regions;  // persistent workgroups for region kernels
  int32_t sampler_block; // threads per sampler workgroup: 256, 512 or 1024
  int32_t grid_docs;     // persistent workgroups for doc kernels
  int32_t big_k;         // the W^' row does not fit LDS: tiled sampler, LDS-light rebuilds (K <= 32768)
  int32_t tile_topics;   // topics per tile of the tiled sampler (a multiple of 16)
  int32_t max_region;    // tokens of the largest region
  int32_t doc_waves;     // waves per workgroup of the doc pass and the D rebuild (LDS tables of K entries per wave)
  int32_t sparse_pre;    // per-word precompute of sparse words from their row and a topic list (large K)
  int32_t top_list;      // length of that topic list
  int32_t skip_marks;    // 0 auto, 1 word-ordered bitmap, 2 document-ordered bitmap (lda_options)
  int32_t always_skip_test;  // steps 2-3 every iteration instead of when they pay (lda_options)
  uint32_t key_base;     // out-of-core chunks: input index of the chunk's first doc-ordered token (else 0)
  int32_t n_heavy;       // entries of heavy_docs
  int64_t light_begin;   // regions [light_begin, n_regions): light words, one wave each in the sampler
  int32_t doc_marks_ok;  // the document-ordered bitmap is usable: keys are document positions, regular sampler
  int32_t q_table;       // the sampler keeps the Q' blocks' partial sums in LDS (search instead of walk)
  uint32_t xcd_doc[kXcds + 1];  // document ranges with equal token counts, one per XCD (D rebuild)
};

// Scheduler counters: one each for the region kernels and the doc pass,
// kXcds (one per document range) for the D rebuild.
enum { CNT_SAMPLER = 0, CNT_DOCPASS = 2, CNT_LOGLIK = 4, CNT_HEAVY_PASS = 5,
       CNT_HEAVY_REBUILD = 6, CNT_LIGHT = 7, CNT_REBUILD_D = 16 };
constexpr int kCounters = 32;
enum { ST_SKIP3 = 0, ST_SKIP_AFTER_S = 1, ST_SAMPLED = 2, ST_NNZ = 3, ST_REGIONS = 4, ST_DENSE_REGIONS = 5, ST_ERRORS = 6,
       ST_ROW_BYTES = 7, ST_MARKS = 8, ST_TEST_RAN = 9 };
constexpr int kStatsPerIter = 16;

// Kernel launchers (all asynchronous on `s`); return hipGetLastError().
hipError_t launch_init_topics(const DevState &d, const Params &p, hipStream_t s);
hipError_t launch_begin_iteration(const DevState &d, const Params &p, hipStream_t s);
hipError_t launch_word_pre(const DevState &d, const Params &p, hipStream_t s);
hipError_t launch_beta_sum(const DevState &d, const Params &p, hipStream_t s);
// reset_count: also clear this iteration's skip count (false for the second
// and later chunks of an out-of-core iteration, which add to it)
hipError_t launch_clear_skips(const DevState &d, const Params &p, uint32_t t, hipStream_t s, bool reset_count = true);
hipError_t launch_reset_counters(uint32_t *counters, hipStream_t s);
hipError_t launch_doc_pass(const DevState &d, const Params &p, uint32_t t, hipStream_t s);
// The sampler of the regions before p.light_begin (or every region with the
// tiled sampler), and that of the light regions, one wave each (nothing when
// there are none); the two touch disjoint topic slots and may run at once.
hipError_t launch_sampler(const DevState &d, const Params &p, uint32_t t, hipStream_t s);
hipError_t launch_sampler_light(const DevState &d, const Params &p, uint32_t t, hipStream_t s);
int sampler_block(int K, int want, bool *q_table);
// The sampler's dynamic LDS for K topics and workgroups of nb threads.
size_t sampler_lds_bytes(int K, int nb, bool q_table);
// Regions of at most this many tokens (one batch of the sampler) are light:
// a wave takes each of them, when the per-wave W^' row is small (K up to
// about 2,000).  They form a suffix of the region table, which lists the
// unsplit words by descending token count after the split ones.
constexpr uint32_t kLightTokens = 64;
constexpr size_t kLightLdsMax = 20 * 1024;
inline int64_t light_region_start(const std::vector<uint32_t> &region, int K, bool big_k) {
  int64_t r = int64_t(region.size() / 3);
  if (big_k || sampler_lds_bytes(K, 64, true) > kLightLdsMax) return r;
  while (r > 0 && region[3 * size_t(r - 1) + 2] - region[3 * size_t(r - 1) + 1] <= kLightTokens) --r;
  return r;
}
// Large K: topics per tile and the tiled sampler's dynamic LDS.
int tiled_topics(int K);
size_t tiled_lds_bytes(int K, int kt);
constexpr int kTiledThreads = 1024;
// Workgroups of the tiled sampler (one per CU: its LDS fills a CU) and of the
// large-K LLPT kernel; the scratch slices are sized for these grids.
inline int tiled_grid(const Params &p) { return p.grid_regions / 8 > 0 ? p.grid_regions / 8 : 1; }
inline int loglik_grid_big_k(const Params &p) { return tiled_grid(p); }
// The W rebuild by bitmap, with T from a histogram of the topics (and its
// scratch rows), from this many topics on: below it a workgroup's tables of K
// counts are small enough to keep several workgroups on a CU.
constexpr int kWBitsK = 4096;
inline bool w_bits(const Params &p) { return p.big_k || p.K >= kWBitsK; }
// The count rebuild (Sec. 4.3): launch_rebuild = launch_zero_split, then
// launch_rebuild_w and launch_rebuild_d.
hipError_t launch_rebuild(const DevState &d, const Params &p, hipStream_t s);
hipError_t launch_zero_split(const DevState &d, const Params &p, hipStream_t s);
hipError_t launch_rebuild_w(const DevState &d, const Params &p, hipStream_t s);
hipError_t launch_rebuild_d(const DevState &d, const Params &p, hipStream_t s);
hipError_t launch_loglik(const DevState &d, const Params &p, hipStream_t s);
// out[0] = sum of part[0..n) in a fixed order (one workgroup).
hipError_t launch_sum_f64(const double *part, int64_t n, double *out, hipStream_t s);
// Allocation-free LLPT: the layout of the fixed scratch array (counters at 0,
// the result at kNoAllocResult, out-of-core per-chunk sums at
// kNoAllocChunkSums, per-region partials from kNoAllocHead), its
// device address on the current device (looked up once per device), and the
// LLPT launches on it.  hipErrorInvalidValue past LDA_NOALLOC_MAX_REGIONS.
constexpr size_t kNoAllocResult = 256;
constexpr size_t kNoAllocChunkSums = 512;
constexpr size_t kNoAllocHead = 4096;
static_assert(kNoAllocChunkSums + sizeof(double) * LDA_MAX_CHUNKS <= kNoAllocHead, "chunk sums overlap the partials");
static_assert(sizeof(uint32_t) * kCounters <= kNoAllocResult, "counters overlap the result");
hipError_t noalloc_scratch_address(void **out);
hipError_t launch_loglik_noalloc(DevState d, const Params &p, void *scratch_dev, hipStream_t s);
hipError_t launch_sum_nnz(const DevState &d, const Params &p, unsigned long long *out, hipStream_t s);

}  // namespace lda
