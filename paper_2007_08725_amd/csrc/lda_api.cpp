// C ABI of liblda (include/lda.h): handle lifetime, validation, device
// memory, the per-iteration launch sequence and the host-side exports.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <numeric>
#include <string>
#include <vector>

#include "handle.h"

using namespace lda;

namespace lda {
thread_local std::string g_create_error = "no error";
}  // namespace lda

namespace {

// Count tables of the current assignment z_w (Sec. 4.3 update step).
lda_status rebuild_counts(lda_handle *h) {
  DevState d = h->d;
  d.stats = h->stats_base;
  HIP_TRY(h, launch_begin_iteration(d, h->p, h->stream));
  HIP_TRY(h, launch_rebuild(d, h->p, h->stream));
  return LDA_OK;
}

}  // namespace

namespace lda {

// Stream, workgroup sizes and grids for this device and K (both modes).
lda_status setup_device(lda_handle *h, const lda_options *o) {
  Layout &L = h->L;
  HIP_TRY(h, hipGetDevice(&h->device));
  int cus = 0, lds_max = 0;
  HIP_TRY(h, hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, h->device));
  HIP_TRY(h, hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device));
  if (o && o->stream) {
    h->stream = static_cast<hipStream_t>(o->stream);
  } else {
    HIP_TRY(h, hipStreamCreateWithFlags(&h->stream, hipStreamNonBlocking));
    h->own_stream = true;
  }
  HIP_TRY(h, hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking));
  HIP_TRY(h, hipEventCreateWithFlags(&h->fork_ev, hipEventDisableTiming));
  HIP_TRY(h, hipEventCreateWithFlags(&h->join_ev, hipEventDisableTiming));
  // the fixed scratch of the allocation-free LLPT, looked up once per device
  HIP_TRY(h, noalloc_scratch_address(&h->noalloc_scratch));
  Params &p = h->p;
  p.grid_regions = std::max(1, cus * 8);
  const int want = o ? o->sampler_block : 0;
  bool q_table = false;
  p.sampler_block = sampler_block(p.K, want, &q_table);
  p.q_table = q_table ? 1 : 0;
  if (!p.sampler_block && want)
    return fail(h, LDA_E_RANGE, "no sampler workgroup of " + std::to_string(want) + " threads fits the LDS of K = " +
                                    std::to_string(L.K));
  if (!p.sampler_block) {
    // the W^' row does not fit one workgroup's LDS: the tiled sampler
    p.big_k = 1;
    p.tile_topics = tiled_topics(p.K);
    p.sampler_block = kTiledThreads;
    if (tiled_lds_bytes(p.K, p.tile_topics) > size_t(lds_max))
      return fail(h, LDA_E_RANGE, "K = " + std::to_string(L.K) + " needs " +
                                      std::to_string(tiled_lds_bytes(p.K, p.tile_topics)) +
                                      " bytes of LDS per workgroup even in tiles; the device allows " +
                                      std::to_string(lds_max));
  }
  // the doc pass keeps a table of K 16-bit counts per wave; the D rebuild
  // the same table plus a bitmap of the touched topics and a list of them.
  // Waves per workgroup: the count that keeps the most waves running on a CU
  // (the larger on a tie), given that the LDS fits lds_max / (w * table)
  // workgroups and the D rebuild's grid offers 4 per CU: 3 at K = 10,000,
  // where 4 waves would fit one workgroup per CU and 3 fit two
  {
    const size_t wave_bytes = sizeof(uint32_t) * d_rebuild_lds_words(p.K);
    int best = 1, best_res = 0;
    for (int w = 1; w <= kBlock / 64; ++w) {
      const int res = w * std::min(4, int(size_t(lds_max) / (size_t(w) * wave_bytes)));
      if (res >= best_res && res > 0) {
        best = w;
        best_res = res;
      }
    }
    p.doc_waves = best;
  }
  p.grid_docs = std::max(1, cus * 8);
  return LDA_OK;
}

}  // namespace lda

namespace {

// Device layout (Sec. 4.2-4.3, 5.1): both token orders are built with radix
// sorts on the GPU; only per-word and per-document counts visit the host.
lda_status create_device(lda_handle *h, const lda_options *o, const int32_t *word, const int32_t *doc, int32_t R,
                         int32_t dense_cutoff) {
  Layout &L = h->L;
  LDA_TRY(setup_device(h, o));
  if (h->chunks_wanted > 1) return chunked_create(h, word, doc, R, h->chunks_wanted);
  Params &p = h->p;
  const size_t n = size_t(L.n);
  const bool identity = L.key_identity;
  DevState &d = h->d;

  // 1. the token list on the device
  int32_t *word_d = nullptr, *doc_d = nullptr;
  LDA_TRY(dalloc(h, &word_d, n));
  LDA_TRY(dalloc(h, &doc_d, n));
  HIP_TRY(h, hipMemcpyAsync(word_d, word, n * 4, hipMemcpyHostToDevice, h->stream));
  HIP_TRY(h, hipMemcpyAsync(doc_d, doc, n * 4, hipMemcpyHostToDevice, h->stream));

  // 2. doc order: stable sort of input indices by document
  uint32_t *doc_sorted = nullptr;
  if (!identity) {
    LDA_TRY(dalloc(h, &doc_sorted, n));
    LDA_TRY(dalloc(h, &d.dt_key, n));
    LDA_TRY(sort_pairs(h, reinterpret_cast<const uint32_t *>(doc_d), doc_sorted, nullptr, d.dt_key,
                       bits_for(uint64_t(L.M) - 1)));
  }
  const uint32_t *doc_keys = identity ? reinterpret_cast<const uint32_t *>(doc_d) : doc_sorted;
  LDA_TRY(dalloc(h, &d.doc_off, size_t(L.M) + 1));
  HIP_TRY(h, launch_boundaries(doc_keys, L.n, uint32_t(L.M), d.doc_off, h->stream));

  // 3. caller word ids in doc order, stably sorted by word
  uint32_t *w_orig = nullptr;
  if (!identity) {
    LDA_TRY(dalloc(h, &w_orig, n));
    HIP_TRY(h, launch_gather_u32(w_orig, word_d, d.dt_key, L.n, h->stream));
  }
  uint32_t *wkey = nullptr, *wpos = nullptr, *woff_orig = nullptr;
  LDA_TRY(dalloc(h, &wkey, n));
  LDA_TRY(dalloc(h, &wpos, n));
  LDA_TRY(sort_pairs(h, identity ? reinterpret_cast<const uint32_t *>(word_d) : w_orig, wkey, nullptr, wpos,
                     bits_for(uint64_t(L.V) - 1)));
  dfree(h, w_orig);
  LDA_TRY(dalloc(h, &woff_orig, size_t(L.V) + 1));
  HIP_TRY(h, launch_boundaries(wkey, L.n, uint32_t(L.V), woff_orig, h->stream));

  // 4. counts to the host: relabel, capacities and regions
  std::vector<uint32_t> woff_h(size_t(L.V) + 1);
  L.doc_off.resize(size_t(L.M) + 1);
  HIP_TRY(h, hipMemcpyAsync(woff_h.data(), woff_orig, woff_h.size() * 4, hipMemcpyDeviceToHost, h->stream));
  HIP_TRY(h, hipMemcpyAsync(L.doc_off.data(), d.doc_off, L.doc_off.size() * 4, hipMemcpyDeviceToHost, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  std::vector<uint32_t> cnt(static_cast<size_t>(L.V));
  for (int32_t v = 0; v < L.V; ++v) cnt[size_t(v)] = woff_h[size_t(v) + 1] - woff_h[size_t(v)];
  std::string msg;
  lda_status st = plan_from_counts(cnt, L.K, R, dense_cutoff, L, msg);
  if (st != LDA_OK) return fail(h, st, msg);
  // document ranges of equal token counts for the document kernels, one per XCD
  p.xcd_doc[0] = 0;
  for (int x = 1; x < kXcds; ++x) {
    const uint64_t target = uint64_t(L.n) * uint64_t(x) / uint64_t(kXcds);
    p.xcd_doc[x] = uint32_t(std::lower_bound(L.doc_off.begin(), L.doc_off.end(), uint32_t(target)) - L.doc_off.begin());
    p.xcd_doc[x] = std::min<uint32_t>(std::max(p.xcd_doc[x], p.xcd_doc[x - 1]), uint32_t(L.M));
  }
  p.xcd_doc[kXcds] = uint32_t(L.M);
  p.n_present = L.n_present;
  p.n_dense = L.n_dense;
  p.n_regions = L.n_regions;
  p.light_begin = light_region_start(L.region, L.K, p.big_k != 0);

  // 5. word order in relabelled ids and the links between the two orders
  int32_t *relabel_d = nullptr;
  LDA_TRY(dalloc(h, &relabel_d, size_t(L.V)));
  LDA_TRY(dalloc(h, &d.word_off, L.word_off.size()));
  LDA_TRY(upload(h, relabel_d, L.relabel));
  LDA_TRY(upload(h, d.word_off, L.word_off));
  LDA_TRY(dalloc(h, &d.dt_word, n));
  LDA_TRY(dalloc(h, &d.dt_wpos, n));
  LDA_TRY(dalloc(h, &d.wt_kr, n));
  LDA_TRY(dalloc(h, &d.d_cap, L.d_cap.size()));
  LDA_TRY(upload(h, d.d_cap, L.d_cap));
  HIP_TRY(h, launch_word_order(wkey, wpos, L.n, relabel_d, woff_orig, d.word_off, doc_sorted, doc_d, d.dt_key,
                               d.dt_word, d.dt_wpos, d.d_cap, d.wt_kr, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  dfree(h, relabel_d);
  dfree(h, woff_orig);
  dfree(h, wpos);
  dfree(h, wkey);
  dfree(h, doc_sorted);
  dfree(h, doc_d);
  dfree(h, word_d);

  // 6. count tables and scheduler state
  LDA_TRY(dalloc(h, &d.region, L.region.size()));
  {
    // heavy documents: one workgroup each in the doc pass and the D rebuild (Sec. 5.1)
    const std::vector<uint32_t> heavy = heavy_documents(L.doc_off.data(), uint32_t(L.M));
    p.n_heavy = int32_t(heavy.size());
    LDA_TRY(dalloc(h, &d.heavy_docs, heavy.size()));
    LDA_TRY(upload(h, d.heavy_docs, heavy));
  }
  LDA_TRY(dalloc(h, &d.split, L.split.size()));
  LDA_TRY(dalloc(h, &d.z_w, n));
  LDA_TRY(dalloc(h, &d.skip_bits, skip_words(int64_t(n))));
  // the document-ordered skip bitmap (bit = the token's key, which is its
  // document position when the input is sorted by document; 64 spare words
  // for the 3-word writes of a document's last chunk) and the per-parity skip
  // counts that choose between the two bitmaps
  p.doc_marks_ok = (identity && !p.big_k) ? 1 : 0;
  d.skip_doc = nullptr;
  if (p.doc_marks_ok) LDA_TRY(dalloc(h, &d.skip_doc, size_t(skip_words(int64_t(n))) + 64));
  LDA_TRY(dalloc(h, &d.skip_hist, 2));
  HIP_TRY(h, hipMemsetAsync(d.skip_hist, 0, 2 * sizeof(unsigned long long), h->stream));
  LDA_TRY(dalloc(h, &d.d_ent, size_t(L.d_cap.back()) + kRowPad));
  LDA_TRY(dalloc(h, &d.w_dense, size_t(L.n_dense) * size_t(L.K)));
  LDA_TRY(dalloc(h, &d.ws_cap, L.ws_cap.size()));
  LDA_TRY(dalloc(h, &d.ws_nnz, L.ws_cap.size()));
  LDA_TRY(dalloc(h, &d.ws_ent, size_t(L.ws_cap.back())));
  LDA_TRY(dalloc(h, &d.T, size_t(L.K)));
  LDA_TRY(dalloc(h, &d.den, size_t(L.K)));
  LDA_TRY(dalloc(h, &d.bden, size_t(L.K)));
  LDA_TRY(dalloc(h, &d.wrec, size_t(L.n_present)));
  LDA_TRY(dalloc(h, &d.wskip, size_t(L.n_present)));
  LDA_TRY(dalloc(h, &d.counters, kCounters));
  LDA_TRY(dalloc(h, &h->stats_base, size_t(kStatSlots) * kStatsPerIter));
  LDA_TRY(dalloc(h, &d.ll_part, size_t(L.n_regions)));
  // large K: sparse words' per-word records from their rows and a list of
  // the topics with the largest beta/den[k] (sorted each iteration)
  p.sparse_pre = L.K >= 4096 ? 1 : 0;
  p.top_list = std::min(L.K, 512);
  if (p.sparse_pre) {
    LDA_TRY(dalloc(h, &d.topic_order, size_t(L.K)));
    LDA_TRY(dalloc(h, &d.topic_keys, size_t(L.K)));
    LDA_TRY(dalloc(h, &d.topic_iota, size_t(L.K)));
    LDA_TRY(dalloc(h, &d.beta_sum, 1));
    std::vector<uint32_t> iota(static_cast<size_t>(L.K));
    std::iota(iota.begin(), iota.end(), 0u);
    LDA_TRY(upload(h, d.topic_iota, iota));
    HIP_TRY(h, sort_pairs_u32(nullptr, d.topic_tmp_bytes, d.T, d.topic_keys, d.topic_iota, d.topic_order,
                              L.K, 32, h->stream));
    uint8_t *tmp = nullptr;
    LDA_TRY(dalloc(h, &tmp, d.topic_tmp_bytes));
    d.topic_tmp = tmp;
  }
  uint32_t max_region = 1;
  for (size_t r = 0; r < L.region.size(); r += 3) max_region = std::max(max_region, L.region[r + 2] - L.region[r + 1]);
  p.max_region = int32_t(max_region);
  if (p.big_k) {
    const size_t slots = size_t(tiled_grid(p)) * size_t(max_region);
    LDA_TRY(dalloc(h, &d.ts_s, slots));
    LDA_TRY(dalloc(h, &d.ts_c1, slots));
    LDA_TRY(dalloc(h, &d.ts_code, slots));
    LDA_TRY(dalloc(h, &d.ts_list, slots));
  }
  if (w_bits(p)) LDA_TRY(dalloc(h, &d.wscratch, size_t(loglik_grid_big_k(p)) * size_t(L.K)));
  LDA_TRY(dalloc(h, &d.ll_out, 1));
  d.stats = h->stats_base;
  LDA_TRY(upload(h, d.region, L.region));
  LDA_TRY(upload(h, d.split, L.split));
  LDA_TRY(upload(h, d.ws_cap, L.ws_cap));
  HIP_TRY(h, hipMemsetAsync(h->stats_base, 0, sizeof(unsigned long long) * kStatSlots * kStatsPerIter, h->stream));
  HIP_TRY(h, launch_init_topics(d, p, h->stream));
  LDA_TRY(rebuild_counts(h));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  unsigned long long stt[kStatsPerIter];
  HIP_TRY(h, hipMemcpy(stt, h->stats_base, sizeof(stt), hipMemcpyDeviceToHost));
  LDA_TRY(check_errors(h, stt));
  std::vector<uint32_t>().swap(L.region);
  return LDA_OK;
}

void release(lda_handle *h) {
  if (!h) return;
  if (h->stream) (void)hipStreamSynchronize(h->stream);
  h->chunks.reset();  // drains the copy streams before the device memory goes
  if (h->side) (void)hipStreamSynchronize(h->side);
  for (hipEvent_t ev : {h->fork_ev, h->join_ev})
    if (ev) (void)hipEventDestroy(ev);
  if (h->side) (void)hipStreamDestroy(h->side);
  for (hipEvent_t ev : h->events)
    if (ev) (void)hipEventDestroy(ev);
  for (void *ptr : h->allocations) {
    if (h->dev_alloc) h->dev_free(ptr, h->alloc_ctx);
    else (void)hipFree(ptr);
  }
  if (h->own_stream && h->stream) (void)hipStreamDestroy(h->stream);
  delete h;
}

}  // namespace

extern "C" {

lda_status lda_create(const int32_t *word, const int32_t *doc, int64_t n_tokens, int32_t V, int32_t K, double alpha,
                      double beta, uint64_t seed, const lda_options *opts, lda_handle **out) {
  if (!out) return fail(nullptr, LDA_E_ARG, "out is NULL");
  *out = nullptr;
  if (!word || !doc) return fail(nullptr, LDA_E_ARG, "word or doc is NULL");
  if (n_tokens <= 0) return fail(nullptr, LDA_E_ARG, "n_tokens must be positive");
  if (V <= 0) return fail(nullptr, LDA_E_ARG, "V must be positive");
  if (K < 2 || K > LDA_MAX_TOPICS) return fail(nullptr, LDA_E_ARG, "K must be in [2, 32768]");
  if (!std::isfinite(alpha) || !(alpha > 0.0)) return fail(nullptr, LDA_E_ARG, "alpha must be finite and positive");
  if (!std::isfinite(beta) || !(beta > 0.0)) return fail(nullptr, LDA_E_ARG, "beta must be finite and positive");
  int32_t g = 2, R = kDefaultRegionTokens, no_skip = 0, dense_cutoff = 0, two_branch = 0, skip_marks = 0;
  int32_t always_skip_test = 0, chunks = 0;
  if (opts) {
    if (opts->g < 0 || opts->g > 3) return fail(nullptr, LDA_E_ARG, "g must be 1, 2 or 3");
    if (opts->g) g = opts->g;
    if (opts->region_tokens < 0) return fail(nullptr, LDA_E_ARG, "region_tokens must be >= 0");
    if (opts->region_tokens) R = opts->region_tokens;
    if ((opts->dev_alloc == nullptr) != (opts->dev_free == nullptr))
      return fail(nullptr, LDA_E_ARG, "dev_alloc and dev_free must be given together");
    no_skip = opts->no_skip ? 1 : 0;
    dense_cutoff = opts->dense_cutoff;
    two_branch = opts->two_branch ? 1 : 0;
    if (two_branch) no_skip = 1;  // the skip test needs the max-topic branch
    const int32_t sb = opts->sampler_block;
    if (sb != 0 && sb != 256 && sb != 512 && sb != 1024)
      return fail(nullptr, LDA_E_ARG, "sampler_block must be 0, 256, 512 or 1024");
    if (opts->skip_marks < 0 || opts->skip_marks > 2) return fail(nullptr, LDA_E_ARG, "skip_marks must be 0, 1 or 2");
    skip_marks = opts->skip_marks;
    if (opts->always_skip_test < 0 || opts->always_skip_test > 1)
      return fail(nullptr, LDA_E_ARG, "always_skip_test must be 0 or 1");
    always_skip_test = opts->always_skip_test;
    if (opts->chunks < 0 || opts->chunks > LDA_MAX_CHUNKS)
      return fail(nullptr, LDA_E_ARG, "chunks must be in [0, " + std::to_string(LDA_MAX_CHUNKS) + "]");
    chunks = opts->chunks;
  }
  lda_handle *h = new (std::nothrow) lda_handle();
  if (!h) return fail(nullptr, LDA_E_NOMEM, "host allocation failed");
  std::string msg;
  int32_t M = 0;
  bool sorted = false;
  lda_status st = scan_tokens(word, doc, n_tokens, V, M, sorted, msg);
  if (st != LDA_OK) {
    delete h;
    return fail(nullptr, st, msg);
  }
  h->L.n = n_tokens;
  h->L.V = V;
  h->L.K = K;
  h->L.M = M;
  h->L.key_identity = sorted;
  if (chunks > 1 && !sorted) {
    delete h;
    return fail(nullptr, LDA_E_ARG, "chunks need the input sorted by document");
  }
  h->chunks_wanted = chunks;
  if (opts) {
    h->dev_alloc = opts->dev_alloc;
    h->dev_free = opts->dev_free;
    h->alloc_ctx = opts->alloc_ctx;
  }
  Params &p = h->p;
  p.n = n_tokens;
  p.n_all = n_tokens;
  p.M = M;
  p.V = V;
  p.K = K;
  p.alpha = alpha;
  p.alpha_f = float(alpha);
  p.beta = beta;
  p.vbeta = double(V) * beta;
  p.seed = seed;
  p.g = g;
  p.no_skip = no_skip;
  p.two_branch = two_branch;
  p.key_identity = sorted ? 1 : 0;
  p.skip_marks = skip_marks;
  p.always_skip_test = always_skip_test;
  try {
    st = create_device(h, opts, word, doc, R, dense_cutoff);
  } catch (const std::bad_alloc &) {
    st = fail(h, LDA_E_NOMEM, "host allocation failed");
  }
  if (st != LDA_OK) {
    g_create_error = h->err;
    release(h);
    return st;
  }
  *out = h;
  return LDA_OK;
}

lda_status lda_iterate(lda_handle *h, int32_t n_iters, lda_iter_stats *stats) {
  LDA_TRY(check_handle(h));
  if (n_iters < 0) return fail(h, LDA_E_ARG, "n_iters must be >= 0");
  if (h->chunks) return chunked_iterate(h, n_iters, stats);
  if (stats && h->events.empty()) {
    h->events.assign(size_t(kStatSlots) * kEventsPerIter, nullptr);
    for (auto &ev : h->events) HIP_TRY(h, hipEventCreate(&ev));
  }
  for (int32_t done = 0; done < n_iters;) {
    const int32_t chunk = std::min<int32_t>(n_iters - done, kStatSlots);
    for (int32_t c = 0; c < chunk; ++c) {
      const uint32_t t = uint32_t(h->iteration);
      DevState d = h->d;
      d.stats = h->stats_base + size_t(c) * kStatsPerIter;
      hipEvent_t *ev = stats ? &h->events[size_t(c) * kEventsPerIter] : nullptr;
      if (ev) HIP_TRY(h, hipEventRecord(ev[0], h->stream));
      HIP_TRY(h, launch_begin_iteration(d, h->p, h->stream));
      HIP_TRY(h, launch_word_pre(d, h->p, h->stream));
      HIP_TRY(h, launch_clear_skips(d, h->p, t, h->stream));
      if (ev) HIP_TRY(h, hipEventRecord(ev[1], h->stream));
      if (!h->p.no_skip) HIP_TRY(h, launch_doc_pass(d, h->p, t, h->stream));  // steps 2-3 only decide skips
      if (ev) HIP_TRY(h, hipEventRecord(ev[2], h->stream));
      LDA_TRY(run_sampler(h, d, h->p, t));
      if (ev) HIP_TRY(h, hipEventRecord(ev[3], h->stream));
      HIP_TRY(h, launch_rebuild(d, h->p, h->stream));
      if (ev) HIP_TRY(h, hipEventRecord(ev[4], h->stream));
      h->iteration++;
    }
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    std::vector<unsigned long long> st(static_cast<size_t>(chunk) * kStatsPerIter);
    HIP_TRY(h, hipMemcpy(st.data(), h->stats_base, st.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost));
    for (int32_t c = 0; c < chunk; ++c) {
      const unsigned long long *s = &st[size_t(c) * kStatsPerIter];
      LDA_TRY(check_errors(h, s));
      if (!stats) continue;
      lda_iter_stats &o = stats[done + c];
      hipEvent_t *ev = &h->events[size_t(c) * kEventsPerIter];
      float ms_all = 0, ms_pre = 0, ms_doc = 0, ms_smp = 0, ms_reb = 0;
      HIP_TRY(h, hipEventElapsedTime(&ms_all, ev[0], ev[4]));
      HIP_TRY(h, hipEventElapsedTime(&ms_pre, ev[0], ev[1]));
      HIP_TRY(h, hipEventElapsedTime(&ms_doc, ev[1], ev[2]));
      HIP_TRY(h, hipEventElapsedTime(&ms_smp, ev[2], ev[3]));
      HIP_TRY(h, hipEventElapsedTime(&ms_reb, ev[3], ev[4]));
      o.iteration = h->iteration - chunk + c;
      o.ms_iter = ms_all;
      o.ms_docpass = ms_doc;
      o.ms_sampler = ms_smp;
      o.ms_rebuild = ms_reb;
      o.ms_precompute = ms_pre;
      o.skip_step3 = int64_t(s[ST_SKIP3]);
      o.skip_after_s = int64_t(s[ST_SKIP_AFTER_S]);
      o.sampled = int64_t(s[ST_SAMPLED]);
      o.nnz_scanned = int64_t(s[ST_NNZ]);
      o.regions = int64_t(s[ST_REGIONS]);
      o.dense_regions = int64_t(s[ST_DENSE_REGIONS]);
      o.row_bytes = int64_t(s[ST_ROW_BYTES]);
      o.sampler_block = h->p.sampler_block;
      o.skip_marks = int64_t(s[ST_MARKS]);
      o.skip_test_ran = int64_t(s[ST_TEST_RAN]);
    }
    done += chunk;
  }
  return LDA_OK;
}

lda_status lda_get_counts(lda_handle *h, lda_counts *out) {
  LDA_TRY(check_handle(h));
  if (!out) return fail(h, LDA_E_ARG, "out is NULL");
  if (h->chunks) return chunked_counts(h, out);
  const Layout &L = h->L;
  const size_t n = size_t(L.n);
  const int32_t K = L.K;
  std::vector<uint32_t> ws_nnz(L.ws_cap.size() - 1);
  unsigned long long *nnz_dev = nullptr;
  LDA_TRY(dalloc(h, &nnz_dev, 1));
  HIP_TRY(h, hipMemsetAsync(nnz_dev, 0, sizeof(unsigned long long), h->stream));
  HIP_TRY(h, launch_sum_nnz(h->d, h->p, nnz_dev, h->stream));
  unsigned long long nnz_D_dev = 0;
  HIP_TRY(h, hipMemcpyAsync(&nnz_D_dev, nnz_dev, sizeof(nnz_D_dev), hipMemcpyDeviceToHost, h->stream));
  if (!ws_nnz.empty())
    HIP_TRY(h, hipMemcpyAsync(ws_nnz.data(), h->d.ws_nnz, ws_nnz.size() * 4, hipMemcpyDeviceToHost, h->stream));
  std::vector<int32_t> wd(static_cast<size_t>(L.n_dense) * static_cast<size_t>(K));
  if (!wd.empty())
    HIP_TRY(h, hipMemcpyAsync(wd.data(), h->d.w_dense, wd.size() * 4, hipMemcpyDeviceToHost, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  dfree(h, nnz_dev);
  int64_t nnz_D = int64_t(nnz_D_dev), nnz_W = 0;
  for (uint32_t x : ws_nnz) nnz_W += x;
  for (int32_t x : wd) nnz_W += x != 0;
  out->iteration = h->iteration;
  out->M = L.M;
  out->V = L.V;
  out->K = K;
  out->n_tokens = L.n;
  out->nnz_D = nnz_D;
  out->nnz_W = nnz_W;
  if (!out->z && !out->T && !out->D_off && !out->D_topic && !out->D_count && !out->W_off && !out->W_topic &&
      !out->W_count)
    return LDA_OK;  // size query
  if (out->z) {
    int32_t *zin = nullptr;
    LDA_TRY(dalloc(h, &zin, n));
    HIP_TRY(h, launch_scatter_z(h->d.z_w, h->d.wt_kr, L.n, zin, h->stream));
    HIP_TRY(h, hipMemcpyAsync(out->z, zin, n * 4, hipMemcpyDeviceToHost, h->stream));
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    dfree(h, zin);
  }
  if (out->T) {
    std::vector<uint32_t> tk(static_cast<size_t>(K));
    HIP_TRY(h, hipMemcpy(tk.data(), h->d.T, size_t(K) * 4, hipMemcpyDeviceToHost));
    for (int32_t k = 0; k < K; ++k) out->T[k] = tk[size_t(k)];
  }
  if (out->D_off || out->D_topic || out->D_count) {
    if (!out->D_off || !out->D_topic || !out->D_count) return fail(h, LDA_E_ARG, "D arrays must be given together");
    std::vector<uint32_t> ent(static_cast<size_t>(L.d_cap.back()));
    if (!ent.empty()) HIP_TRY(h, hipMemcpy(ent.data(), h->d.d_ent, ent.size() * 4, hipMemcpyDeviceToHost));
    int64_t o = 0;
    for (int32_t dd = 0; dd < L.M; ++dd) {
      out->D_off[dd] = o;
      const uint32_t hdr = ent[size_t(L.d_cap[size_t(dd)])];
      for (uint32_t q = 0; q < (hdr & 0xFFFFu); ++q) {
        const uint32_t e = ent[size_t(L.d_cap[size_t(dd)]) + 1 + q];
        out->D_topic[o] = int32_t(e >> 16);
        out->D_count[o] = int32_t(e & 0xFFFFu);
        ++o;
      }
    }
    out->D_off[L.M] = o;
  }
  if (out->W_off || out->W_topic || out->W_count) {
    if (!out->W_off || !out->W_topic || !out->W_count) return fail(h, LDA_E_ARG, "W arrays must be given together");
    std::vector<uint32_t> went(static_cast<size_t>(L.ws_cap.back()));
    if (!went.empty()) HIP_TRY(h, hipMemcpy(went.data(), h->d.ws_ent, went.size() * 4, hipMemcpyDeviceToHost));
    int64_t o = 0;
    for (int32_t v = 0; v < L.V; ++v) {
      out->W_off[v] = o;
      const int32_t r = L.relabel[size_t(v)];
      if (r >= L.n_present) continue;
      if (r < L.n_dense) {
        const int32_t *row = &wd[size_t(r) * size_t(K)];
        for (int32_t k = 0; k < K; ++k)
          if (row[k]) {
            out->W_topic[o] = k;
            out->W_count[o] = row[k];
            ++o;
          }
      } else {
        const size_t s = size_t(r - L.n_dense);
        for (uint32_t q = 0; q < ws_nnz[s]; ++q) {
          const uint32_t e = went[size_t(L.ws_cap[s]) + q];
          out->W_topic[o] = int32_t(e >> 16);
          out->W_count[o] = int32_t(e & 0xFFFFu);
          ++o;
        }
      }
    }
    out->W_off[L.V] = o;
  }
  return LDA_OK;
}

lda_status lda_loglik(lda_handle *h, double *llpt) {
  LDA_TRY(check_handle(h));
  if (!llpt) return fail(h, LDA_E_ARG, "llpt is NULL");
  if (h->chunks) return chunked_loglik(h, llpt, nullptr);
  DevState d = h->d;
  d.stats = h->stats_base;
  HIP_TRY(h, launch_begin_iteration(d, h->p, h->stream));
  HIP_TRY(h, launch_word_pre(d, h->p, h->stream));
  HIP_TRY(h, launch_loglik(d, h->p, h->stream));
  double sum = 0.0;
  HIP_TRY(h, hipMemcpyAsync(&sum, h->d.ll_out, sizeof(double), hipMemcpyDeviceToHost, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  *llpt = sum / double(h->L.n);
  return LDA_OK;
}

lda_status lda_loglik_noalloc(lda_handle *h, double *llpt) {
  LDA_TRY(check_handle(h));
  if (!llpt) return fail(h, LDA_E_ARG, "llpt is NULL");
  if (h->chunks) return chunked_loglik(h, llpt, h->noalloc_scratch);
  if (h->p.n_regions > int64_t(LDA_NOALLOC_MAX_REGIONS))
    return fail(h, LDA_E_RANGE, "lda_loglik_noalloc holds partial sums for at most " +
                                    std::to_string(LDA_NOALLOC_MAX_REGIONS) + " regions; this layout has " +
                                    std::to_string(h->p.n_regions) + " (use lda_loglik)");
  HIP_TRY(h, launch_loglik_noalloc(h->d, h->p, h->noalloc_scratch, h->stream));
  double sum = 0.0;
  const double *result = reinterpret_cast<const double *>(static_cast<unsigned char *>(h->noalloc_scratch) +
                                                          kNoAllocResult);
  HIP_TRY(h, hipMemcpyAsync(&sum, result, sizeof(double), hipMemcpyDeviceToHost, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  *llpt = sum / double(h->L.n);
  return LDA_OK;
}

lda_status lda_set_assignments(lda_handle *h, const int32_t *z, int64_t iteration) {
  LDA_TRY(check_handle(h));
  if (!z) return fail(h, LDA_E_ARG, "z is NULL");
  if (iteration < 0 || iteration >= (int64_t(1) << 32)) return fail(h, LDA_E_ARG, "iteration out of range");
  if (h->chunks) return chunked_set_assignments(h, z, iteration);
  const Layout &L = h->L;
  const size_t n = size_t(L.n);
  for (size_t i = 0; i < n; ++i)
    if (z[i] < 0 || z[i] >= L.K) return fail(h, LDA_E_ARG, "topic out of range at token " + std::to_string(i));
  int32_t *zin = nullptr;
  LDA_TRY(dalloc(h, &zin, n));
  HIP_TRY(h, hipMemcpyAsync(zin, z, n * 4, hipMemcpyHostToDevice, h->stream));
  HIP_TRY(h, hipMemsetAsync(h->stats_base, 0, sizeof(unsigned long long) * kStatsPerIter, h->stream));
  HIP_TRY(h, launch_gather_z(zin, h->d.wt_kr, L.n, L.K, h->d.z_w, h->stats_base + ST_ERRORS, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  dfree(h, zin);
  unsigned long long st[kStatsPerIter];
  HIP_TRY(h, hipMemcpy(st, h->stats_base, sizeof(st), hipMemcpyDeviceToHost));
  LDA_TRY(check_errors(h, st));
  LDA_TRY(rebuild_counts(h));
  // the skip counts of earlier iterations describe another assignment
  HIP_TRY(h, hipMemsetAsync(h->d.skip_hist, 0, 2 * sizeof(unsigned long long), h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  HIP_TRY(h, hipMemcpy(st, h->stats_base, sizeof(st), hipMemcpyDeviceToHost));
  LDA_TRY(check_errors(h, st));
  h->iteration = iteration;
  return LDA_OK;
}

void lda_destroy(lda_handle *h) { release(h); }

const char *lda_last_error(const lda_handle *h) { return h ? h->err.c_str() : g_create_error.c_str(); }

lda_status lda_describe_layout(const int32_t *word, const int32_t *doc, int64_t n_tokens, int32_t V, int32_t K,
                               int32_t region_tokens, int32_t dense_cutoff, int32_t *relabel, int32_t *n_present,
                               int32_t *n_dense,
                               int64_t *n_regions, int32_t *n_docs, uint32_t *word_off, uint32_t *wt_key,
                               uint32_t *region) {
  if (!word || !doc || n_tokens <= 0 || V <= 0 || K < 2 || K > LDA_MAX_TOPICS || region_tokens < 0)
    return fail(nullptr, LDA_E_ARG, "bad argument");
  Layout L;
  std::string msg;
  lda_status st;
  try {
    st = build_layout(word, doc, n_tokens, V, K, region_tokens ? region_tokens : kDefaultRegionTokens, dense_cutoff, L,
                      msg);
  } catch (const std::bad_alloc &) {
    return fail(nullptr, LDA_E_NOMEM, "host allocation failed");
  }
  if (st != LDA_OK) return fail(nullptr, st, msg);
  if (n_present) *n_present = L.n_present;
  if (n_dense) *n_dense = L.n_dense;
  if (n_regions) *n_regions = L.n_regions;
  if (n_docs) *n_docs = L.M;
  if (relabel) std::memcpy(relabel, L.relabel.data(), L.relabel.size() * 4);
  if (word_off) std::memcpy(word_off, L.word_off.data(), L.word_off.size() * 4);
  if (wt_key) std::memcpy(wt_key, L.wt_key.data(), L.wt_key.size() * 4);
  if (region) std::memcpy(region, L.region.data(), L.region.size() * 4);
  return LDA_OK;
}

}  // extern "C"
