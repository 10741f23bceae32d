// Out-of-core chunked corpus (Sec. 4.1 and 4.3 of the paper: the token list
// is partitioned into chunks of documents, streamed to the device, and the
// transfers are hidden behind the computation).
//
// With lda_options.chunks = C > 1 the documents are cut into C ranges of
// near-equal token counts.  Per chunk only two per-token arrays live on the
// host, in pinned memory: dt_wpos (the word-order slot of each doc-ordered
// token, u32) and the topics in word order (u16), 6 bytes a token.  Each
// chunk's small tables (document offsets, D-row offsets, word offsets,
// regions) stay on the device.  W is dense for every word (partial rows from
// several chunks add up) and double-buffered, like T: the chunks of an
// iteration sample against W_cur and T_cur while their new counts accumulate
// in W_next and T_next, which become current at the end of the iteration, so
// every chunk samples the same snapshot and the draws equal the resident
// path's.
//
// A chunk's turn on the device: upload dt_wpos and topics (one stream), derive
// the doc-ordered word ids, the keys and the D-row offsets (k_inflate),
// rebuild the chunk's D rows from the loaded topics (they never cross PCIe),
// the doc pass, the sampler, the chunk's W and T into W_next/T_next, and
// download the topics (another stream).  Two device slots alternate, so the
// turn of chunk c overlaps the upload of chunk c+1 and the download of c-1.
#include <cstring>

#include "handle.h"

namespace lda {

struct ChunkInfo {
  uint32_t tok0 = 0, ntok = 0;  // first doc-order position (= input index) and token count
  uint32_t doc0 = 0, ndoc = 0;  // first document and document count
  uint32_t *h_wpos = nullptr;   // pinned host [ntok]
  uint16_t *h_z = nullptr;      // pinned host [ntok]
  uint32_t *doc_off = nullptr, *d_cap = nullptr, *word_off = nullptr, *region = nullptr;  // device, chunk-local
  uint32_t *heavy_docs = nullptr;  // device: the chunk's documents longer than kHeavyDocTokens (chunk-local ids)
  uint32_t d_slots = 0;         // D-row slots of the chunk's documents
  Params p{};                   // launch parameters of the chunk
};

struct ChunkSlot {
  uint32_t *dt_word = nullptr, *dt_wpos = nullptr;
  uint2 *wt_kr = nullptr;
  uint32_t *skip_bits = nullptr, *d_ent = nullptr;
  uint16_t *z_w = nullptr;
  hipEvent_t loaded = nullptr, computed = nullptr, unloaded = nullptr;
};

struct ChunkMode {
  std::vector<ChunkInfo> c;
  ChunkSlot slot[2];
  // topics on their way home: a chunk's new topics are copied here on the
  // device, so that its slot takes the next upload without waiting for the
  // download (two buffers, alternating like the slots)
  uint16_t *z_out[2] = {nullptr, nullptr};
  hipEvent_t z_out_free[2] = {nullptr, nullptr};
  hipStream_t h2d = nullptr, d2h = nullptr;
  std::vector<hipEvent_t> z_home;  // per chunk: its topics are back in host memory
  int32_t *w_next = nullptr;
  uint32_t *t_next = nullptr;
  double *ll_chunk = nullptr;
  uint32_t max_tok = 0, max_slots = 0;
  int64_t max_regions = 0;
};

void release_chunks(ChunkMode *cm) {
  if (!cm) return;
  if (cm->h2d) (void)hipStreamSynchronize(cm->h2d);
  if (cm->d2h) (void)hipStreamSynchronize(cm->d2h);
  for (ChunkInfo &ci : cm->c) {
    if (ci.h_wpos) (void)hipHostFree(ci.h_wpos);
    if (ci.h_z) (void)hipHostFree(ci.h_z);
  }
  for (ChunkSlot &s : cm->slot)
    for (hipEvent_t ev : {s.loaded, s.computed, s.unloaded})
      if (ev) (void)hipEventDestroy(ev);
  for (hipEvent_t ev : cm->z_home)
    if (ev) (void)hipEventDestroy(ev);
  for (hipEvent_t ev : cm->z_out_free)
    if (ev) (void)hipEventDestroy(ev);
  if (cm->h2d) (void)hipStreamDestroy(cm->h2d);
  if (cm->d2h) (void)hipStreamDestroy(cm->d2h);
  delete cm;
}

namespace {

lda_status alloc_slot(lda_handle *h, ChunkSlot &s, uint32_t max_tok, uint32_t max_slots) {
  LDA_TRY(dalloc(h, &s.dt_word, max_tok));
  LDA_TRY(dalloc(h, &s.dt_wpos, max_tok));
  LDA_TRY(dalloc(h, &s.wt_kr, max_tok));
  LDA_TRY(dalloc(h, &s.z_w, max_tok));
  LDA_TRY(dalloc(h, &s.skip_bits, size_t(skip_words(max_tok))));
  LDA_TRY(dalloc(h, &s.d_ent, size_t(max_slots) + kRowPad));
  HIP_TRY(h, hipEventCreateWithFlags(&s.loaded, hipEventDisableTiming));
  HIP_TRY(h, hipEventCreateWithFlags(&s.computed, hipEventDisableTiming));
  HIP_TRY(h, hipEventCreateWithFlags(&s.unloaded, hipEventDisableTiming));
  return LDA_OK;
}

// The handle's state seen by one chunk in one slot: the global tables (W, T,
// per-word records, counters), the chunk's own document, word and region
// tables, and the slot's per-token arrays and D rows.
DevState chunk_state(const lda_handle *h, const ChunkInfo &ci, const ChunkSlot &sl) {
  DevState d = h->d;
  d.doc_off = ci.doc_off;
  d.d_cap = ci.d_cap;
  d.word_off = ci.word_off;
  d.region = ci.region;
  d.heavy_docs = ci.heavy_docs;
  d.dt_word = sl.dt_word;
  d.dt_wpos = sl.dt_wpos;
  d.wt_kr = sl.wt_kr;
  d.z_w = sl.z_w;
  d.skip_bits = sl.skip_bits;
  d.d_ent = sl.d_ent;
  d.dt_key = nullptr;
  d.skip_doc = nullptr;
  return d;
}

// A loaded chunk's derived arrays and D rows (from the topics in the slot),
// on stream st.
lda_status prepare_chunk(lda_handle *h, const ChunkInfo &ci, const DevState &d, hipStream_t st) {
  HIP_TRY(h, launch_inflate(ci.region, ci.p.n_regions, ci.doc_off, ci.d_cap, int32_t(ci.ndoc), d.dt_wpos, ci.tok0,
                            d.dt_word, d.wt_kr, st));
  HIP_TRY(h, launch_reset_counters(d.counters, st));
  HIP_TRY(h, launch_rebuild_d(d, ci.p, st));
  return LDA_OK;
}

// Load chunk c into slot 0 on the compute stream (no overlap: the calls that
// inspect or reset the state) and prepare it.
lda_status load_chunk_now(lda_handle *h, const ChunkInfo &ci, const DevState &d) {
  HIP_TRY(h, hipMemcpyAsync(d.dt_wpos, ci.h_wpos, size_t(ci.ntok) * 4, hipMemcpyHostToDevice, h->stream));
  HIP_TRY(h, hipMemcpyAsync(d.z_w, ci.h_z, size_t(ci.ntok) * 2, hipMemcpyHostToDevice, h->stream));
  return prepare_chunk(h, ci, d, h->stream);
}

lda_status check_stats(lda_handle *h, const unsigned long long *st) {
  if (st[ST_ERRORS]) return fail(h, LDA_E_DEVICE, "kernel found " + std::to_string(st[ST_ERRORS]) + " topic slots outside [0, K)");
  return LDA_OK;
}

}  // namespace

lda_status chunked_create(lda_handle *h, const int32_t *word, const int32_t *doc, int32_t R, int32_t n_chunks) {
  Layout &L = h->L;
  Params &p = h->p;
  DevState &d = h->d;
  const int64_t n = L.n;
  const int32_t M = L.M, V = L.V, K = L.K;
  h->chunks.reset(new ChunkMode());
  ChunkMode &cm = *h->chunks;

  // 1. tokens per word and per document (the input is sorted by document)
  std::vector<uint32_t> cnt(static_cast<size_t>(V), 0u);
  L.doc_off.assign(size_t(M) + 1, 0u);
  for (int64_t i = 0; i < n; ++i) {
    cnt[size_t(word[i])]++;
    L.doc_off[size_t(doc[i]) + 1]++;
  }
  for (int32_t q = 0; q < M; ++q) L.doc_off[size_t(q) + 1] += L.doc_off[size_t(q)];
  // 2. relabel by count, every word dense: the partial rows of the chunks add up
  std::string msg;
  lda_status st = plan_from_counts(cnt, K, R, -1, L, msg, false);
  if (st != LDA_OK) return fail(h, st, msg);
  p.n_present = L.n_present;
  p.n_dense = L.n_dense;
  p.doc_marks_ok = 0;   // the sampler reads skip decisions in word order only
  p.sparse_pre = 0;     // no sparse rows
  p.key_identity = 1;

  // 3. chunks: document ranges of near-equal token counts
  std::vector<uint32_t> cut(size_t(n_chunks) + 1, 0u);
  for (int32_t c = 1; c < n_chunks; ++c) {
    const uint64_t target = uint64_t(n) * uint64_t(c) / uint64_t(n_chunks);
    cut[size_t(c)] = uint32_t(std::lower_bound(L.doc_off.begin(), L.doc_off.end(), uint32_t(target)) - L.doc_off.begin());
    cut[size_t(c)] = std::min<uint32_t>(std::max(cut[size_t(c)], cut[size_t(c) - 1]), uint32_t(M));
  }
  cut[size_t(n_chunks)] = uint32_t(M);
  for (int32_t c = 0; c < n_chunks; ++c) {
    ChunkInfo ci;
    ci.doc0 = cut[size_t(c)];
    ci.ndoc = cut[size_t(c) + 1] - ci.doc0;
    ci.tok0 = L.doc_off[ci.doc0];
    ci.ntok = L.doc_off[ci.doc0 + ci.ndoc] - ci.tok0;
    if (ci.ntok == 0) continue;  // only empty documents: nothing to sample
    uint64_t slots = 0;
    for (uint32_t q = 0; q < ci.ndoc; ++q)
      slots += d_row_slots(std::min<uint32_t>(L.doc_off[ci.doc0 + q + 1] - L.doc_off[ci.doc0 + q], uint32_t(K)));
    if (slots + kRowPad >= (uint64_t(1) << 32)) return fail(h, LDA_E_RANGE, "a chunk's D rows exceed 32-bit offsets");
    ci.d_slots = uint32_t(slots);
    cm.max_tok = std::max(cm.max_tok, ci.ntok);
    cm.max_slots = std::max(cm.max_slots, ci.d_slots);
    cm.c.push_back(ci);
  }

  // 4. the global device state: W and T twice (snapshot and next), the
  // per-word records, counters and statistics
  const size_t wsize = size_t(p.n_dense) * size_t(K);
  LDA_TRY(dalloc(h, &d.w_dense, wsize));
  LDA_TRY(dalloc(h, &cm.w_next, wsize));
  LDA_TRY(dalloc(h, &d.T, size_t(K)));
  LDA_TRY(dalloc(h, &cm.t_next, size_t(K)));
  LDA_TRY(dalloc(h, &d.den, size_t(K)));
  LDA_TRY(dalloc(h, &d.bden, size_t(K)));
  LDA_TRY(dalloc(h, &d.wrec, size_t(p.n_present)));
  LDA_TRY(dalloc(h, &d.wskip, size_t(p.n_present)));
  LDA_TRY(dalloc(h, &d.counters, kCounters));
  LDA_TRY(dalloc(h, &h->stats_base, size_t(kStatSlots) * kStatsPerIter));
  LDA_TRY(dalloc(h, &d.skip_hist, 2));
  LDA_TRY(dalloc(h, &d.ll_out, 1));
  LDA_TRY(dalloc(h, &cm.ll_chunk, cm.c.size()));
  LDA_TRY(dalloc(h, &d.split, size_t(p.n_dense)));
  LDA_TRY(upload(h, d.split, std::vector<uint8_t>(size_t(p.n_dense), uint8_t(1))));
  HIP_TRY(h, hipMemsetAsync(d.skip_hist, 0, 2 * sizeof(unsigned long long), h->stream));
  HIP_TRY(h, hipMemsetAsync(h->stats_base, 0, sizeof(unsigned long long) * kStatSlots * kStatsPerIter, h->stream));
  d.stats = h->stats_base;

  // 5. two device slots, the copy streams, pinned host arrays
  for (ChunkSlot &sl : cm.slot) LDA_TRY(alloc_slot(h, sl, cm.max_tok, cm.max_slots));
  HIP_TRY(h, hipStreamCreateWithFlags(&cm.h2d, hipStreamNonBlocking));
  HIP_TRY(h, hipStreamCreateWithFlags(&cm.d2h, hipStreamNonBlocking));
  cm.z_home.assign(cm.c.size(), nullptr);
  for (hipEvent_t &ev : cm.z_home) HIP_TRY(h, hipEventCreateWithFlags(&ev, hipEventDisableTiming));
  for (int q = 0; q < 2; ++q) {
    LDA_TRY(dalloc(h, &cm.z_out[q], cm.max_tok));
    HIP_TRY(h, hipEventCreateWithFlags(&cm.z_out_free[q], hipEventDisableTiming));
  }
  for (ChunkInfo &ci : cm.c) {
    HIP_TRY(h, hipHostMalloc(reinterpret_cast<void **>(&ci.h_wpos), size_t(ci.ntok) * 4, hipHostMallocDefault));
    HIP_TRY(h, hipHostMalloc(reinterpret_cast<void **>(&ci.h_z), size_t(ci.ntok) * 2, hipHostMallocDefault));
  }

  // 6. every chunk's layout, built on the device through slot 0: relabelled
  // word ids, a stable sort by word (documents ascend inside a word), the
  // inverted index, word offsets and regions; its initial topics; its share
  // of the initial W and T
  int32_t *relabel_d = nullptr;
  LDA_TRY(dalloc(h, &relabel_d, size_t(V)));
  LDA_TRY(upload(h, relabel_d, L.relabel));
  ChunkSlot &s0 = cm.slot[0], &s1 = cm.slot[1];
  int32_t *word_tmp = reinterpret_cast<int32_t *>(s1.dt_word);  // scratch of the build
  // (the second slot's 8-byte records hold two max_tok arrays of 4 bytes)
  uint32_t *wnew = s1.dt_wpos, *wkey = reinterpret_cast<uint32_t *>(s1.wt_kr), *wpos = wkey + cm.max_tok;
  HIP_TRY(h, launch_zero_split(d, p, h->stream));
  // large K: the scratch rows the W rebuild builds T in (it runs per chunk below)
  if (w_bits(p)) LDA_TRY(dalloc(h, &d.wscratch, size_t(loglik_grid_big_k(p)) * size_t(K)));
  int64_t total_regions = 0;
  uint32_t max_region = 1;
  for (ChunkInfo &ci : cm.c) {
    HIP_TRY(h, hipMemcpyAsync(word_tmp, word + ci.tok0, size_t(ci.ntok) * 4, hipMemcpyHostToDevice, h->stream));
    HIP_TRY(h, launch_gather_u32(wnew, relabel_d, reinterpret_cast<const uint32_t *>(word_tmp), ci.ntok, h->stream));
    LDA_TRY(sort_pairs(h, wnew, wkey, nullptr, wpos, bits_for(uint64_t(std::max(p.n_present, 1)) - 1), ci.ntok));
    HIP_TRY(h, launch_invert(wpos, ci.ntok, s0.dt_wpos, h->stream));
    LDA_TRY(dalloc(h, &ci.word_off, size_t(p.n_present) + 1));
    HIP_TRY(h, launch_boundaries(wkey, ci.ntok, uint32_t(p.n_present), ci.word_off, h->stream));
    std::vector<uint32_t> woff(size_t(p.n_present) + 1);
    HIP_TRY(h, hipMemcpyAsync(woff.data(), ci.word_off, woff.size() * 4, hipMemcpyDeviceToHost, h->stream));
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    std::vector<uint8_t> split_local;
    std::vector<uint32_t> region;
    int64_t ndr = 0;
    make_regions(woff, p.n_dense, R, split_local, region, ndr);
    LDA_TRY(dalloc(h, &ci.region, region.size()));
    LDA_TRY(upload(h, ci.region, region));
    for (size_t r = 0; r < region.size(); r += 3) max_region = std::max(max_region, region[r + 2] - region[r + 1]);
    // chunk-local document and D-row offsets
    std::vector<uint32_t> doff(size_t(ci.ndoc) + 1), dcap(size_t(ci.ndoc) + 1, 0u);
    for (uint32_t q = 0; q <= ci.ndoc; ++q) doff[q] = L.doc_off[ci.doc0 + q] - ci.tok0;
    for (uint32_t q = 0; q < ci.ndoc; ++q)
      dcap[q + 1] = dcap[q] + d_row_slots(std::min<uint32_t>(doff[q + 1] - doff[q], uint32_t(K)));
    LDA_TRY(dalloc(h, &ci.doc_off, doff.size()));
    LDA_TRY(dalloc(h, &ci.d_cap, dcap.size()));
    LDA_TRY(upload(h, ci.doc_off, doff));
    LDA_TRY(upload(h, ci.d_cap, dcap));
    const std::vector<uint32_t> heavy = heavy_documents(doff.data(), ci.ndoc);
    LDA_TRY(dalloc(h, &ci.heavy_docs, heavy.size()));
    LDA_TRY(upload(h, ci.heavy_docs, heavy));
    ci.p = p;
    ci.p.n_heavy = int32_t(heavy.size());
    ci.p.n = ci.ntok;
    ci.p.M = int32_t(ci.ndoc);
    ci.p.n_regions = int64_t(region.size() / 3);
    ci.p.light_begin = light_region_start(region, K, p.big_k != 0);
    ci.p.key_base = ci.tok0;
    ci.p.xcd_doc[0] = 0;
    for (int x = 1; x < kXcds; ++x) {
      const uint64_t target = uint64_t(ci.ntok) * uint64_t(x) / uint64_t(kXcds);
      ci.p.xcd_doc[x] = uint32_t(std::lower_bound(doff.begin(), doff.end(), uint32_t(target)) - doff.begin());
      ci.p.xcd_doc[x] = std::min<uint32_t>(std::max(ci.p.xcd_doc[x], ci.p.xcd_doc[x - 1]), ci.ndoc);
    }
    ci.p.xcd_doc[kXcds] = ci.ndoc;
    total_regions += ci.p.n_regions;
    cm.max_regions = std::max(cm.max_regions, ci.p.n_regions);
    DevState dc = chunk_state(h, ci, s0);
    HIP_TRY(h, launch_inflate(ci.region, ci.p.n_regions, ci.doc_off, ci.d_cap, int32_t(ci.ndoc), s0.dt_wpos, ci.tok0,
                              s0.dt_word, s0.wt_kr, h->stream));
    HIP_TRY(h, launch_init_topics(dc, ci.p, h->stream));
    HIP_TRY(h, launch_reset_counters(d.counters, h->stream));
    HIP_TRY(h, launch_rebuild_w(dc, ci.p, h->stream));
    HIP_TRY(h, hipMemcpyAsync(ci.h_wpos, s0.dt_wpos, size_t(ci.ntok) * 4, hipMemcpyDeviceToHost, h->stream));
    HIP_TRY(h, hipMemcpyAsync(ci.h_z, s0.z_w, size_t(ci.ntok) * 2, hipMemcpyDeviceToHost, h->stream));
    HIP_TRY(h, hipStreamSynchronize(h->stream));
  }
  dfree(h, relabel_d);
  p.n_regions = total_regions;
  p.max_region = int32_t(max_region);
  for (ChunkInfo &ci : cm.c) ci.p.max_region = p.max_region;
  LDA_TRY(dalloc(h, &d.ll_part, size_t(std::max<int64_t>(cm.max_regions, 1))));
  if (p.big_k) {
    const size_t sl = size_t(tiled_grid(p)) * size_t(max_region);
    LDA_TRY(dalloc(h, &d.ts_s, sl));
    LDA_TRY(dalloc(h, &d.ts_c1, sl));
    LDA_TRY(dalloc(h, &d.ts_code, sl));
    LDA_TRY(dalloc(h, &d.ts_list, sl));
  }
  unsigned long long stt[kStatsPerIter];
  HIP_TRY(h, hipMemcpy(stt, h->stats_base, sizeof(stt), hipMemcpyDeviceToHost));
  return check_stats(h, stt);
}

lda_status chunked_iterate(lda_handle *h, int32_t n_iters, lda_iter_stats *stats) {
  ChunkMode &cm = *h->chunks;
  const Params &p = h->p;
  if (stats && h->events.empty()) {
    h->events.assign(size_t(kStatSlots) * kEventsPerIter, nullptr);
    for (auto &ev : h->events) HIP_TRY(h, hipEventCreate(&ev));
  }
  for (int32_t done = 0; done < n_iters;) {
    const int32_t chunk = std::min<int32_t>(n_iters - done, kStatSlots);
    for (int32_t it = 0; it < chunk; ++it) {
      const uint32_t t = uint32_t(h->iteration);
      DevState g = h->d;  // W and T of the snapshot
      g.stats = h->stats_base + size_t(it) * kStatsPerIter;
      hipEvent_t *ev = stats ? &h->events[size_t(it) * kEventsPerIter] : nullptr;
      if (ev) HIP_TRY(h, hipEventRecord(ev[0], h->stream));
      HIP_TRY(h, launch_begin_iteration(g, p, h->stream));
      HIP_TRY(h, launch_word_pre(g, p, h->stream));
      DevState nx = g;  // the counts of this iteration's draws accumulate here
      nx.w_dense = cm.w_next;
      nx.T = cm.t_next;
      HIP_TRY(h, launch_zero_split(nx, p, h->stream));
      for (size_t c = 0; c < cm.c.size(); ++c) {
        const ChunkInfo &ci = cm.c[c];
        ChunkSlot &sl = cm.slot[c & 1];
        // upload, once the slot's previous chunk is home and this chunk's topics are too
        HIP_TRY(h, hipStreamWaitEvent(cm.h2d, sl.unloaded, 0));
        HIP_TRY(h, hipStreamWaitEvent(cm.h2d, cm.z_home[c], 0));
        HIP_TRY(h, hipMemcpyAsync(sl.dt_wpos, ci.h_wpos, size_t(ci.ntok) * 4, hipMemcpyHostToDevice, cm.h2d));
        HIP_TRY(h, hipMemcpyAsync(sl.z_w, ci.h_z, size_t(ci.ntok) * 2, hipMemcpyHostToDevice, cm.h2d));
        HIP_TRY(h, hipEventRecord(sl.loaded, cm.h2d));
        // the chunk's turn: derived arrays, D rows of the snapshot, steps 2-6, its counts into W_next/T_next
        HIP_TRY(h, hipStreamWaitEvent(h->stream, sl.loaded, 0));
        DevState dc = chunk_state(h, ci, sl);
        dc.stats = g.stats;
        LDA_TRY(prepare_chunk(h, ci, dc, h->stream));
        HIP_TRY(h, launch_clear_skips(dc, ci.p, t, h->stream, c == 0));
        if (!p.no_skip) HIP_TRY(h, launch_doc_pass(dc, ci.p, t, h->stream));
        LDA_TRY(run_sampler(h, dc, ci.p, t));
        DevState dw = dc;
        dw.w_dense = cm.w_next;
        dw.T = cm.t_next;
        HIP_TRY(h, launch_rebuild_w(dw, ci.p, h->stream));
        // the new topics leave the slot for a download buffer (once that
        // buffer's previous download is done), which frees the slot
        uint16_t *zo = cm.z_out[c & 1];
        HIP_TRY(h, hipStreamWaitEvent(h->stream, cm.z_out_free[c & 1], 0));
        HIP_TRY(h, hipMemcpyAsync(zo, sl.z_w, size_t(ci.ntok) * 2, hipMemcpyDeviceToDevice, h->stream));
        HIP_TRY(h, hipEventRecord(sl.computed, h->stream));
        HIP_TRY(h, hipEventRecord(sl.unloaded, h->stream));
        // download the new topics
        HIP_TRY(h, hipStreamWaitEvent(cm.d2h, sl.computed, 0));
        HIP_TRY(h, hipMemcpyAsync(ci.h_z, zo, size_t(ci.ntok) * 2, hipMemcpyDeviceToHost, cm.d2h));
        HIP_TRY(h, hipEventRecord(cm.z_home[c], cm.d2h));
        HIP_TRY(h, hipEventRecord(cm.z_out_free[c & 1], cm.d2h));
      }
      if (ev) HIP_TRY(h, hipEventRecord(ev[4], h->stream));
      std::swap(h->d.w_dense, cm.w_next);
      std::swap(h->d.T, cm.t_next);
      h->iteration++;
    }
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    HIP_TRY(h, hipStreamSynchronize(cm.d2h));
    std::vector<unsigned long long> st(static_cast<size_t>(chunk) * kStatsPerIter);
    HIP_TRY(h, hipMemcpy(st.data(), h->stats_base, st.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost));
    for (int32_t it = 0; it < chunk; ++it) {
      const unsigned long long *s = &st[size_t(it) * kStatsPerIter];
      LDA_TRY(check_stats(h, s));
      if (!stats) continue;
      lda_iter_stats &o = stats[done + it];
      std::memset(&o, 0, sizeof(o));
      float ms_all = 0;
      hipEvent_t *ev = &h->events[size_t(it) * kEventsPerIter];
      HIP_TRY(h, hipEventElapsedTime(&ms_all, ev[0], ev[4]));
      o.iteration = h->iteration - chunk + it;
      o.ms_iter = ms_all;
      o.skip_step3 = int64_t(s[ST_SKIP3]);
      o.skip_after_s = int64_t(s[ST_SKIP_AFTER_S]);
      o.sampled = int64_t(s[ST_SAMPLED]);
      o.nnz_scanned = int64_t(s[ST_NNZ]);
      o.regions = int64_t(s[ST_REGIONS]);
      o.dense_regions = int64_t(s[ST_DENSE_REGIONS]);
      o.row_bytes = int64_t(s[ST_ROW_BYTES]);
      o.sampler_block = p.sampler_block;
      o.skip_marks = int64_t(s[ST_MARKS]);
      o.skip_test_ran = int64_t(s[ST_TEST_RAN]);
    }
    done += chunk;
  }
  return LDA_OK;
}

lda_status chunked_counts(lda_handle *h, lda_counts *out) {
  ChunkMode &cm = *h->chunks;
  const Layout &L = h->L;
  const Params &p = h->p;
  const int32_t K = L.K;
  const bool want_d = out->D_off || out->D_topic || out->D_count;
  if (want_d && (!out->D_off || !out->D_topic || !out->D_count))
    return fail(h, LDA_E_ARG, "D arrays must be given together");
  if ((out->W_off || out->W_topic || out->W_count) && (!out->W_off || !out->W_topic || !out->W_count))
    return fail(h, LDA_E_ARG, "W arrays must be given together");
  std::vector<int32_t> wd(size_t(p.n_dense) * size_t(K));
  if (!wd.empty()) HIP_TRY(h, hipMemcpy(wd.data(), h->d.w_dense, wd.size() * 4, hipMemcpyDeviceToHost));
  int64_t nnz_W = 0;
  for (int32_t x : wd) nnz_W += x != 0;
  // D: each chunk's rows rebuilt from its topics on the device, then read back
  const bool size_query = !out->z && !out->T && !want_d && !out->W_off && !out->W_topic && !out->W_count;
  int64_t nnz_D = 0, o = 0;
  ChunkSlot &s0 = cm.slot[0];
  unsigned long long *nnz_dev = reinterpret_cast<unsigned long long *>(cm.slot[1].d_ent);
  std::vector<uint32_t> ent;
  size_t next_doc = 0;
  for (const ChunkInfo &ci : cm.c) {
    DevState dc = chunk_state(h, ci, s0);
    dc.stats = h->stats_base;
    LDA_TRY(load_chunk_now(h, ci, dc));
    if (!want_d) {
      HIP_TRY(h, hipMemsetAsync(nnz_dev, 0, sizeof(unsigned long long), h->stream));
      HIP_TRY(h, launch_sum_nnz(dc, ci.p, nnz_dev, h->stream));
      unsigned long long c_nnz = 0;
      HIP_TRY(h, hipMemcpyAsync(&c_nnz, nnz_dev, sizeof(c_nnz), hipMemcpyDeviceToHost, h->stream));
      HIP_TRY(h, hipStreamSynchronize(h->stream));
      nnz_D += int64_t(c_nnz);
      continue;
    }
    ent.resize(ci.d_slots);
    HIP_TRY(h, hipMemcpyAsync(ent.data(), s0.d_ent, ent.size() * 4, hipMemcpyDeviceToHost, h->stream));
    std::vector<uint32_t> dcap(size_t(ci.ndoc) + 1);
    HIP_TRY(h, hipMemcpyAsync(dcap.data(), ci.d_cap, dcap.size() * 4, hipMemcpyDeviceToHost, h->stream));
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    for (; next_doc < ci.doc0; ++next_doc) out->D_off[next_doc] = o;  // empty documents between chunks
    for (uint32_t q = 0; q < ci.ndoc; ++q, ++next_doc) {
      out->D_off[next_doc] = o;
      const uint32_t hdr = ent[dcap[q]];
      for (uint32_t e = 0; e < (hdr & 0xFFFFu); ++e) {
        const uint32_t v = ent[size_t(dcap[q]) + 1 + e];
        out->D_topic[o] = int32_t(v >> 16);
        out->D_count[o] = int32_t(v & 0xFFFFu);
        ++o;
      }
    }
  }
  if (want_d) {
    for (; next_doc <= size_t(L.M); ++next_doc) out->D_off[next_doc] = o;
    nnz_D = o;
  }
  out->iteration = h->iteration;
  out->M = L.M;
  out->V = L.V;
  out->K = K;
  out->n_tokens = L.n;
  out->nnz_D = nnz_D;
  out->nnz_W = nnz_W;
  if (size_query) return LDA_OK;
  if (out->z) {
    // input order is document order: the topic of position p sits at its word-order slot
    for (const ChunkInfo &ci : cm.c)
      for (uint32_t q = 0; q < ci.ntok; ++q) out->z[size_t(ci.tok0) + q] = int32_t(ci.h_z[ci.h_wpos[q]]);
  }
  if (out->T) {
    std::vector<uint32_t> tk(static_cast<size_t>(K));
    HIP_TRY(h, hipMemcpy(tk.data(), h->d.T, size_t(K) * 4, hipMemcpyDeviceToHost));
    for (int32_t k = 0; k < K; ++k) out->T[k] = tk[size_t(k)];
  }
  if (out->W_off) {
    int64_t w = 0;
    for (int32_t v = 0; v < L.V; ++v) {
      out->W_off[v] = w;
      const int32_t r = L.relabel[size_t(v)];
      if (r >= L.n_present) continue;
      const int32_t *row = &wd[size_t(r) * size_t(K)];
      for (int32_t k = 0; k < K; ++k)
        if (row[k]) {
          out->W_topic[w] = k;
          out->W_count[w] = row[k];
          ++w;
        }
    }
    out->W_off[L.V] = w;
  }
  return LDA_OK;
}

lda_status chunked_loglik(lda_handle *h, double *llpt, void *scratch) {
  ChunkMode &cm = *h->chunks;
  const Params &p = h->p;
  DevState g = h->d;
  double *sums = cm.ll_chunk;
  if (scratch) {
    // the fixed array of lda_loglik_noalloc: counters, statistics, result,
    // per-chunk sums, per-region partials of the largest chunk
    if (cm.max_regions > int64_t(LDA_NOALLOC_MAX_REGIONS))
      return fail(h, LDA_E_RANGE, "lda_loglik_noalloc holds partial sums for at most " +
                                      std::to_string(LDA_NOALLOC_MAX_REGIONS) + " regions of a chunk; this layout has " +
                                      std::to_string(cm.max_regions) + " (use lda_loglik)");
    unsigned char *base = static_cast<unsigned char *>(scratch);
    g.counters = reinterpret_cast<uint32_t *>(base);
    g.stats = reinterpret_cast<unsigned long long *>(base + sizeof(uint32_t) * kCounters);
    g.ll_out = reinterpret_cast<double *>(base + kNoAllocResult);
    sums = reinterpret_cast<double *>(base + kNoAllocChunkSums);
    g.ll_part = reinterpret_cast<double *>(base + kNoAllocHead);
  } else {
    g.stats = h->stats_base;
  }
  HIP_TRY(h, launch_begin_iteration(g, p, h->stream));
  HIP_TRY(h, launch_word_pre(g, p, h->stream));
  for (size_t c = 0; c < cm.c.size(); ++c) {
    const ChunkInfo &ci = cm.c[c];
    DevState dc = chunk_state(h, ci, cm.slot[0]);
    dc.counters = g.counters;
    dc.stats = g.stats;
    dc.ll_part = g.ll_part;
    dc.ll_out = sums + c;  // the chunk's sum of its regions' partials
    LDA_TRY(load_chunk_now(h, ci, dc));
    HIP_TRY(h, launch_reset_counters(dc.counters, h->stream));
    HIP_TRY(h, launch_loglik(dc, ci.p, h->stream));
  }
  HIP_TRY(h, launch_sum_f64(sums, int64_t(cm.c.size()), g.ll_out, h->stream));
  double sum = 0.0;
  HIP_TRY(h, hipMemcpyAsync(&sum, g.ll_out, sizeof(double), hipMemcpyDeviceToHost, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  *llpt = sum / double(h->L.n);
  return LDA_OK;
}

lda_status chunked_set_assignments(lda_handle *h, const int32_t *z, int64_t iteration) {
  ChunkMode &cm = *h->chunks;
  const Layout &L = h->L;
  const Params &p = h->p;
  for (int64_t i = 0; i < L.n; ++i)
    if (z[i] < 0 || z[i] >= L.K) return fail(h, LDA_E_ARG, "topic out of range at token " + std::to_string(i));
  DevState g = h->d;
  g.stats = h->stats_base;
  HIP_TRY(h, hipMemsetAsync(h->stats_base, 0, sizeof(unsigned long long) * kStatsPerIter, h->stream));
  HIP_TRY(h, launch_zero_split(g, p, h->stream));  // W and T of the snapshot, rebuilt below
  ChunkSlot &s0 = cm.slot[0];
  int32_t *z_doc = reinterpret_cast<int32_t *>(cm.slot[1].dt_word);
  for (const ChunkInfo &ci : cm.c) {
    DevState dc = chunk_state(h, ci, s0);
    dc.stats = g.stats;
    HIP_TRY(h, hipMemcpyAsync(z_doc, z + ci.tok0, size_t(ci.ntok) * 4, hipMemcpyHostToDevice, h->stream));
    HIP_TRY(h, hipMemcpyAsync(s0.dt_wpos, ci.h_wpos, size_t(ci.ntok) * 4, hipMemcpyHostToDevice, h->stream));
    HIP_TRY(h, launch_doc_scatter_z(z_doc, s0.dt_wpos, ci.ntok, L.K, s0.z_w, g.stats + ST_ERRORS, h->stream));
    HIP_TRY(h, launch_reset_counters(g.counters, h->stream));
    HIP_TRY(h, launch_rebuild_w(dc, ci.p, h->stream));
    HIP_TRY(h, hipMemcpyAsync(ci.h_z, s0.z_w, size_t(ci.ntok) * 2, hipMemcpyDeviceToHost, h->stream));
    HIP_TRY(h, hipStreamSynchronize(h->stream));
  }
  // the skip counts of earlier iterations describe another assignment
  HIP_TRY(h, hipMemsetAsync(h->d.skip_hist, 0, 2 * sizeof(unsigned long long), h->stream));
  unsigned long long st[kStatsPerIter];
  HIP_TRY(h, hipMemcpyAsync(st, h->stats_base, sizeof(st), hipMemcpyDeviceToHost, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  LDA_TRY(check_stats(h, st));
  h->iteration = iteration;
  return LDA_OK;
}

}  // namespace lda
