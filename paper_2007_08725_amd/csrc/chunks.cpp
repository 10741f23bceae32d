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
  uint32_t d_slots = 0;         // D-row slots of the chunk's documents
  Params p{};                   // launch parameters of the chunk
};

struct ChunkSlot {
  uint32_t *dt_word = nullptr, *dt_wpos = nullptr, *wt_key = nullptr, *wt_rowoff = nullptr;
  uint32_t *skip_bits = nullptr, *d_ent = nullptr;
  uint16_t *z_w = nullptr;
  hipEvent_t loaded = nullptr, computed = nullptr, unloaded = nullptr;
};

struct ChunkMode {
  std::vector<ChunkInfo> c;
  ChunkSlot slot[2];
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
  if (cm->h2d) (void)hipStreamDestroy(cm->h2d);
  if (cm->d2h) (void)hipStreamDestroy(cm->d2h);
  delete cm;
}

}  // namespace lda
