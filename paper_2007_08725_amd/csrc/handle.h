// The handle behind the C ABI (include/lda.h) and the host helpers shared by
// the resident path (lda_api.cpp) and the out-of-core chunked path
// (chunks.cpp): status reporting, device allocation through the caller's
// hooks, and the launch bookkeeping.
#pragma once

#include <algorithm>
#include <memory>
#include <string>
#include <vector>

#include "lda_internal.h"

namespace lda {

extern thread_local std::string g_create_error;
constexpr int kStatSlots = 256;  // iterations between two statistics read-backs
constexpr int kEventsPerIter = 5;
struct ChunkMode;
void release_chunks(ChunkMode *cm);
struct ChunkModeDeleter {
  void operator()(ChunkMode *cm) const { release_chunks(cm); }
};

}  // namespace lda

struct lda_handle {
  // lda:: types; the handle itself is the opaque type of the C ABI
  lda::Layout L;  // host copy of the layout (only the parts needed later are kept)
  lda::DevState d{};
  lda::Params p{};
  hipStream_t stream = nullptr;
  bool own_stream = false;
  int device = 0;
  void *(*dev_alloc)(size_t, void *) = nullptr;
  void (*dev_free)(void *, void *) = nullptr;
  void *alloc_ctx = nullptr;
  std::vector<void *> allocations;
  unsigned long long *stats_base = nullptr;  // [kStatSlots * kStatsPerIter]
  std::vector<hipEvent_t> events;            // [kStatSlots * kEventsPerIter]
  void *noalloc_scratch = nullptr;           // this device's fixed LLPT scratch (lda_loglik_noalloc)
  // the light-word sampler runs beside the main sampler on a second stream
  hipStream_t side = nullptr;
  hipEvent_t fork_ev = nullptr, join_ev = nullptr;
  // out-of-core mode (lda_options.chunks > 1): the chunks, their host arrays
  // and the device slots they stream through; null when everything is resident
  std::unique_ptr<lda::ChunkMode, lda::ChunkModeDeleter> chunks;
  int32_t chunks_wanted = 0;  // lda_options.chunks
  int64_t iteration = 0;
  bool poisoned = false;
  std::string err = "no error";
};

namespace lda {

inline lda_status fail(lda_handle *h, lda_status st, const std::string &msg) {
  if (h) {
    h->err = msg;
    if (st == LDA_E_DEVICE) h->poisoned = true;
  } else {
    g_create_error = msg;
  }
  return st;
}

inline lda_status hip_fail(lda_handle *h, hipError_t e, const char *what) {
  return fail(h, e == hipErrorOutOfMemory ? LDA_E_NOMEM : LDA_E_DEVICE,
              std::string(what) + ": " + hipGetErrorString(e));
}

#define HIP_TRY(h, expr)                                  \
  do {                                                    \
    hipError_t e_ = (expr);                               \
    if (e_ != hipSuccess) return hip_fail((h), e_, #expr); \
  } while (0)

template <typename T>
inline lda_status dalloc(lda_handle *h, T **out, size_t count) {
  size_t bytes = std::max<size_t>(count, 1) * sizeof(T);
  bytes = (bytes + 255) & ~size_t(255);
  void *ptr = nullptr;
  if (h->dev_alloc) {
    ptr = h->dev_alloc(bytes, h->alloc_ctx);
    if (!ptr) return fail(h, LDA_E_NOMEM, "device allocation of " + std::to_string(bytes) + " bytes failed");
  } else {
    hipError_t e = hipMalloc(&ptr, bytes);
    if (e != hipSuccess) return fail(h, LDA_E_NOMEM, "hipMalloc(" + std::to_string(bytes) + "): " + hipGetErrorString(e));
  }
  h->allocations.push_back(ptr);
  *out = static_cast<T *>(ptr);
  return LDA_OK;
}

template <typename T>
inline lda_status upload(lda_handle *h, T *dst, const std::vector<T> &src) {
  if (src.empty()) return LDA_OK;
  HIP_TRY(h, hipMemcpyAsync(dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice, h->stream));
  return LDA_OK;
}

#define LDA_TRY(expr)                 \
  do {                                \
    lda_status s_ = (expr);           \
    if (s_ != LDA_OK) return s_;      \
  } while (0)

inline lda_status check_handle(lda_handle *h) {
  if (!h) return LDA_E_ARG;
  if (h->poisoned) return LDA_E_STATE;
  return LDA_OK;
}

inline lda_status check_errors(lda_handle *h, const unsigned long long *st) {
  if (st[ST_ERRORS]) return fail(h, LDA_E_DEVICE, "kernel found " + std::to_string(st[ST_ERRORS]) + " topic slots outside [0, K)");
  return LDA_OK;
}

template <typename T>
inline void dfree(lda_handle *h, T *&ptr) {
  if (!ptr) return;
  void *v = static_cast<void *>(ptr);
  auto it = std::find(h->allocations.begin(), h->allocations.end(), v);
  if (it != h->allocations.end()) h->allocations.erase(it);
  if (h->dev_alloc) h->dev_free(v, h->alloc_ctx);
  else (void)hipFree(v);
  ptr = nullptr;
}

// Stable radix sort of n (default: every token) key/value pairs on the
// handle's stream, with temporary storage allocated for the call.
inline lda_status sort_pairs(lda_handle *h, const uint32_t *keys_in, uint32_t *keys_out, const uint32_t *vals_in,
                      uint32_t *vals_out, unsigned end_bit, int64_t n = -1) {
  if (n < 0) n = h->L.n;
  size_t bytes = 0;
  HIP_TRY(h, sort_pairs_u32(nullptr, bytes, keys_in, keys_out, vals_in, vals_out, n, end_bit, h->stream));
  uint8_t *tmp = nullptr;
  LDA_TRY(dalloc(h, &tmp, bytes));
  HIP_TRY(h, sort_pairs_u32(tmp, bytes, keys_in, keys_out, vals_in, vals_out, n, end_bit, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  dfree(h, tmp);
  return LDA_OK;
}


// The documents of doc_off (M + 1 offsets) longer than kHeavyDocTokens.
inline std::vector<uint32_t> heavy_documents(const uint32_t *doc_off, uint32_t M) {
  std::vector<uint32_t> out;
  for (uint32_t q = 0; q < M; ++q)
    if (doc_off[q + 1] - doc_off[q] > kHeavyDocTokens) out.push_back(q);
  return out;
}

// Steps 4-6 of one iteration on h->stream: the light regions (one wave each)
// on the side stream, forked after the work queued so far and joined before
// whatever is queued next, beside the main sampler.
inline lda_status run_sampler(lda_handle *h, const DevState &d, const Params &p, uint32_t t) {
  const bool light = p.light_begin < p.n_regions;
  if (light) {
    HIP_TRY(h, hipEventRecord(h->fork_ev, h->stream));
    HIP_TRY(h, hipStreamWaitEvent(h->side, h->fork_ev, 0));
    HIP_TRY(h, launch_sampler_light(d, p, t, h->side));
    HIP_TRY(h, hipEventRecord(h->join_ev, h->side));
  }
  HIP_TRY(h, launch_sampler(d, p, t, h->stream));
  if (light) HIP_TRY(h, hipStreamWaitEvent(h->stream, h->join_ev, 0));
  return LDA_OK;
}

// Stream, workgroup sizes and grids for this device and K (lda_api.cpp).
lda_status setup_device(lda_handle *h, const lda_options *o);

// The out-of-core chunked mode (chunks.cpp); each mirrors the resident call.
// chunked_loglik with scratch = the fixed array of lda_loglik_noalloc keeps its
// partial sums there instead of in handle memory.
lda_status chunked_create(lda_handle *h, const int32_t *word, const int32_t *doc, int32_t R, int32_t n_chunks);
lda_status chunked_iterate(lda_handle *h, int32_t n_iters, lda_iter_stats *stats);
lda_status chunked_counts(lda_handle *h, lda_counts *out);
lda_status chunked_loglik(lda_handle *h, double *llpt, void *scratch);
lda_status chunked_set_assignments(lda_handle *h, const int32_t *z, int64_t iteration);

}  // namespace lda
