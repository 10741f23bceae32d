// Token layout on the device (lda_create): the two stable orders of Sec. 4.3
// built with rocPRIM radix sorts, plus the gathers/scatters that link them.
//
//   doc order : stable sort of input indices by document (skipped when the
//               input is already sorted by document)
//   word order: stable sort of doc-order positions by caller word id, then a
//               permutation of whole word segments into relabelled order
//               (descending count, Sec. 4.2), so that within a word the
//               documents ascend.
#include <rocprim/device/device_radix_sort.hpp>
#include <rocprim/iterator/counting_iterator.hpp>

#include "lda_internal.h"

namespace lda {
namespace {

constexpr int kThreads = 256;

inline uint32_t grid_for(int64_t n) {
  const int64_t b = (n + kThreads - 1) / kThreads;
  return uint32_t(std::min<int64_t>(std::max<int64_t>(b, 1), 1 << 20));
}

__global__ void k_gather_u32(uint32_t *__restrict__ dst, const int32_t *__restrict__ src,
                             const uint32_t *__restrict__ idx, int64_t n) {
  for (int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; p < n; p += int64_t(gridDim.x) * blockDim.x)
    dst[p] = uint32_t(src[idx[p]]);
}

// off[b] = first position whose key is >= b, for b in [0, nbins]; keys ascending.
__global__ void k_boundaries(const uint32_t *__restrict__ keys, int64_t n, uint32_t nbins, uint32_t *__restrict__ off) {
  for (int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; p < n; p += int64_t(gridDim.x) * blockDim.x) {
    const uint32_t k = keys[p];
    const int64_t prev = p == 0 ? -1 : int64_t(keys[p - 1]);
    for (int64_t b = prev + 1; b <= int64_t(k); ++b) off[b] = uint32_t(p);
    if (p == n - 1)
      for (int64_t b = int64_t(k) + 1; b <= int64_t(nbins); ++b) off[b] = uint32_t(n);
  }
}

// Word-order slot of every token: its position in the caller-id sort, moved
// with its whole word segment to the relabelled segment start.  Each
// word-ordered token records the offset of its document's D row.
__global__ void k_word_order(const uint32_t *__restrict__ wkey, const uint32_t *__restrict__ wpos, int64_t n,
                             const int32_t *__restrict__ relabel, const uint32_t *__restrict__ woff_orig,
                             const uint32_t *__restrict__ woff_new, const uint32_t *__restrict__ doc_sorted,
                             const int32_t *__restrict__ doc_in, const uint32_t *__restrict__ dt_key,
                             uint32_t *__restrict__ dt_word, uint32_t *__restrict__ dt_wpos,
                             const uint32_t *__restrict__ d_cap, uint2 *__restrict__ wt_kr) {
  for (int64_t q = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; q < n; q += int64_t(gridDim.x) * blockDim.x) {
    const uint32_t v = wkey[q];
    const uint32_t r = uint32_t(relabel[v]);
    const uint32_t j = woff_new[r] + (uint32_t(q) - woff_orig[v]);
    const uint32_t p = wpos[q];
    dt_word[p] = r;
    dt_wpos[p] = j;
    wt_kr[j] = make_uint2(dt_key ? dt_key[p] : p, d_cap[doc_sorted ? doc_sorted[p] : uint32_t(doc_in[p])]);
  }
}

__global__ void k_scatter_z(const uint16_t *__restrict__ z_w, const uint2 *__restrict__ wt_kr, int64_t n,
                            int32_t *__restrict__ z_in) {
  for (int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; j < n; j += int64_t(gridDim.x) * blockDim.x)
    z_in[wt_kr[j].x] = int32_t(z_w[j]);
}

__global__ void k_gather_z(const int32_t *__restrict__ z_in, const uint2 *__restrict__ wt_kr, int64_t n,
                           int32_t K, uint16_t *__restrict__ z_w, unsigned long long *__restrict__ bad) {
  unsigned long long nbad = 0;
  for (int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; j < n; j += int64_t(gridDim.x) * blockDim.x) {
    const int32_t z = z_in[wt_kr[j].x];
    if (z >= 0 && z < K) z_w[j] = uint16_t(z);
    else {
      z_w[j] = 0;
      nbad++;
    }
  }
  if (nbad) atomicAdd(bad, nbad);
}

// ----------------------------------------------------- out-of-core chunks --
// A chunk keeps only dt_wpos (word-order slot of each doc-ordered token) and
// its topics in host memory; the other per-token arrays are derived on the
// device when the chunk is loaded.

// dt_wpos[wpos[q]] = q: the word-order slot of each doc-order position, from
// the doc-order positions listed in word order.
__global__ void k_invert(const uint32_t *__restrict__ wpos, int64_t n, uint32_t *__restrict__ dt_wpos) {
  for (int64_t q = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; q < n; q += int64_t(gridDim.x) * blockDim.x)
    dt_wpos[wpos[q]] = uint32_t(q);
}

// slot_word[s] = the word of word-order slot s, one workgroup per region
// (the regions cover every slot exactly once).
__global__ void k_slot_words(const uint32_t *__restrict__ region, int64_t n_regions, uint2 *__restrict__ wt_kr) {
  for (int64_t r = blockIdx.x; r < n_regions; r += gridDim.x) {
    const uint32_t v = region[3 * r], b = region[3 * r + 1], e = region[3 * r + 2];
    for (uint32_t s = b + threadIdx.x; s < e; s += blockDim.x) wt_kr[s] = make_uint2(0u, v);
  }
}

// Per document, one wave: for each of its tokens p (slot s = dt_wpos[p]) the
// word id in doc order, and the key (key_base + p, the input index: chunks
// need input sorted by document) and D-row offset in word order.  The word of
// slot s (k_slot_words) waits in the second half of its (key, row offset)
// record, which the one token that owns the slot reads and then overwrites:
// one scattered 8-byte record per token, read and written in the same line.
__global__ void k_inflate(const uint32_t *__restrict__ doc_off, const uint32_t *__restrict__ d_cap, int32_t M,
                          const uint32_t *__restrict__ dt_wpos, uint32_t key_base, uint32_t *__restrict__ dt_word,
                          uint2 *__restrict__ wt_kr) {
  const int lane = threadIdx.x & 63, waves = int(blockDim.x) / 64;
  for (int64_t d = int64_t(blockIdx.x) * waves + threadIdx.x / 64; d < M; d += int64_t(gridDim.x) * waves) {
    const uint32_t b = doc_off[d], e = doc_off[d + 1], cap = d_cap[d];
    for (uint32_t p = b + uint32_t(lane); p < e; p += 64u) {
      const uint32_t s = dt_wpos[p];
      dt_word[p] = wt_kr[s].y;
      wt_kr[s] = make_uint2(key_base + p, cap);
    }
  }
}

// Topics in doc order (int32) from topics in word order, and back with a
// range check (bad counts topics outside [0, K), which are stored as 0).
__global__ void k_doc_gather_z(const uint32_t *__restrict__ dt_wpos, const uint16_t *__restrict__ z_w, int64_t n,
                               int32_t *__restrict__ z_doc) {
  for (int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; p < n; p += int64_t(gridDim.x) * blockDim.x)
    z_doc[p] = int32_t(z_w[dt_wpos[p]]);
}

__global__ void k_doc_scatter_z(const int32_t *__restrict__ z_doc, const uint32_t *__restrict__ dt_wpos, int64_t n,
                                int32_t K, uint16_t *__restrict__ z_w, unsigned long long *__restrict__ bad) {
  unsigned long long nbad = 0;
  for (int64_t p = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; p < n; p += int64_t(gridDim.x) * blockDim.x) {
    const int32_t z = z_doc[p];
    const bool ok = z >= 0 && z < K;
    z_w[dt_wpos[p]] = ok ? uint16_t(z) : uint16_t(0);
    nbad += ok ? 0ull : 1ull;
  }
  if (nbad) atomicAdd(bad, nbad);
}

}  // namespace

hipError_t launch_invert(const uint32_t *wpos, int64_t n, uint32_t *dt_wpos, hipStream_t s) {
  hipLaunchKernelGGL(k_invert, dim3(grid_for(n)), dim3(kThreads), 0, s, wpos, n, dt_wpos);
  return hipGetLastError();
}

hipError_t launch_inflate(const uint32_t *region, int64_t n_regions, const uint32_t *doc_off, const uint32_t *d_cap,
                          int32_t M, const uint32_t *dt_wpos, uint32_t key_base, uint32_t *dt_word, uint2 *wt_kr,
                          hipStream_t s) {
  const uint32_t rg = uint32_t(std::min<int64_t>(std::max<int64_t>(n_regions, 1), 1 << 16));
  hipLaunchKernelGGL(k_slot_words, dim3(rg), dim3(kThreads), 0, s, region, n_regions, wt_kr);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  const int64_t waves = kThreads / 64;
  const uint32_t dg = uint32_t(std::min<int64_t>(std::max<int64_t>((int64_t(M) + waves - 1) / waves, 1), 1 << 16));
  hipLaunchKernelGGL(k_inflate, dim3(dg), dim3(kThreads), 0, s, doc_off, d_cap, M, dt_wpos, key_base, dt_word, wt_kr);
  return hipGetLastError();
}

hipError_t launch_doc_gather_z(const uint32_t *dt_wpos, const uint16_t *z_w, int64_t n, int32_t *z_doc, hipStream_t s) {
  hipLaunchKernelGGL(k_doc_gather_z, dim3(grid_for(n)), dim3(kThreads), 0, s, dt_wpos, z_w, n, z_doc);
  return hipGetLastError();
}

hipError_t launch_doc_scatter_z(const int32_t *z_doc, const uint32_t *dt_wpos, int64_t n, int32_t K, uint16_t *z_w,
                                unsigned long long *bad, hipStream_t s) {
  hipLaunchKernelGGL(k_doc_scatter_z, dim3(grid_for(n)), dim3(kThreads), 0, s, z_doc, dt_wpos, n, K, z_w, bad);
  return hipGetLastError();
}

unsigned bits_for(uint64_t max_value) {
  unsigned b = 1;
  while (b < 32 && (max_value >> b)) ++b;
  return b;
}

hipError_t sort_pairs_u32(void *tmp, size_t &tmp_bytes, const uint32_t *keys_in, uint32_t *keys_out,
                          const uint32_t *vals_in, uint32_t *vals_out, int64_t n, unsigned end_bit, hipStream_t s) {
  const size_t size = size_t(n);
  if (vals_in)
    return rocprim::radix_sort_pairs(tmp, tmp_bytes, keys_in, keys_out, vals_in, vals_out, size, 0u, end_bit, s);
  return rocprim::radix_sort_pairs(tmp, tmp_bytes, keys_in, keys_out, rocprim::counting_iterator<uint32_t>(0u),
                                   vals_out, size, 0u, end_bit, s);
}

hipError_t launch_gather_u32(uint32_t *dst, const int32_t *src, const uint32_t *idx, int64_t n, hipStream_t s) {
  hipLaunchKernelGGL(k_gather_u32, dim3(grid_for(n)), dim3(kThreads), 0, s, dst, src, idx, n);
  return hipGetLastError();
}

hipError_t launch_boundaries(const uint32_t *keys, int64_t n, uint32_t nbins, uint32_t *off, hipStream_t s) {
  hipLaunchKernelGGL(k_boundaries, dim3(grid_for(n)), dim3(kThreads), 0, s, keys, n, nbins, off);
  return hipGetLastError();
}

hipError_t launch_word_order(const uint32_t *wkey, const uint32_t *wpos, int64_t n, const int32_t *relabel,
                             const uint32_t *woff_orig, const uint32_t *woff_new, const uint32_t *doc_sorted,
                             const int32_t *doc_in, const uint32_t *dt_key, uint32_t *dt_word, uint32_t *dt_wpos,
                             const uint32_t *d_cap, uint2 *wt_kr, hipStream_t s) {
  hipLaunchKernelGGL(k_word_order, dim3(grid_for(n)), dim3(kThreads), 0, s, wkey, wpos, n, relabel, woff_orig,
                     woff_new, doc_sorted, doc_in, dt_key, dt_word, dt_wpos, d_cap, wt_kr);
  return hipGetLastError();
}

hipError_t launch_scatter_z(const uint16_t *z_w, const uint2 *wt_kr, int64_t n, int32_t *z_in, hipStream_t s) {
  hipLaunchKernelGGL(k_scatter_z, dim3(grid_for(n)), dim3(kThreads), 0, s, z_w, wt_kr, n, z_in);
  return hipGetLastError();
}

hipError_t launch_gather_z(const int32_t *z_in, const uint2 *wt_kr, int64_t n, int32_t K, uint16_t *z_w,
                           unsigned long long *bad, hipStream_t s) {
  hipLaunchKernelGGL(k_gather_z, dim3(grid_for(n)), dim3(kThreads), 0, s, z_in, wt_kr, n, K, z_w, bad);
  return hipGetLastError();
}

}  // namespace lda
