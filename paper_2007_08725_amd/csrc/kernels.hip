// Device kernels of liblda for gfx950 (CDNA4, wave64).
//
// One synchronous iteration (Sec. 2.2, 3.2, 4.3):
//   k_begin      den[k] = T[k] + V*beta; scheduler counters reset
//   k_word_pre_wave
//                per word: top-3 of W^[v] (K1, K2, a1..a3), Q' and sum W^   (step 1, Sec. 3.2)
//   k_clear_skips
//                the skip bitmap (one bit per word-ordered token) cleared
//   k_doc_pass   per document: C1, C2 by lookup in the D row, u, M, S_est
//                and the skip test; sets the bit of every skipped token    (steps 2-3, Sec. 3.3)
//   k_sampler    per region of a word: W^ row and Q' block prefix in LDS,
//                then for every token whose bit is clear C1 and S' over
//                nz(D[d]) and the final draw over [K1 | S' | Q']; every
//                topic slot of the region written (K1 for the skipped)     (steps 4-6, Sec. 4.3)
//   k_zero_split, k_rebuild_w_wave, k_rebuild_d
//                count tables of the new assignment: dense rows of W by
//                histogram (integer atomics for split words), sparse rows of
//                W and rows of D as packed (topic << 16 | count) entries, T
//                                                                          (Sec. 4.2-4.3)
// All floating point is fp64 (IEEE divide for W^), built without
// contraction so that the values match a plain sequential evaluation.
#include "lda_internal.h"

#include <mutex>

namespace lda {
namespace {

constexpr int kWave = 64;
constexpr int kGroup = 16;  // lanes that cooperate on one token in the sampler
constexpr uint32_t kGroupMask = (1u << kGroup) - 1u;

// ------------------------------------------------------------- Philox ----
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of
//   (c0, c1, c2, c3) -> (hi(M1*c2) ^ c1 ^ k0, lo(M1*c2), hi(M0*c0) ^ c3 ^ k1, lo(M0*c0))
// with the key bumped by the Weyl constants between rounds.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint64_t p0 = uint64_t(0xD2511F53u) * c.x, p1 = uint64_t(0xCD9E8D57u) * c.z;  // one 32x32->64 product each
    const uint32_t lo0 = uint32_t(p0), hi0 = uint32_t(p0 >> 32);
    const uint32_t lo1 = uint32_t(p1), hi1 = uint32_t(p1 >> 32);
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// u in [0,1) for token i (input order) at iteration t: counter (i, 0, t, 0).
// The key and t pass through an empty asm so that the compiler computes the
// key schedule where the draw is made instead of keeping twenty hoisted
// round keys live (in the sampler they would spill).
__device__ __forceinline__ double uniform_draw(uint64_t seed, uint32_t t, uint32_t i) {
  uint32_t k0 = uint32_t(seed), k1 = uint32_t(seed >> 32);
  asm volatile("" : "+s"(k0), "+s"(k1), "+s"(t));
  const uint4 x = philox4x32_10(make_uint4(i, 0u, t, 0u), k0, k1);
  const uint64_t bits = (uint64_t(x.x) << 32) | uint64_t(x.y);
  return double(bits >> 11) * 0x1p-53;
}

// W^[v][k] exactly as the paper defines it: an IEEE fp64 divide.
__device__ __forceinline__ double what(uint32_t count, double beta, double den) { return (double(count) + beta) / den; }

// -------------------------------------------------- wave / group helpers --
template <int W>
__device__ __forceinline__ double group_sum(double v) {
#pragma unroll
  for (int o = W / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, W);
  return v;
}

template <int W>
__device__ __forceinline__ uint32_t group_sum_u32(uint32_t v) {
#pragma unroll
  for (int o = W / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, W);
  return v;
}

template <int W>
__device__ __forceinline__ unsigned long long group_sum_u64(unsigned long long v) {
#pragma unroll
  for (int o = W / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, W);
  return v;
}

template <int W>
__device__ __forceinline__ double group_incl_scan(double v, int li) {
#pragma unroll
  for (int o = 1; o < W; o <<= 1) {
    const double y = __shfl_up(v, o, W);
    if (li >= o) v += y;
  }
  return v;
}

// Shift a double right by S lanes inside each row of 16 lanes (DPP
// row_shr); lanes below S read 0.
template <int S>
__device__ __forceinline__ double row_shr(double v) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), 0x110 + S, 0xF, 0xF, true);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), 0x110 + S, 0xF, 0xF, true);
  return __hiloint2double(hi, lo);
}

// Inclusive prefix sum over each row of 16 lanes.
__device__ __forceinline__ double row_incl_scan(double v) {
  v += row_shr<1>(v);
  v += row_shr<2>(v);
  v += row_shr<4>(v);
  v += row_shr<8>(v);
  return v;
}

// A double from another lane by a DPP control, in the rows of row_mask only
// (the other rows read 0).
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_rows_f64(double v) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, ROWS, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, ROWS, 0xF, false);
  return __hiloint2double(hi, lo);
}

// Inclusive prefix sum over the 64 lanes of a wave: a scan per row, then
// row 0's total added to row 1 and row 2's to row 3 (row_bcast:15), then the
// total of rows 0 and 1 added to rows 2 and 3 (row_bcast:31).
__device__ __forceinline__ double wave_incl_scan(double v) {
  v = row_incl_scan(v);
  v += dpp_rows_f64<0x142, 0xA>(v);
  v += dpp_rows_f64<0x143, 0xC>(v);
  return v;
}

constexpr int kTop = 4;  // top values of W^[v] kept per word (a1..a4 of Eq. 9, g <= 3)

struct TopN {
  double v[kTop];
  uint32_t k[kTop];
};

__device__ __forceinline__ bool better(double va, uint32_t ka, double vb, uint32_t kb) {
  return va > vb || (va == vb && ka < kb);
}

// Insert (v, k) into a list kept in order of `better` (value descending,
// lowest topic id first among equal values).
__device__ __forceinline__ void top_insert(TopN &t, double v, uint32_t k) {
  if (!better(v, k, t.v[kTop - 1], t.k[kTop - 1])) return;
  t.v[kTop - 1] = v;
  t.k[kTop - 1] = k;
#pragma unroll
  for (int q = kTop - 1; q > 0; --q) {
    if (better(t.v[q], t.k[q], t.v[q - 1], t.k[q - 1])) {
      const double tv = t.v[q - 1];
      const uint32_t tk = t.k[q - 1];
      t.v[q - 1] = t.v[q];
      t.k[q - 1] = t.k[q];
      t.v[q] = tv;
      t.k[q] = tk;
    }
  }
}

// Block-wide sum of a double over 256 threads (fixed order).
__device__ double block_sum(double v, double *red) {
  v = group_sum<kWave>(v);
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  __syncthreads();
  if (lane == 0) red[wave] = v;
  __syncthreads();
  double s = 0.0;
  for (int q = 0; q < kBlock / kWave; ++q) s += red[q];
  __syncthreads();
  return s;
}

// Block-wide exclusive prefix of a uint32 over 256 threads; *total gets the sum.
__device__ uint32_t block_exclusive_u32(uint32_t v, uint32_t *red, uint32_t *total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  uint32_t incl = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t y = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += y;
  }
  __syncthreads();
  if (lane == kWave - 1) red[wave] = incl;
  __syncthreads();
  uint32_t off = 0, all = 0;
  for (int q = 0; q < kBlock / kWave; ++q) {
    if (q < wave) off += red[q];
    all += red[q];
  }
  *total = all;
  return off + incl - v;
}

// First index in [0, nnz) whose packed topic is >= k.
__device__ __forceinline__ uint32_t row_lower_bound(const uint32_t *__restrict__ row, uint32_t nnz, uint32_t k) {
  uint32_t lo = 0, hi = nnz;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if ((row[mid] >> 16) < k) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// ------------------------------------------------------------ kernels ----

__device__ __forceinline__ uint16_t initial_topic(uint64_t seed, uint32_t i, int32_t K) {
  const uint4 x = philox4x32_10(make_uint4(i, 0u, 0u, 1u), uint32_t(seed), uint32_t(seed >> 32));
  return uint16_t((uint64_t(x.x) * uint64_t(uint32_t(K))) >> 32);
}

__global__ void k_init_topics(const uint2 *__restrict__ wt_kr, uint16_t *__restrict__ z_w, int64_t n, int32_t K,
                              uint64_t seed) {
  for (int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; j < n; j += int64_t(gridDim.x) * blockDim.x)
    z_w[j] = initial_topic(seed, wt_kr[j].x, K);
}

// The skip bitmaps start every iteration clear, and so does this
// iteration's skip count (the other parity's count, the previous
// iteration's, stays for the choice of bitmap).
__global__ void k_clear_skips(uint32_t *__restrict__ bits, uint32_t *__restrict__ doc_bits, int64_t n, int64_t n_doc,
                              unsigned long long *__restrict__ hist, uint32_t t, int reset_count) {
  const int64_t i0 = int64_t(blockIdx.x) * blockDim.x + threadIdx.x, step = int64_t(gridDim.x) * blockDim.x;
  for (int64_t q = i0; q < n; q += step) bits[q] = 0u;
  if (doc_bits)
    for (int64_t q = i0; q < n_doc; q += step) doc_bits[q] = 0u;
  if (i0 == 0 && reset_count) hist[t & 1u] = 0ull;
}

__global__ void k_reset_counters(uint32_t *__restrict__ counters) {
  if (threadIdx.x < kCounters) counters[threadIdx.x] = 0u;
}

// Whether iteration t carries its skip decisions in the document-ordered
// bitmap: coalesced writes in the doc pass and one dependent read per token
// in the sampler, against one scattered write per skipped token for the
// word-ordered bitmap.  By default it does once the previous iteration
// skipped more than a fifth of the tokens, where the scattered writes cost
// more than the reads.
__device__ __forceinline__ bool doc_marks(const DevState &d, const Params &p, uint32_t t) {
  if (!p.doc_marks_ok || p.skip_marks == 1) return false;
  if (p.skip_marks == 2) return true;
  return t > 0u && 5ull * d.skip_hist[(t + 1u) & 1u] > uint64_t(p.n_all);
}

// Whether steps 2-3 run in iteration t.  They only save work: a token they
// skip costs the sampler a bit test instead of its D row, so they pay once
// enough tokens skip (the doc pass costs about as much as the sampler work of
// a tenth of the tokens).  By default they run in every kProbeEvery-th
// iteration, which measures the skip rate, and in every iteration after one
// that skipped at least an eighth of the tokens; a token left unmarked is
// drawn in full, so the draws are the same either way.
constexpr uint32_t kProbeEvery = 8;
__device__ __forceinline__ bool skip_test_runs(const DevState &d, const Params &p, uint32_t t) {
  if (p.no_skip) return false;
  if (p.always_skip_test || t % kProbeEvery == 0u) return true;
  return 8ull * d.skip_hist[(t + 1u) & 1u] >= uint64_t(p.n_all);
}

__global__ void k_begin(const uint32_t *__restrict__ T, double *__restrict__ den, double *__restrict__ bden, int32_t K,
                        double beta, double vbeta, uint32_t *__restrict__ counters,
                        unsigned long long *__restrict__ stats) {
  const int k = blockIdx.x * blockDim.x + threadIdx.x;
  if (k < K) {
    const double dk = double(T[k]) + vbeta;
    den[k] = dk;
    bden[k] = what(0u, beta, dk);  // W^[v][k] of every topic that word v does not hold
  }
  if (blockIdx.x == 0 && threadIdx.x < kCounters) {
    counters[threadIdx.x] = 0u;
    if (stats && threadIdx.x < kStatsPerIter) stats[threadIdx.x] = 0ull;
  }
}

// Step 1 of Sec. 3.2 and the per-word Q' of Sec. 2.2 (built once per word).
struct WordTop {
  uint32_t k1, k2, k3;
  double a1, a2, a3, a4;
};

// The sampler's and the skip test's per-word records.  In two-branch mode
// (Sec. 2.2) the max-topic branch is empty (a1 = 0, K1 = K, a topic no row
// holds with a count) and Q' is the full Q.
__device__ void write_word_records(const DevState &d, const Params &p, int r, const WordTop &top, double q, double sw) {
  const int K = p.K;
  const uint32_t K3 = K >= 3 ? top.k3 : 0xFFFFFFFFu;
  WordRec rec;
  rec.a1 = p.two_branch ? 0.0 : top.a1;
  rec.a2 = top.a2;
  rec.a3 = K >= 3 ? top.a3 : 0.0;
  rec.qp = q;
  rec.sumw = sw;
  rec.k1 = p.two_branch ? uint32_t(K) : top.k1;
  rec.k2 = top.k2;
  d.wrec[r] = rec;
  SkipRec sr;
  sr.k12 = top.k1 | (top.k2 << 16);
  sr.k3 = K3;
  sr.a1 = float(top.a1);
  sr.a2 = float(top.a2);
  sr.a3 = float(K >= 3 ? top.a3 : 0.0);
  sr.a4 = float(K >= 4 ? top.a4 : 0.0);
  sr.qp = float(q);
  sr.pad = 0u;
  d.wskip[r] = sr;
}

// Large K: the sum over all topics of beta/den[k] (one workgroup, a fixed
// order), for the sparse words' sums in k_word_pre_wave.
__global__ __launch_bounds__(kBlock) void k_beta_sum(DevState d, Params p) {
  __shared__ double red[kBlock / kWave];
  const int K = p.K;
  const int cs = (K + kBlock - 1) / kBlock;
  const int c0 = min(K, int(threadIdx.x) * cs), c1 = min(K, c0 + cs);
  double s = 0.0;
  for (int k = c0; k < c1; ++k) s += d.bden[k];
  s = block_sum(s, red);
  if (threadIdx.x == 0) d.beta_sum[0] = s;
}

// Step 1 (Sec. 3.2) and Q' (Sec. 2.2), one wave per word, four words per
// workgroup, no workgroup barriers.  Lane l takes topics l, l + 64, ...: its top values, then a merge
// across the wave by exchanges at distances 32 down to 1 (the top set is
// unique under `better`, so every lane ends with the same list), then Q' and
// the sum of W^[v] per lane in topic order, summed over the wave.  Below
// K = 4,096 a sparse row is spread into the wave's table of K counts first.
// From K = 4,096 on (p.sparse_pre) a sparse word's W^ is beta/den[k] outside
// its row: its top values come from the row and from the first topics
// outside the row in the list of all topics by ascending T (descending
// beta/den[k], lowest id first on ties), 64 candidates of the list at a time;
// its sums from the sum of beta/den[k] over all topics, corrected on the
// row.  Should the list run out, every topic is scanned.
__device__ __forceinline__ void wave_top_merge(TopN &t) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) {
    double pv[kTop];
    uint32_t pk[kTop];
#pragma unroll
    for (int q = 0; q < kTop; ++q) {
      pv[q] = __shfl_xor(t.v[q], o, kWave);
      pk[q] = uint32_t(__shfl_xor(int(t.k[q]), o, kWave));
    }
#pragma unroll
    for (int q = 0; q < kTop; ++q) top_insert(t, pv[q], pk[q]);
  }
}
__device__ __forceinline__ WordTop word_top_of(const TopN &t) {
  WordTop top;
  top.k1 = t.k[0];
  top.k2 = t.k[1];
  top.k3 = t.k[2];
  top.a1 = t.v[0];
  top.a2 = t.v[1];
  top.a3 = t.v[2] > 0.0 ? t.v[2] : 0.0;
  top.a4 = t.v[3] > 0.0 ? t.v[3] : 0.0;
  return top;
}
__global__ __launch_bounds__(kBlock) void k_word_pre_wave(DevState d, Params p) {
  extern __shared__ uint16_t wtab[];  // below K = 4,096: [kBlock / kWave][(K + 1) & ~1]
  const int K = p.K, lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int r = blockIdx.x * (kBlock / kWave) + wave;
  if (r >= p.n_present) return;  // a whole wave; nothing below waits on the workgroup
  const bool dense = r < p.n_dense;
  const int32_t *wrow = dense ? d.w_dense + size_t(r) * size_t(K) : nullptr;
  const uint32_t *ents = nullptr;
  uint32_t nnz = 0;
  if (!dense) {
    const int s = r - p.n_dense;
    ents = d.ws_ent + d.ws_cap[s];
    nnz = d.ws_nnz[s];
  }
  TopN t;
  auto reset = [&]() {
    for (int q = 0; q < kTop; ++q) {
      t.v[q] = -1.0;
      t.k[q] = 0xFFFFFFFFu;
    }
  };
  reset();
  if (!dense && p.sparse_pre) {
    double snz = 0.0, sb = 0.0;
    for (uint32_t q = uint32_t(lane); q < nnz; q += kWave) {
      const uint32_t ent = ents[q], k = ent >> 16;
      const double w = what(ent & 0xFFFFu, p.beta, d.den[k]);
      top_insert(t, w, k);
      snz += w;
      sb += d.bden[k];
    }
    const uint32_t want = uint32_t(min(kTop, K - int(nnz)));
    uint32_t found = 0;
    for (int i0 = 0; i0 < p.top_list && found < want; i0 += kWave) {
      const int i = i0 + lane;
      bool cand = false;
      uint32_t k = 0;
      if (i < p.top_list) {
        k = d.topic_order[i];
        const uint32_t lb = row_lower_bound(ents, nnz, k);
        cand = !(lb < nnz && (ents[lb] >> 16) == k);
      }
      const unsigned long long m = __ballot(cand);
      const uint32_t rank = __builtin_amdgcn_mbcnt_hi(uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u));
      if (cand && rank < want - found) top_insert(t, d.bden[k], k);
      found += min(uint32_t(__popcll(m)), want - found);
    }
    wave_top_merge(t);
    snz = group_sum<kWave>(snz);
    sb = group_sum<kWave>(sb);
    if (found >= want) {
      const WordTop top = word_top_of(t);
      if (lane == 0) {
        const double sw = (d.beta_sum[0] - sb) + snz;
        write_word_records(d, p, r, top, p.two_branch ? p.alpha * sw : p.alpha * (sw - top.a1), sw);
      }
      return;
    }
    reset();  // the list ran out: every topic below
  }
  const bool tab = !dense && !p.sparse_pre;
  uint16_t *ct = wtab + size_t(wave) * size_t((K + 1) & ~1);
  if (tab) {
    for (int k = lane; k < K; k += kWave) ct[k] = 0;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");  // a wave's LDS accesses run in order
    for (uint32_t q = uint32_t(lane); q < nnz; q += kWave) {
      const uint32_t ent = ents[q];
      ct[ent >> 16] = uint16_t(ent & 0xFFFFu);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  // counts: the dense row, the table, or (a large-K sparse row whose topic
  // list ran out) a search of the row
  auto count_of = [&](int k) -> uint32_t {
    if (dense) return uint32_t(wrow[k]);
    if (tab) return uint32_t(ct[k]);
    const uint32_t lb = row_lower_bound(ents, nnz, uint32_t(k));
    return lb < nnz && (ents[lb] >> 16) == uint32_t(k) ? (ents[lb] & 0xFFFFu) : 0u;
  };
  // kPreAhead topics per lane at a time, their loads issued together (a
  // dense row at K = 32,768 is 512 topics per lane)
  constexpr int kPreAhead = 8;
  auto batch = [&](int k0, double (&w)[kPreAhead]) {
    uint32_t c[kPreAhead];
    double dn[kPreAhead];
#pragma unroll
    for (int u = 0; u < kPreAhead; ++u) {
      const int k = min(k0 + u * kWave, K - 1);
      c[u] = count_of(k);
      dn[u] = d.den[k];
    }
#pragma unroll
    for (int u = 0; u < kPreAhead; ++u) w[u] = what(c[u], p.beta, dn[u]);
  };
  for (int k0 = lane; k0 < K; k0 += kPreAhead * kWave) {
    double w[kPreAhead];
    batch(k0, w);
#pragma unroll
    for (int u = 0; u < kPreAhead; ++u)
      if (k0 + u * kWave < K) top_insert(t, w[u], uint32_t(k0 + u * kWave));
  }
  wave_top_merge(t);
  const WordTop top = word_top_of(t);
  double q = 0.0, sw = 0.0;
  for (int k0 = lane; k0 < K; k0 += kPreAhead * kWave) {
    double w[kPreAhead];
    batch(k0, w);
#pragma unroll
    for (int u = 0; u < kPreAhead; ++u) {
      const int k = k0 + u * kWave;
      if (k < K) {
        sw += w[u];
        if (p.two_branch || uint32_t(k) != top.k1) q += p.alpha * w[u];
      }
    }
  }
  q = group_sum<kWave>(q);
  sw = group_sum<kWave>(sw);
  if (lane == 0) write_word_records(d, p, r, top, q, sw);
}

// Steps 2 and 3: per document, C1 = D[d][K1], C2 = D[d][K2], u, M, S_est and
// the skip test (Eq. 7 and 9).  One wave per document; documents are handed
// out in batches through an atomic counter.  The document's D row is spread
// into a per-wave topic -> count table in LDS, so each token's C1 and C2 are
// two LDS reads; the table is cleared again from the row afterwards.
constexpr uint32_t kDocBatch = 32;
// Documents per batch of the D rebuild: a smaller window of documents in
// flight keeps more of its topic gathers in the caches (at 16 and below the
// counters' atomics start to bound the kernel).
constexpr uint32_t kRebuildBatch = 24;

// Next batch [d0, d1) of documents for a wave of the D rebuild.  The
// documents are split into kXcds ranges of equal token counts; workgroups are
// dealt to the XCDs in turn, so blockIdx.x % kXcds names the wave's XCD, and
// a wave takes batches from its own XCD's range first, then from the others
// in turn.  Each XCD's L2 then sees a compact window of documents, and the
// word-ordered topic slots that window gathers are fetched by one XCD
// instead of all of them.
__device__ __forceinline__ bool next_docs(uint32_t *__restrict__ cnt, const Params &p, int &part, int lane,
                                          uint32_t &d0, uint32_t &d1) {
  const int x = int(blockIdx.x % kXcds);
  while (part < kXcds) {
    const int r = (x + part) % kXcds;
    uint32_t o = 0;
    if (lane == 0) o = atomicAdd(&cnt[r], kRebuildBatch);
    o = __shfl(o, 0);
    const uint32_t b = p.xcd_doc[r] + o, e = p.xcd_doc[r + 1];
    if (o < e - p.xcd_doc[r]) {
      d0 = b;
      d1 = min(b + kRebuildBatch, e);
      return true;
    }
    ++part;
  }
  return false;
}

// The fields of a skip record that the test needs at g <= 2 (the first 20
// bytes of the record: one 16-byte and one 4-byte load).
struct SkipHead {
  uint32_t k12;
  float a1, a2, a3, qp;
};
__device__ __forceinline__ SkipHead skip_head(const SkipRec *__restrict__ r) {
  return SkipHead{r->k12, r->a1, r->a2, r->a3, r->qp};
}

constexpr int kDocAhead = 2;  // chunks of 64 tokens per document loaded one document ahead

// Documents longer than this are walked by a whole workgroup in the doc pass
// and the D rebuild (the skew-aware mapping of Sec. 5.1: heavy units to
// workgroups, light ones to waves); the per-wave kernels skip them.
constexpr uint32_t kHeavyDoc = kHeavyDocTokens;

// Step 3 for token pp of a document of length len, in single precision with a
// relative margin of 2^-15, far above the fp32 rounding of these few
// operations (a few 2^-24): a token is skipped only if u*(M + S_est + Q') < M
// holds exactly, so its draw is K1 (S' <= S_est, Eq. 8-9).  cmap is the
// document's topic -> count table.
template <bool KeyId>
__device__ __forceinline__ bool skip_test(const DevState &d, const Params &p, uint32_t t, const uint16_t *cmap,
                                          uint32_t pp, uint32_t len, const SkipHead &h, uint32_t v) {
  const uint32_t K1 = h.k12 & 0xFFFFu, K2 = h.k12 >> 16;
  const uint32_t C1 = cmap[K1], C2 = cmap[K2];
  const uint32_t key = KeyId ? p.key_base + pp : d.dt_key[pp];
  const float u = float(uniform_draw(p.seed, t, key));
  const float Mm = h.a1 * (float(C1) + p.alpha_f);
  float Sest;
  if (p.g == 1) {
    Sest = h.a2 * float(len - C1);
  } else if (p.g == 2) {
    Sest = h.a2 * float(C2) + h.a3 * float(len - C1 - C2);
  } else {
    const SkipRec &r = d.wskip[v];
    const uint32_t C3 = r.k3 < uint32_t(p.K) ? uint32_t(cmap[r.k3]) : 0u;
    Sest = h.a2 * float(C2) + h.a3 * float(C3) + r.a4 * float(len - C1 - C2 - C3);
  }
  return !p.no_skip && (u * ((Mm + Sest) + h.qp) < Mm * (1.0f - 0x1p-15f));
}

// A skipped token's decision goes to the sampler either as a bit at its
// word-order slot (one scattered write per skipped token) or, in the
// document-ordered bitmap, as a bit at its document position: a chunk's 64
// bits (lanes = positions p0 + lane) from a ballot, in at most three words,
// whose neighbours other waves may set too.
__device__ __forceinline__ void mark_slot(const DevState &d, uint32_t slot) {
  atomicOr(&d.skip_bits[slot >> 5], 1u << (slot & 31u));
}
__device__ __forceinline__ void mark_chunk(const DevState &d, unsigned long long m, uint32_t p0, int lane) {
  if (m == 0ull) return;
  const uint32_t sh = p0 & 31u;
  const uint32_t v0 = uint32_t(m << sh);
  const uint32_t v1 = sh ? uint32_t(m >> (32u - sh)) : uint32_t(m >> 32);
  const uint32_t v2 = sh ? uint32_t(m >> (64u - sh)) : 0u;
  const uint32_t v = lane == 0 ? v0 : lane == 1 ? v1 : v2;
  if (lane < 3 && v != 0u) atomicOr(&d.skip_doc[(p0 >> 5) + uint32_t(lane)], v);
}

template <bool KeyId>
__device__ void heavy_doc_pass(const DevState &d, const Params &p, uint32_t t, uint16_t *__restrict__ cmap,
                               bool by_doc, unsigned long long &nskip);

// Steps 2-3 per document (Sec. 3.3): the D row spread into a per-wave
// topic -> count table in LDS, then for every token C1 and C2 by lookup, u,
// M, S_est and the skip test.  A skipped token's bit is set in the
// word-ordered skip bitmap (one scattered bit at its word-order slot) or, in
// the iterations doc_marks chooses, in the document-ordered one (coalesced
// bits at its document position); the sampler writes K1 into its slot with
// the rest of its batch.  KeyId: the input is sorted by document, so a
// token's key (its input index) is its document-order position.
template <bool KeyId>
__global__ __launch_bounds__(kBlock) void k_doc_pass(DevState d, Params p, uint32_t t,
                                                     unsigned long long *__restrict__ stats) {
  extern __shared__ uint16_t cmap_all[];
  if (!skip_test_runs(d, p, t)) return;  // uniform over the grid
  if (blockIdx.x == 0 && threadIdx.x == 0) stats[ST_TEST_RAN] = 1ull;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int K = p.K;
  uint16_t *cmap = cmap_all + size_t(wave) * size_t(K);
  for (int k = lane; k < K; k += kWave) cmap[k] = 0;
  unsigned long long nskip = 0;
  const bool by_doc = doc_marks(d, p, t);
  // the heavy documents first, each by the whole workgroup (wave 0's table shared)
  if (p.n_heavy) heavy_doc_pass<KeyId>(d, p, t, cmap_all, by_doc, nskip);
  const uint32_t M = uint32_t(p.M);
  const uint32_t last = uint32_t(p.n - 1);
  auto test = [&](uint32_t pp, uint32_t len, const SkipHead &h, uint32_t v) -> bool {
    return skip_test<KeyId>(d, p, t, cmap, pp, len, h, v);
  };
  for (;;) {
    uint32_t d0 = 0;
    if (lane == 0) d0 = atomicAdd(&d.counters[CNT_DOCPASS], kDocBatch);
    d0 = __builtin_amdgcn_readfirstlane(__shfl(d0, 0));
    if (d0 >= M) break;
    const int nd = int(min(M, d0 + kDocBatch) - d0);
    // the batch's document offsets and row offsets, one per lane
    const uint32_t offv = lane <= nd ? d.doc_off[d0 + uint32_t(lane)] : 0u;
    const uint32_t capv = lane < nd ? d.d_cap[d0 + uint32_t(lane)] : 0u;
    // Pipeline over the first kDocAhead*64 tokens and row slots of each
    // document: while document i is processed, the first row slots of
    // document i+1 (its header and entries), the skip records of the words
    // of document i+1 and the word ids of document i+2 are loaded.  Every
    // load is issued (indexes past the batch are clamped; lanes past a
    // document's end read word 0's record), so that the waits count a fixed
    // number of loads.
    auto rows_of = [&](int doc, uint32_t (&r)[kDocAhead]) {
      const uint32_t cap = __builtin_amdgcn_readlane(capv, doc);  // 0 past the batch; kRowPad covers the reach
#pragma unroll
      for (int c = 0; c < kDocAhead; ++c) r[c] = d.d_ent[cap + uint32_t(c * kWave + lane)];
    };
    auto words_of = [&](int doc, uint32_t (&w)[kDocAhead]) {
      const uint32_t bn = __builtin_amdgcn_readlane(offv, doc);
#pragma unroll
      for (int c = 0; c < kDocAhead; ++c) w[c] = d.dt_word[min(bn + uint32_t(c * kWave + lane), last)];
    };
    auto heads_of = [&](int doc, const uint32_t (&w)[kDocAhead], SkipHead (&h)[kDocAhead]) {
      const uint32_t bn = __builtin_amdgcn_readlane(offv, doc), en = __builtin_amdgcn_readlane(offv, doc + 1);
#pragma unroll
      for (int c = 0; c < kDocAhead; ++c) {
        const uint32_t pn = bn + uint32_t(c * kWave + lane);
        h[c] = skip_head(d.wskip + (pn < en ? w[c] : 0u));
      }
    };
    uint32_t rowA[kDocAhead], wA[kDocAhead], wB[kDocAhead];
    SkipHead hA[kDocAhead];
    rows_of(0, rowA);
    words_of(0, wA);
    words_of(1, wB);
    heads_of(0, wA, hA);
    for (int i = 0; i < nd; ++i) {
      const uint32_t b = __builtin_amdgcn_readlane(offv, i), e = __builtin_amdgcn_readlane(offv, i + 1);
      const uint32_t cap = __builtin_amdgcn_readlane(capv, i);
      const uint32_t len = e - b;
      uint32_t rowv[kDocAhead], wv[kDocAhead];
      SkipHead hv[kDocAhead];
#pragma unroll
      for (int c = 0; c < kDocAhead; ++c) {
        rowv[c] = rowA[c];
        hv[c] = hA[c];
        wv[c] = wA[c];
        wA[c] = wB[c];
      }
      rows_of(i + 1, rowA);
      words_of(i + 2, wB);
      heads_of(i + 1, wA, hA);
      if (len > kHeavyDoc) continue;  // a workgroup's document (heavy_doc_pass)
      const uint32_t *row = d.d_ent + cap + 1;  // entries; slot 0 is the header
      const uint32_t nnz = uint32_t(__builtin_amdgcn_readfirstlane(int(rowv[0]))) & 0xFFFFu;
      // spread the row into the topic -> count table
#pragma unroll
      for (int c = 0; c < kDocAhead; ++c) {
        const uint32_t q = uint32_t(c * kWave + lane);  // slot; entry q - 1
        if (q >= 1u && q <= nnz) cmap[rowv[c] >> 16] = uint16_t(rowv[c] & 0xFFFFu);
      }
      for (uint32_t q = uint32_t(kDocAhead * kWave - 1 + lane); q < nnz; q += kWave) {
        const uint32_t ent = row[q];
        cmap[ent >> 16] = uint16_t(ent & 0xFFFFu);
      }
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int c = 0; c < kDocAhead; ++c) {
        const uint32_t pp = b + uint32_t(c * kWave + lane);
        const bool skip = pp < e && test(pp, len, hv[c], wv[c]);
        nskip += skip ? 1ull : 0ull;
        if (by_doc) mark_chunk(d, __ballot(skip), b + uint32_t(c * kWave), lane);
        else if (skip) mark_slot(d, d.dt_wpos[pp]);
      }
      // the rest of a long document, two chunks per step
      for (uint32_t p0 = b + uint32_t(kDocAhead * kWave); p0 < e; p0 += 2u * kWave) {
        uint32_t v[2];
        SkipHead h[2];
#pragma unroll
        for (int c = 0; c < 2; ++c) v[c] = d.dt_word[min(p0 + uint32_t(c * kWave + lane), last)];
#pragma unroll
        for (int c = 0; c < 2; ++c) h[c] = skip_head(d.wskip + (p0 + uint32_t(c * kWave + lane) < e ? v[c] : 0u));
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const uint32_t pp = p0 + uint32_t(c * kWave + lane);
          const bool skip = pp < e && test(pp, len, h[c], v[c]);
          nskip += skip ? 1ull : 0ull;
          if (by_doc) mark_chunk(d, __ballot(skip), p0 + uint32_t(c * kWave), lane);
          else if (skip) mark_slot(d, d.dt_wpos[pp]);
        }
      }
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int c = 0; c < kDocAhead; ++c) {
        const uint32_t q = uint32_t(c * kWave + lane);
        if (q >= 1u && q <= nnz) cmap[rowv[c] >> 16] = 0;
      }
      for (uint32_t q = uint32_t(kDocAhead * kWave - 1 + lane); q < nnz; q += kWave) cmap[row[q] >> 16] = 0;
      __builtin_amdgcn_wave_barrier();
    }
  }
  nskip = group_sum_u64<kWave>(nskip);
  if (lane == 0 && nskip) {
    atomicAdd(&stats[ST_SKIP3], nskip);
    atomicAdd(&d.skip_hist[t & 1u], nskip);
  }
}

// Steps 2-3 for the heavy documents (longer than kHeavyDoc), one workgroup
// per document, taken from a list (d.heavy_docs) through one atomic counter
// before the workgroup's waves turn to the light documents: the D row spread
// into a topic -> count table shared by the workgroup (cmap, left clear),
// then each wave tests chunks of 64 consecutive tokens.
template <bool KeyId>
__device__ void heavy_doc_pass(const DevState &d, const Params &p, uint32_t t, uint16_t *__restrict__ cmap,
                               bool by_doc, unsigned long long &nskip) {
  __shared__ uint32_t s_next;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave, nthr = int(blockDim.x);
  for (;;) {
    __syncthreads();  // the table is clear, s_next is free
    if (tid == 0) s_next = atomicAdd(&d.counters[CNT_HEAVY_PASS], 1u);
    __syncthreads();
    const uint32_t h = s_next;
    if (h >= uint32_t(p.n_heavy)) break;
    const uint32_t dd = d.heavy_docs[h];
    const uint32_t b = d.doc_off[dd], e = d.doc_off[dd + 1], len = e - b;
    const uint32_t *row = d.d_ent + d.d_cap[dd];  // header, then the entries
    const uint32_t nnz = row[0] & 0xFFFFu;
    for (uint32_t q = uint32_t(tid); q < nnz; q += uint32_t(nthr)) {
      const uint32_t ent = row[1u + q];
      cmap[ent >> 16] = uint16_t(ent & 0xFFFFu);
    }
    __syncthreads();
    for (uint32_t p0 = b + uint32_t(wave * kWave); p0 < e; p0 += uint32_t(nthr)) {
      const uint32_t pp = p0 + uint32_t(lane);
      bool skip = false;
      if (pp < e) {
        const uint32_t v = d.dt_word[pp];
        skip = skip_test<KeyId>(d, p, t, cmap, pp, len, skip_head(d.wskip + v), v);
      }
      nskip += skip ? 1ull : 0ull;
      if (by_doc) mark_chunk(d, __ballot(skip), p0, lane);
      else if (skip) mark_slot(d, d.dt_wpos[pp]);
    }
    __syncthreads();
    for (uint32_t q = uint32_t(tid); q < nnz; q += uint32_t(nthr)) cmap[row[1u + q] >> 16] = 0;
  }
  __syncthreads();  // wave 0's table is clear again
}

// Steps 4-6 for the tokens of one region that step 3 left to draw; the W^ row of the word
// sits in LDS (Sec. 4.3, last paragraph) together with the Q' prefix over
// blocks of kGroup topics.
//
// Work split: a wave takes 64 consecutive word-ordered tokens.  Each lane
// loads its token's skip bit, key and D-row offset, and for a token left to
// draw its row header and u, staged in the wave's slice of LDS.  Those
// tokens are listed by row length and drawn in rounds by groups of 4, 8 or
// 16 lanes (draw_batch_small); rows over 512 slots by 16-lane groups in
// chunks (draw_long).  A group holds the row in registers (lane l a
// contiguous run, so lane partial sums are in ascending topic order), picks
// out C1 = D[d][K1], sums S', splits x between M, S' and Q', and records the
// selected run (S') or the remainder (Q'); one lane per token then finishes
// the draw (finish_draw).  The batch's topics, K1 for the skipped tokens,
// leave in one coalesced store.
static_assert(kGroup == 16, "the row scans use DPP rows of 16 lanes");
constexpr int kMaxRun = 8;                            // D entries per lane in registers
constexpr uint32_t kChunk = kGroup * kMaxRun;         // 128 entries per group per chunk

// One batch of 64 word-ordered tokens, staged in the wave's slice of LDS
// (entry q = lane q's token): D-row offset, row length, u, and the drawn topic.
struct BatchLds {
  uint32_t *off, *nnz;
  double *u;
  uint16_t *top;
  uint32_t *hand;  // kMaxRun slots per group: the selected lane's run
  uint8_t *list;   // the batch's lanes, sorted by row length, for the small-group draws
};

// The word of the current region: W^ row (with W^[K1] = 0) and Q' block
// prefix in LDS, and its per-word scalars.
struct WordState {
  const double *wh, *qb;
  int nb, K;
  int qhalf;  // half the padded block count of qb (0 for a single block): the binary search's first step
  uint32_t K1;
  double a1, qp, alpha;
  const double *qw;   // kQwStride per block: the partial sums before each of its kGroup topics, then its total (or null)
  const uint8_t *ql;  // per block: the offset of its last topic with a positive term (or its first)
};
constexpr int kQwStride = kGroup + 1;


// W^' of a packed D entry's topic (entry = topic << 16 | count) from the
// row in LDS: the address, topic * 8 + the row's LDS offset, is one
// v_mad_u32_u16 on the entry's high half (op_sel), read as an LDS pointer.
typedef const __attribute__((address_space(3))) double lds_f64;
__device__ __forceinline__ double wh_of(const double *__restrict__ wh, uint32_t e) {
  uint32_t a;
  asm("v_mad_u32_u16 %0, %1, 8, %2 op_sel:[1,0,0,0]"
      : "=v"(a)
      : "v"(e), "s"(uint32_t(reinterpret_cast<uintptr_t>(wh))));
  return *(lds_f64 *)(size_t)a;
}

// Load C entries per lane from `row` (lane li gets entries [li*C, li*C + C),
// topics ascending).  The row is padded to its length class with count-0
// entries of topic K, so all 16*C entries are in the row's slots.
template <int C>
__device__ __forceinline__ void load_run(const uint32_t *__restrict__ row, int li, uint32_t (&r)[C]) {
  const uint32_t q0 = uint32_t(li) * C;
#pragma unroll
  for (int i = 0; i < C; ++i) r[i] = row[q0 + i];
}

// This lane's S' terms in ascending topic order (W^[K1] = 0 in LDS).  The
// lane sums are fused multiply-adds: S' is a sum in another association than
// the sequential one anyway, so only draws within rounding distance of a
// segment boundary can depend on it.
template <int C>
__device__ __forceinline__ double run_sum(const uint32_t (&r)[C], const double *__restrict__ wh) {
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < C; ++i) s = __builtin_fma(double(r[i] & 0xFFFFu), wh_of(wh, r[i]), s);
  return s;
}

// min(c, D[d][K1]) if this lane's run holds topic K1, else c unchanged or
// larger than 0xFFFF: an entry minus (K1 << 16) is its count when its topic
// is K1 and at least 2^16 (modulo 2^32) for any other topic, since topics
// (and the padding topic K) are below 2^16.
template <int C>
__device__ __forceinline__ uint32_t run_count_of(const uint32_t (&r)[C], uint32_t K1, uint32_t c) {
  const uint32_t key = K1 << 16;
#pragma unroll
  for (int i = 0; i < C; ++i) c = min(c, r[i] - key);
  return c;
}

// Sum of a uint32 over each row of 16 lanes, in every lane of the row.
__device__ __forceinline__ uint32_t row_sum_u32(uint32_t v) {
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x111, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x112, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x114, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x118, 0xF, 0xF, true));
  return __shfl(v, kGroup - 1, kGroup);
}

// Sum of a uint32 over the wave (the total must fit in 32 bits), as a
// wave-uniform value.
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x111, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x112, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x114, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x118, 0xF, 0xF, true));
  return uint32_t(__builtin_amdgcn_readlane(int(v), 15)) + uint32_t(__builtin_amdgcn_readlane(int(v), 31)) +
         uint32_t(__builtin_amdgcn_readlane(int(v), 47)) + uint32_t(__builtin_amdgcn_readlane(int(v), 63));
}

// Lane of the row whose run holds x: the first lane with terms whose
// inclusive prefix passes x, else (rounding) the last lane with terms.
__device__ __forceinline__ int run_lane(double s, double incl, double base, double x, int grp) {
  const uint32_t hm = uint32_t(__ballot(s > 0.0 && x < base + incl) >> (grp * kGroup)) & kGroupMask;
  const uint32_t pm = uint32_t(__ballot(s > 0.0) >> (grp * kGroup)) & kGroupMask;
  return hm ? __ffs(hm) - 1 : (pm ? 31 - __clz(pm) : 0);
}

// Block b of the Q' prefix holding xq: the largest b in [0, nb) with
// qb[b] <= xq, found 16 candidates at a time.
__device__ __forceinline__ int q_block(double xq, const WordState &w, int grp, int li) {
  int lo = 0, span = w.nb;
  while (span > 1) {
    const int step = (span + kGroup - 1) / kGroup;
    const int off = li * step;
    const bool ok = off < span && w.qb[lo + off] <= xq;
    const uint32_t bm = uint32_t(__ballot(ok) >> (grp * kGroup)) & kGroupMask;
    const int best = bm ? 31 - __clz(bm) : 0;
    lo += best * step;
    span = min(step, span - best * step);
  }
  return lo;
}

// The last step of every draw: 16 candidate segments, one per lane (lane li
// holds topic k_li with width term_li >= 0, in canonical order after
// `start`); returns the topic of the first segment whose running sum passes
// x (the last positive one if rounding leaves x past them all).
__device__ __forceinline__ uint32_t pick_segment(uint32_t k, double term, double start, double x, int grp) {
  const double in2 = row_incl_scan(term);
  const uint32_t hm = uint32_t(__ballot(term > 0.0 && x < start + in2) >> (grp * kGroup)) & kGroupMask;
  const uint32_t pm = uint32_t(__ballot(term > 0.0) >> (grp * kGroup)) & kGroupMask;
  const int h = hm ? __ffs(hm) - 1 : (pm ? 31 - __clz(pm) : 0);
  return __shfl(k, h, kGroup);
}

// Draw the tokens of `mask` (rows longer than the small-group rounds take),
// four at a time, one per 16-lane group, walking each row in chunks of
// kChunk entries.  `foll` marks the later tokens of runs of one word in one
// document (same row; `starts` marks where runs begin): they share the row,
// M, S' and Q' with the run's first token (Sec. 3.3), so the group that draws
// the first one also draws them from the sums it holds, reading at most the
// one chunk that holds each x.  Every draw is the one the token would get on
// its own, bit for bit.
__device__ void draw_long(unsigned long long mask, unsigned long long foll, unsigned long long starts,
                          const BatchLds &bt, const WordState &w, const uint32_t *__restrict__ d_ent, int grp, int li,
                          unsigned long long &after_s) {
  constexpr int R = kMaxRun;
  mask &= ~foll;  // the runs' first tokens
  while (mask) {
    // the four lowest tokens of the mask, one per group (wave-uniform bit
    // arithmetic; a group with none gets src = -1)
    const unsigned long long m1 = mask & (mask - 1ull), m2 = m1 & (m1 - 1ull), m3 = m2 & (m2 - 1ull);
    const int f0 = __ffsll((long long)mask) - 1, f1 = __ffsll((long long)m1) - 1;
    const int f2 = __ffsll((long long)m2) - 1, f3 = __ffsll((long long)m3) - 1;
    mask = m3 & (m3 - 1ull);
    const int src = grp == 0 ? f0 : grp == 1 ? f1 : grp == 2 ? f2 : f3;
    uint32_t n_m = 0;  // draws of this group in the max-topic branch
    if (src >= 0) {
    const uint32_t t_off = bt.off[src];
    const uint32_t t_nnz = bt.nnz[src];
    const uint32_t *row = d_ent + t_off;  // slot 0 is the row header
    const uint32_t pad = uint32_t(w.K) << 16;
    const uint32_t nch = (t_nnz + 1u + kChunk - 1) / kChunk;
    uint32_t r[R];
    double s = 0.0, incl = 0.0, S = 0.0;
    double tot = 0.0;  // lane c of the group (c < kGroup): the total of chunk c
    uint32_t c1 = 0xFFFFFFFFu;
    for (uint32_t ch = 0; ch < nch; ++ch) {
      load_run<R>(row + ch * kChunk, li, r);
      if (ch == 0u && li == 0) r[0] = pad;
      c1 = run_count_of<R>(r, w.K1, c1);
      s = run_sum<R>(r, w.wh);
      incl = row_incl_scan(s);
      const double tch = __shfl(incl, kGroup - 1, kGroup);
      S += tch;
      tot = uint32_t(li) == ch ? tch : tot;
    }
    // max-topic branch, Eq. 7: M = W^[v][K1] * (D[d][K1] + alpha)
    const double Mm = w.a1 * (double(row_sum_u32(c1 <= 0xFFFFu ? c1 : 0u)) + w.alpha);
    // with the totals kept in the lanes: lane c's chunk base
    // M + t_0 + ... + t_(c-1), added left to right as the walk over the
    // chunks adds them, and the base after the last chunk
    const bool kept = nch > 1 && nch <= uint32_t(kGroup);
    double mine = Mm, cb_end = Mm;
    if (kept) {
      for (uint32_t c = 0; c < nch; ++c) {
        mine = uint32_t(li) == c ? cb_end : mine;
        cb_end += __shfl(tot, int(c), kGroup);
      }
    }
    // the draw of one token of the row from x = u * Z
    auto draw_x = [&](double x) -> uint32_t {
      if (x < Mm) {
        n_m++;
        return w.K1;
      }
      // locate the chunk, then 16 candidate segments
      double cbase = Mm;
      bool in_s = false;
      if (kept) {
        // only the chunk that holds x is read again
        const uint32_t hm = uint32_t(__ballot(uint32_t(li) < nch && x < mine + tot) >> (grp * kGroup)) & kGroupMask;
        cbase = cb_end;
        if (hm) {
          const int cs = __ffs(hm) - 1;
          in_s = true;
          cbase = __shfl(mine, cs, kGroup);
          load_run<R>(row + uint32_t(cs) * kChunk, li, r);
          if (cs == 0 && li == 0) r[0] = pad;
          s = run_sum<R>(r, w.wh);
          incl = row_incl_scan(s);
        }
      } else {
        for (uint32_t ch = 0; ch < nch && !in_s; ++ch) {
          if (nch > 1) {
            load_run<R>(row + ch * kChunk, li, r);
            if (ch == 0u && li == 0) r[0] = pad;
            s = run_sum<R>(r, w.wh);
            incl = row_incl_scan(s);
          }
          const double total = __shfl(incl, kGroup - 1, kGroup);
          if (x < cbase + total) in_s = true;
          else cbase += total;
        }
      }
      uint32_t k;
      double term, start;
      if (in_s) {
        // S' run of one lane, moved across the group
        const int sel = run_lane(s, incl, cbase, x, grp);
        start = cbase + __shfl(incl - s, sel, kGroup);
        // lane li < R of the group takes entry li of the selected run
        uint32_t *hand = bt.hand + grp * kMaxRun;
        if (li == sel) {
#pragma unroll
          for (int i = 0; i < R; ++i) hand[i] = r[i];
        }
        const uint32_t own = li < R ? hand[li] : 0u;
        k = own >> 16;
        term = double(own & 0xFFFFu) * w.wh[k];
      } else {
        // Q' branch: boundaries (M + S') + Qcdf
        const double qstart = cbase;
        const double xq = x - qstart;
        if (!(xq < w.qb[w.nb])) {
          k = (w.K1 == uint32_t(w.K - 1)) ? uint32_t(w.K - 2) : uint32_t(w.K - 1);  // last positive segment
          term = 0.0;
          start = 0.0;
        } else {
          const int lo = q_block(xq, w, grp, li);
          k = uint32_t(lo * kGroup + li);
          term = int(k) < w.K ? w.alpha * w.wh[k] : 0.0;
          start = qstart + w.qb[lo];
        }
      }
      const bool fallback = !in_s && term == 0.0 && start == 0.0;
      const uint32_t picked = pick_segment(k, term, start, x, grp);
      return fallback ? k : picked;
    };
    const uint32_t topic = draw_x(bt.u[src] * ((Mm + S) + w.qp));
    if (li == 0) bt.top[src] = uint16_t(topic);
    // the run's later tokens: lanes after src up to the next run start
    const unsigned long long after = ~((2ull << src) - 1ull);  // the lanes above src
    const unsigned long long nxt = starts & after;
    unsigned long long fl = foll & after & (nxt ? (nxt & (0ull - nxt)) - 1ull : ~0ull);
    while (fl) {
      const int f = __ffsll((long long)fl) - 1;
      fl &= fl - 1ull;
      const uint32_t tf = draw_x(bt.u[f] * ((Mm + S) + w.qp));
      if (li == 0) bt.top[f] = uint16_t(tf);
    }
    }
    // outside the divergent part, so the count stays wave-uniform
    after_s += wave_sum_u32(li == 0 ? n_m : 0u);
  }
}

// Entries of the sampler's W^' row in LDS: K + 1 (topic K is the padding of
// D rows) rounded up to whole blocks of kGroup topics, zeros past K.
__host__ __device__ inline int wh_entries(int K) { return (K + 1 + kGroup - 1) / kGroup * kGroup; }

// Blocks of the Q' prefix rounded up to a power of 2 (its binary search).
__host__ __device__ inline int q_blocks_padded(int nb) {
  int q = 1;
  while (q < nb) q *= 2;
  return q;
}

// ------------------------------------------------ small-group draws ----
// Rows of at most 512 slots are drawn by groups of G = 4 lanes (rows of up
// to 128 slots, 16 tokens per wave at a time), G = 8 lanes (up to 256 slots,
// 8 tokens at a time) or G = 16 lanes (up to 512 slots, 4 tokens), in chunks
// of G*kRun slots whose loads are all issued before the first is used.
// Group-wide sums and scans are DPP moves inside quads (quad_perm), half
// rows (row_half_mirror) and rows (row_mirror); the selected entry is found
// by a walk inside one lane.
constexpr int kRun = 8;
constexpr int kDppXor1 = 0xB1;         // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;         // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // lane i <- lane 7-i inside each 8 lanes
constexpr int kDppMirror = 0x140;      // lane i <- lane 15-i inside each 16 lanes

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
  return uint32_t(__builtin_amdgcn_update_dpp(0, int(v), CTRL, 0xF, 0xF, true));
}
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
  const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, 0xF, 0xF, true);
  const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, 0xF, 0xF, true);
  return __hiloint2double(hi, lo);
}

// Sum over a group of G (4, 8 or 16) aligned lanes; every lane gets the
// same bits (each step adds a pair in both orders, and IEEE addition
// commutes).
template <int G>
__device__ __forceinline__ double gsum(double v) {
  v += dpp_f64<kDppXor1>(v);
  v += dpp_f64<kDppXor2>(v);
  if (G >= 8) v += dpp_f64<kDppHalfMirror>(v);
  if (G >= 16) v += dpp_f64<kDppMirror>(v);
  return v;
}
template <int G>
__device__ __forceinline__ uint32_t gsum_u32(uint32_t v) {
  v += dpp_u32<kDppXor1>(v);
  v += dpp_u32<kDppXor2>(v);
  if (G >= 8) v += dpp_u32<kDppHalfMirror>(v);
  if (G >= 16) v += dpp_u32<kDppMirror>(v);
  return v;
}
template <int G>
__device__ __forceinline__ uint32_t gmin_u32(uint32_t v) {
  v = min(v, dpp_u32<kDppXor1>(v));
  v = min(v, dpp_u32<kDppXor2>(v));
  if (G >= 8) v = min(v, dpp_u32<kDppHalfMirror>(v));
  if (G >= 16) v = min(v, dpp_u32<kDppMirror>(v));
  return v;
}
template <int G>
__device__ __forceinline__ uint32_t gmax_u32(uint32_t v) {
  v = max(v, dpp_u32<kDppXor1>(v));
  v = max(v, dpp_u32<kDppXor2>(v));
  if (G >= 8) v = max(v, dpp_u32<kDppHalfMirror>(v));
  if (G >= 16) v = max(v, dpp_u32<kDppMirror>(v));
  return v;
}
// Inclusive prefix sum over a group of G lanes (li = lane in the group).
template <int G>
__device__ __forceinline__ double gscan(double v, int li) {
  { const double t = row_shr<1>(v); v += li >= 1 ? t : 0.0; }
  { const double t = row_shr<2>(v); v += li >= 2 ? t : 0.0; }
  if (G >= 8) { const double t = row_shr<4>(v); v += li >= 4 ? t : 0.0; }
  if (G >= 16) { const double t = row_shr<8>(v); v += li >= 8 ? t : 0.0; }
  return v;
}

// Segment of a group's CDF that holds x: the group's lanes carry terms s >= 0
// (in canonical order, lane by lane) whose inclusive scan is incl, starting at
// base.  Returns the first lane whose range passes x, or, when rounding puts x
// at or past the end, the last lane with a positive term.
template <int G>
__device__ __forceinline__ int pick_lane(double s, double incl, double base, double x, int li) {
  const uint32_t n = gsum_u32<G>(x >= base + incl ? 1u : 0u);
  if (n < uint32_t(G)) return int(n);
  return int(gmax_u32<G>(s > 0.0 ? uint32_t(li) : 0u));
}

// First of kRun packed entries whose running S' sum (fused multiply-adds from
// 0, as in run_sum) passes xs >= 0; the last entry with a positive term if
// rounding leaves xs at or past the lane's total.  Such an entry always has
// a positive term.
__device__ __forceinline__ uint32_t walk_run(const uint32_t (&r)[kRun], const double *__restrict__ wh, double xs) {
  double p = 0.0;
  uint32_t ent = r[0];
#pragma unroll
  for (int i = 0; i < kRun; ++i) {
    const bool open = p <= xs;
    p = __builtin_fma(double(r[i] & 0xFFFFu), wh_of(wh, r[i]), p);
    ent = open ? r[i] : ent;
  }
  if (!(xs < p)) {
#pragma unroll
    for (int i = 0; i < kRun; ++i)
      if ((r[i] & 0xFFFFu) != 0u && wh_of(wh, r[i]) > 0.0) ent = r[i];
  }
  return ent;
}

// The lane's index in the wave, computed where it is used: an opaque value
// keeps the compiler from hoisting the many lane-derived offsets and masks of
// the rounds out of the loops, where they would all stay live and spill.
__device__ __forceinline__ int lane_here() {
  int v;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(v));
  return v;
}

// Codes left in a token's topic slot by the small-group rounds: the draw
// fell in S' (the entry is found by a walk over the recorded run) or in Q'
// (a search of the word's Q' prefix).  Topics are below 2^15.
constexpr uint16_t kDrawS = 0xFFFF;
constexpr uint16_t kDrawQ = 0xFFFE;

// Topic of x in [0, Q') by the word's Q' prefix: the block by a binary
// search of qb (blocks of kGroup topics, +inf past the last), then a walk
// over the block's alpha * W^' terms (W^' is 0 from K up to the block end).  A rounding that leaves x at or past
// the end selects the last positive term.
__device__ __forceinline__ uint32_t q_draw(double xq, const WordState &w) {
  if (!(xq < w.qb[w.nb])) return (w.K1 == uint32_t(w.K - 1)) ? uint32_t(w.K - 2) : uint32_t(w.K - 1);
  int lo = 0;  // the largest block with qb[lo] <= xq (qb is +inf from nb + 1 up to 2 * qhalf)
  for (int step = w.qhalf; step > 0; step >>= 1) lo = w.qb[lo + step] <= xq ? lo + step : lo;
  const double xs = xq - w.qb[lo];
  if (w.qw) {
    // the walk below, by a binary search over the same partial sums (kept
    // per region): the last topic whose partial sum before it is <= xs
    const double *pw = w.qw + lo * kQwStride;
    if (!(xs < pw[kGroup])) return uint32_t(lo * kGroup + w.ql[lo]);
    int i = 0;
#pragma unroll
    for (int step = kGroup / 2; step > 0; step >>= 1) i = pw[i + step] <= xs ? i + step : i;
    return uint32_t(lo * kGroup + i);
  }
  const int k0 = lo * kGroup;
  double p = 0.0;
  int kk = k0, last = k0;
#pragma unroll
  for (int i = 0; i < kGroup; ++i) {
    const int k = k0 + i;
    const double t = w.alpha * w.wh[k];  // zeros past K (the row is padded to whole blocks)
    const bool open = p <= xs;
    p += t;
    kk = open ? k : kk;
    last = t > 0.0 ? k : last;
  }
  return uint32_t(xs < p ? kk : last);
}

// The drawn topic of a batch token, one lane per token: the topic itself,
// or the end of an S' or Q' draw recorded by the rounds.
__device__ __forceinline__ uint32_t finish_draw(int q, const BatchLds &bt, const WordState &w,
                                                const uint32_t *__restrict__ d_ent) {
  const uint32_t code = bt.top[q];
  if (code == kDrawS) {
    const uint32_t a = bt.off[q];
    uint32_t r[kRun];
    load_run<kRun>(d_ent + (a & ~uint32_t(kRun - 1)), 0, r);
    if (a & 1u) r[0] = uint32_t(w.K) << 16;  // the run starts with the row header
    return walk_run(r, w.wh, bt.u[q]) >> 16;
  }
  if (code == kDrawQ) return q_draw(bt.u[q], w);
  return code;
}

// One round of small-group draws: group g of the wave draws the token in
// list slot `slot` (if slot < n).  The row is read in chunks of G*kRun
// entries, lane l holding entries [l*kRun, l*kRun + kRun) of each chunk (the
// group's loads of a chunk share cache lines); NC is the largest chunk count
// in the round, and a group whose row has fewer chunks skips the rest.
template <int G, int NC>
__device__ void draw_small(const BatchLds &bt, int slot, int n, const WordState &w,
                           const uint32_t *__restrict__ d_ent, int li, unsigned long long &after_s) {
  constexpr uint32_t kSpan = uint32_t(G) * kRun;  // entries per chunk
  bool in_m = false;
  if (slot < n) {
    const int src = bt.list[slot];
    const uint32_t nc = (bt.nnz[src] + 1u + kSpan - 1) / kSpan;  // slots: header + entries
    const uint32_t off0 = bt.off[src];
    const uint32_t *run = d_ent + off0 + uint32_t(li) * kRun;
    const uint32_t pad = uint32_t(w.K) << 16;
    const double u = bt.u[src];
    // pass over the row: every chunk's loads are issued before the first is
    // used (one memory latency per row, not one per chunk); then per lane
    // and chunk the S' sum of kRun entries, and C1
    uint32_t r[NC][kRun];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      if (uint32_t(c) < nc) load_run<kRun>(run + c * kSpan, 0, r[c]);
    }
    if (li == 0) r[0][0] = pad;  // the row header
    double s[NC], T[NC];
    uint32_t c1 = 0xFFFFFFFFu;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      s[c] = 0.0;
      if (uint32_t(c) < nc) {
        c1 = run_count_of<kRun>(r[c], w.K1, c1);
        s[c] = run_sum<kRun>(r[c], w.wh);
      }
    }
    // group totals, cumulative over the chunks (a missing chunk adds 0)
    double S = 0.0;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      S += gsum<G>(s[c]);
      T[c] = S;
    }
    c1 = gmin_u32<G>(c1);
    // max-topic branch, Eq. 7: M = W^[v][K1] * (D[d][K1] + alpha)
    const double Mm = w.a1 * (double(c1 <= 0xFFFFu ? c1 : 0u) + w.alpha);
    const double x = u * ((Mm + S) + w.qp);
    in_m = x < Mm;
    if (!in_m) {
      if (x < Mm + S) {
        // S': the chunk (the first whose cumulative total passes x; it has a
        // positive total), the lane, then the entry
        int cs = 0;
        double base = Mm, sc = s[0];
#pragma unroll
        for (int c = 1; c < NC; ++c) {
          if (uint32_t(c) < nc && x >= Mm + T[c - 1]) {
            cs = c;
            base = Mm + T[c - 1];
            sc = s[c];
          }
        }
        const double incl = gscan<G>(sc, li);
        const int sel = pick_lane<G>(sc, incl, base, x, li);
        if (li == sel) {
          // the selected lane's run and x inside it, for the walk after the rounds
          bt.off[src] = (off0 + uint32_t(cs) * kSpan + uint32_t(li) * kRun) | (cs == 0 && li == 0 ? 1u : 0u);
          bt.u[src] = fmax(x - (base + (incl - sc)), 0.0);
          bt.top[src] = kDrawS;
        }
      } else if (li == 0) {
        // Q': x past M + S', searched after the rounds
        bt.u[src] = x - (Mm + S);
        bt.top[src] = kDrawQ;
      }
    }
    if (in_m && li == 0) bt.top[src] = uint16_t(w.K1);
  }
  // outside the divergent part, so the count stays wave-uniform
  after_s += uint32_t(__popcll(__ballot(in_m && li == 0)));
}

// Row-length buckets of a batch (slots, header included): upper bounds.
// Buckets 0-3 are rows padded to 32-slot multiples, 4-5 to 64, 6-7 to 128.
__device__ constexpr uint32_t kBucketEnd[8] = {32, 64, 96, 128, 192, 256, 384, 512};

// The small-group rounds over list places [from, to) (rows in ascending
// bucket order), G lanes per token and 64/G tokens a round.  A round reads
// as many chunks of G*kRun slots as its last (longest) row needs.
template <int G, int MaxNC>
__device__ void draw_rounds(int from, int to, const int (&ends)[8], const BatchLds &bt, const WordState &w,
                            const uint32_t *__restrict__ d_ent, unsigned long long &after_s) {
  constexpr uint32_t kSpan = uint32_t(G) * kRun;
  for (int base = from; base < to; base += kWave / G) {
    const int ln = lane_here(), g = ln / G, li = ln % G;
    const int last = min(base + kWave / G, to) - 1;
    uint32_t upper = kBucketEnd[7];
#pragma unroll
    for (int k = 6; k >= 0; --k) upper = last < ends[k] ? kBucketEnd[k] : upper;
    const uint32_t nc = (upper + kSpan - 1) / kSpan;
    const int slot = base + g;
    if (nc <= 1) {
      draw_small<G, 1>(bt, slot, to, w, d_ent, li, after_s);
    } else if (nc == 2) {
      draw_small<G, 2>(bt, slot, to, w, d_ent, li, after_s);
    } else if (nc == 3) {
      draw_small<G, 3>(bt, slot, to, w, d_ent, li, after_s);
    } else if (MaxNC <= 4 || nc == 4) {
      draw_small<G, 4>(bt, slot, to, w, d_ent, li, after_s);
    } else {
      if constexpr (MaxNC > 4) {
        if (nc <= 6) draw_small<G, 6>(bt, slot, to, w, d_ent, li, after_s);
        else draw_small<G, MaxNC>(bt, slot, to, w, d_ent, li, after_s);
      }
    }
  }
}

// The small-group draws of one batch.  The lanes left to draw are listed in
// ascending bucket order; rows of up to 128 slots are drawn by groups of 4
// lanes (16 a round), up to 256 by 8 lanes, up to 512 by 16 lanes.  When the
// 4-lane rounds would end with a partial round of at most 8 rows, all of
// 97-128 slots (two whole 64-slot chunks), those rows join the 8-lane
// rounds instead: they fill free places there, or make a round that reads
// half as many entries per lane as the partial 4-lane round would.
// Wide (the 1024-thread workgroups, whose waves have registers to spare):
// rows of up to 512 slots by 8 lanes as well, 8 tokens a round, so that a
// round's per-token work (sums, scans, the split of x) serves twice the
// tokens.
template <bool Wide>
__device__ void draw_batch_small(bool und, uint32_t nnz, const BatchLds &bt, const WordState &w,
                                 const uint32_t *__restrict__ d_ent, int lane, unsigned long long &after_s) {
  int n = 0, ends[8];
  const uint32_t slots = nnz + 1u;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const uint32_t lo = k ? kBucketEnd[k - 1] : 0u;
    const unsigned long long m = __ballot(und && slots > lo && slots <= kBucketEnd[k]);
    if ((m >> lane) & 1ull)
      bt.list[n + int(__builtin_amdgcn_mbcnt_hi(uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u)))] =
          uint8_t(lane);
    n += __popcll(m);
    ends[k] = n;
  }
  const int left = ends[3] % 16;
  const int a = left > 0 && left <= 8 && ends[3] - ends[2] >= left ? ends[3] - left : ends[3];
  draw_rounds<4, 4>(0, a, ends, bt, w, d_ent, after_s);
  if (Wide) {
    draw_rounds<8, 8>(a, ends[7], ends, bt, w, d_ent, after_s);
  } else {
    draw_rounds<8, 4>(a, ends[5], ends, bt, w, d_ent, after_s);
    draw_rounds<16, 4>(ends[5], ends[7], ends, bt, w, d_ent, after_s);
  }
}

// The sampler for workgroups of NB threads (NB / 64 waves); every wave works
// on its own batches, so NB only changes how many waves share a region's W^
// row in LDS (larger workgroups for large K, where LDS bounds the residency).
// Light: the workgroup is one wave and takes the light regions (the suffix
// [p.light_begin, n_regions) of the region table: words with at most
// kLightTokens tokens, one batch each) from their own counter; otherwise the
// regions before p.light_begin.
template <int NB, bool Light>
__device__ __forceinline__ void sampler_body(DevState d, Params p, uint32_t t, unsigned long long *__restrict__ stats) {
  extern __shared__ double lds[];
  const int K = p.K;
  const int nb = (K + kGroup - 1) / kGroup;
  const int nbp = q_blocks_padded(nb);
  const bool by_doc = doc_marks(d, p, t);  // which bitmap carries this iteration's skip decisions
  // dynamic LDS only (sampler_lds_bytes)
  double *wh = lds;                  // [wh_entries(K)]: W^' of the region's word, zeros past K
  double *qb = lds + wh_entries(K);  // [nbp + 1]: qb[b] = sum of alpha*W^' over topics < b*kGroup; +inf past nb
  double *s_u = qb + nbp + 1;        // [NB]: the batch slices of the waves
  uint32_t *s_off = reinterpret_cast<uint32_t *>(s_u + NB);  // [NB]
  uint32_t *s_nnz = s_off + NB;                              // [NB]
  uint32_t *s_hand = s_nnz + NB;                             // [NB / kGroup * kMaxRun]
  uint32_t *s_reg = s_hand + NB / kGroup * kMaxRun;          // [4]: the region (word, begin, end) and a valid flag
  uint16_t *s_top = reinterpret_cast<uint16_t *>(s_reg + 4); // [NB]
  uint8_t *s_list = reinterpret_cast<uint8_t *>(s_top + NB); // [NB]
  // with p.q_table: [nb * kQwStride] partial sums of the Q' blocks, then [nb] last-positive offsets
  // (the 21 * NB + 16 bytes after s_u keep them 8-byte aligned)
  static_assert((21 * NB + 16) % 8 == 0, "the Q' partial sums must be 8-byte aligned");
  double *s_qw = p.q_table ? reinterpret_cast<double *>(s_list + NB) : nullptr;
  uint8_t *s_ql = p.q_table ? reinterpret_cast<uint8_t *>(s_qw + nb * kQwStride) : nullptr;

  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  if (blockIdx.x == 0 && tid == 0) stats[ST_MARKS] = by_doc ? 2ull : 1ull;
  const BatchLds bt{s_off + wave * kWave, s_nnz + wave * kWave, s_u + wave * kWave, s_top + wave * kWave,
                    s_hand + wave * (kWave / kGroup) * kMaxRun, s_list + wave * kWave};
  const int qhalf = nbp / 2;
  for (int q = nb + 1 + tid; q < nbp; q += NB) qb[q] = __builtin_inf();
  for (int k = K + 1 + tid; k < wh_entries(K); k += NB) wh[k] = 0.0;
  // region, word and count variables are uniform over the block (scalar registers)
  uint32_t cur = 0xFFFFFFFFu, K1 = 0;
  double a1 = 0.0, qp = 0.0;
  // the sparse word whose row wh holds (null if a dense row or none): the
  // next sparse word only restores that word's topics and K1 to beta/den[k]
  const uint32_t *held = nullptr;
  uint32_t held_nnz = 0, held_k1 = 0;
  unsigned long long n_sampled = 0, n_after_s = 0, nnz_sum = 0;
  unsigned long long n_reg = 0, n_dreg = 0, row_bytes = 0;

  for (;;) {
    if (tid == 0) {
      const int64_t r = Light ? p.light_begin + int64_t(atomicAdd(&d.counters[CNT_LIGHT], 1u))
                              : int64_t(atomicAdd(&d.counters[CNT_SAMPLER], 1u));
      s_reg[3] = r < (Light ? p.n_regions : p.light_begin) ? 1u : 0u;
      if (s_reg[3]) {
        s_reg[0] = d.region[3 * size_t(r)];
        s_reg[1] = d.region[3 * size_t(r) + 1];
        s_reg[2] = d.region[3 * size_t(r) + 2];
      }
    }
    __syncthreads();
    if (!s_reg[3]) break;
    const uint32_t v = __builtin_amdgcn_readfirstlane(s_reg[0]);
    const uint32_t b = __builtin_amdgcn_readfirstlane(s_reg[1]);
    const uint32_t e = __builtin_amdgcn_readfirstlane(s_reg[2]);
    n_reg++;
    if (int32_t(v) < p.n_dense) n_dreg++;
    if (b == d.word_off[v])
      row_bytes += int32_t(v) < p.n_dense ? 4ull * uint64_t(K) : 4ull * d.ws_nnz[int(v) - p.n_dense];
    if (v != cur) {
      cur = v;
      const WordRec rec = d.wrec[v];
      K1 = rec.k1;
      a1 = rec.a1;
      qp = rec.qp;
      if (int32_t(v) < p.n_dense) {
        const int32_t *wrow = d.w_dense + size_t(v) * size_t(K);
        for (int k = tid; k < K; k += NB) wh[k] = what(uint32_t(wrow[k]), p.beta, d.den[k]);
        held = nullptr;
      } else {
        const int s = int(v) - p.n_dense;
        const uint32_t *ents = d.ws_ent + d.ws_cap[s];
        const uint32_t nnz = d.ws_nnz[s];
        if (held) {
          for (uint32_t q = tid; q < held_nnz; q += NB) {
            const uint32_t k = held[q] >> 16;
            wh[k] = d.bden[k];
          }
          if (tid == 0 && held_k1 < uint32_t(K)) wh[held_k1] = d.bden[held_k1];  // K1 = K in two-branch mode
        } else {
          for (int k = tid; k < K; k += NB) wh[k] = d.bden[k];
        }
        __syncthreads();
        for (uint32_t q = tid; q < nnz; q += NB) {
          const uint32_t ent = ents[q];
          wh[ent >> 16] = what(ent & 0xFFFFu, p.beta, d.den[ent >> 16]);
        }
        held = ents;
        held_nnz = nnz;
        held_k1 = K1;
      }
      __syncthreads();
      // the max topic is its own branch: W^' has a 0 there (Eq. 5)
      if (tid == 0) {
        wh[K1] = 0.0;
        wh[K] = 0.0;  // topic of the padding entries of D rows
      }
      __syncthreads();
      // the Q' prefix over blocks of kGroup topics: thread i sums blocks i,
      // i + NB, ..., then per round a scan per wave (DPP) leaves the block's
      // prefix inside its wave in qb and the wave's total in s_u; after the
      // barrier each block adds the totals before its wave, in round and wave
      // order.  Without the partial-sum table a block is summed from topic
      // i % 16 on, wrapping, so that the 16 lanes of a row read 16 different
      // LDS bank pairs (wh past K holds zeros).
      double *s_tot = s_u;  // [rounds * waves <= NB]; s_u is next written by the token batches
      uint32_t rot;         // i % 16, opaque to the compiler: otherwise it keeps the 16 rotated addresses live
      asm volatile("v_mov_b32 %0, %1" : "=v"(rot) : "v"(uint32_t(lane & (kGroup - 1))));
      for (int r = 0; r * NB < nb; ++r) {
        const int blk = r * NB + tid;
        double s = 0.0;
        if (blk < nb) {
          if (s_qw) {
            // every topic of the block (zeros past K), as q_draw's walk adds them
            double *pw = s_qw + blk * kQwStride;
            int last = 0;
            for (int i = 0; i < kGroup; ++i) {
              pw[i] = s;
              const double t = p.alpha * wh[blk * kGroup + i];
              s += t;
              last = t > 0.0 ? i : last;
            }
            pw[kGroup] = s;
            s_ql[blk] = uint8_t(last);
          } else {
            const double *wb = wh + blk * kGroup;
#pragma unroll
            for (uint32_t i = 0; i < uint32_t(kGroup); ++i) s += p.alpha * wb[(i + rot) & uint32_t(kGroup - 1)];
          }
        }
        const double incl = wave_incl_scan(s);
        if (blk < nb) qb[blk + 1] = incl;
        if (lane == kWave - 1) s_tot[r * (NB / kWave) + wave] = incl;
      }
      __syncthreads();
      {
        double acc = 0.0;
        for (int r = 0; r * NB < nb; ++r) {
          double own = 0.0;
          for (int w = 0; w < NB / kWave; ++w) {
            if (w == wave) own = acc;
            acc += s_tot[r * (NB / kWave) + w];
          }
          const int blk = r * NB + tid;
          if (blk < nb) qb[blk + 1] = own + qb[blk + 1];
        }
        if (tid == 0) qb[0] = 0.0;
      }
      __syncthreads();
    }

    const WordState w{wh, qb, nb, K, qhalf, K1, a1, qp, p.alpha, s_qw, s_ql};
    // tokens per batch: 64, or fewer when the region has too few tokens to
    // give every wave a whole batch, so that a small region's batches (each
    // a chain of dependent loads and rounds) run side by side on several
    // waves instead of one after another on one
    const uint32_t bsz = min(uint32_t(kWave), max(16u, ((e - b + uint32_t(NB / kWave) - 1u) / uint32_t(NB / kWave) + 15u) & ~15u));
    for (uint32_t base = b + uint32_t(wave) * bsz; base < e; base += uint32_t(NB / kWave) * bsz) {
      const int ln = lane_here();  // the lane, recomputed per batch
      const uint32_t j = base + uint32_t(ln);
      const uint32_t be = min(e, base + bsz);  // the batch's end
      // the slot, key and row offset are loaded together (one latency); the
      // row header only for the tokens left to draw
      uint32_t sk = 0, key = 0, off = 0;
      if (j < be) {
        const uint2 kr = d.wt_kr[j];
        key = kr.x;
        off = kr.y;  // the row's first slot (its header)
        // the skip bit at the word-order slot, or at the key (the token's
        // document position) in the document-ordered bitmap
        sk = by_doc ? d.skip_doc[key >> 5] >> (key & 31u) : d.skip_bits[j >> 5] >> (j & 31u);
      }
      const bool und = j < be && !(sk & 1u);
      uint32_t nnz = 0;
      if (und) {
        nnz = d.d_ent[off] & 0xFFFFu;
        bt.off[ln] = off;
        bt.nnz[ln] = nnz;
        bt.u[ln] = uniform_draw(p.seed, t, key);
      }
      // long rows: runs of tokens of one document (same row offset), whose
      // later tokens draw from the sums of the run's first one
      const unsigned long long lmask = __ballot(und && nnz + 1u > 512u);
      unsigned long long starts = 0ull;
      bool fol = false;
      if (lmask) {
        const uint32_t prev_off = uint32_t(__shfl(int(off), ln - 1));
        starts = __ballot(ln == 0 || off != prev_off);
        const unsigned long long below = ln ? ~0ull >> (64 - ln) : 0ull;
        const int rs = 63 - __clzll((long long)(starts & (below | (1ull << ln))));  // this lane's run start
        fol = ((lmask >> ln) & 1ull) && (lmask & below & (~0ull << rs)) != 0ull;
      }
      n_sampled += uint32_t(__popcll(__ballot(und)));
      nnz_sum += wave_sum_u32(fol ? min(nnz, uint32_t(kChunk)) : nnz);  // a follower reads one chunk of its row
      // rows of up to 128 slots (header and entries): 4 lanes per token; up
      // to 256: 8 lanes; up to 512: 16 lanes; longer rows: 16 lanes, one
      // chunk of kChunk slots at a time
      draw_batch_small<(NB >= 1024)>(und, nnz, bt, w, d.d_ent, ln, n_after_s);
      if (lmask) draw_long(lmask, __ballot(fol), starts, bt, w, d.d_ent, ln / kGroup, ln % kGroup, n_after_s);
      // the S' walks and Q' searches, one lane per token; the batch's topics
      // (K1 for the tokens the step-3 test decided) leave in one coalesced store
      uint32_t topic = K1;
      if (und) topic = finish_draw(ln, bt, w, d.d_ent);
      if (j < be) d.z_w[j] = uint16_t(topic);
    }
    __syncthreads();
  }
  if (lane == 0) {
    if (n_sampled) atomicAdd(&stats[ST_SAMPLED], n_sampled);
    if (n_after_s) atomicAdd(&stats[ST_SKIP_AFTER_S], n_after_s);
    if (nnz_sum) atomicAdd(&stats[ST_NNZ], nnz_sum);
  }
  if (tid == 0) {
    if (n_reg) atomicAdd(&stats[ST_REGIONS], n_reg);
    if (n_dreg) atomicAdd(&stats[ST_DENSE_REGIONS], n_dreg);
    if (row_bytes) atomicAdd(&stats[ST_ROW_BYTES], row_bytes);
  }
}


__global__ __launch_bounds__(256, 7) void k_sampler(DevState d, Params p, uint32_t t,
                                                 unsigned long long *__restrict__ stats) {
  sampler_body<256, false>(d, p, t, stats);
}
__global__ __launch_bounds__(512, 4) void k_sampler_512(DevState d, Params p, uint32_t t,
                                                     unsigned long long *__restrict__ stats) {
  sampler_body<512, false>(d, p, t, stats);
}
__global__ __launch_bounds__(1024, 4) void k_sampler_1024(DevState d, Params p, uint32_t t,
                                                       unsigned long long *__restrict__ stats) {
  sampler_body<1024, false>(d, p, t, stats);
}
// The light regions, one wave each (Sec. 5.1: light units to wavefronts): a
// word of at most kLightTokens tokens stages its W^' row and Q' prefix with
// one wave and wave-local barriers instead of tying up a whole workgroup.
__global__ __launch_bounds__(64) void k_sampler_light(DevState d, Params p, uint32_t t,
                                                      unsigned long long *__restrict__ stats) {
  sampler_body<64, true>(d, p, t, stats);
}

// ---------------------------------------------------------- large K ----
// When the fp64 W^' row does not fit in LDS (K above about 17,000 topics,
// up to 32,768), the topics are split in two tiles, [0, KT) and [KT, K]
// (topic K is the padding of D rows), and a region is walked three times:
//   pass 0, tile 0: per token the S' terms of topics below KT and C1;
//   pass 1, tile 1: the S' terms of the other topics, then the draw (Eq. 5);
//                   draws in M, in the tile-1 part of S' or in a tile-1 Q'
//                   block finish here, the others are recorded;
//   pass 2, tile 0: the recorded draws finish, over the list of their
//                   tokens that pass 1 keeps.
// A row is in ascending topic order, so pass 0 reads its chunks only up to
// the first one that reaches topic KT (the split chunk, kept per token),
// pass 1 only from there on, and pass 2's S' walk ends there: every chunk
// left out holds only terms of the other tile, which add exact zeros.
// The canonical order [K1 | S' ascending | Q' ascending] is unchanged: the
// tile-0 part of S' precedes the tile-1 part.  A 16-lane group draws one
// token at a time and reads its D row in chunks of kChunk slots; entries of
// the other tile read a zero.  Per-token results between passes live in a
// per-workgroup slice of global scratch.
struct TileState {
  const double *wt;  // the tile: W^' of topics [base, base + KT), zeros past the tile's end
  uint32_t base, kt;
  uint32_t rel;      // -base * 8 (mod 2^32)
};

// W^' of a packed D entry's topic if it lies in the tile, else 0 (wt[kt] is
// 0).  The tile starts at LDS address 0 (the kernel's LDS is all dynamic,
// which launch_sampler checks), so the address (topic - base) * 8 is one
// v_mad_u32_u16 on the entry's high half; topics below the tile wrap to
// addresses near 2^32, and one unsigned min sends every topic outside the
// tile to wt[kt].
__device__ __forceinline__ double wt_of(const TileState &ts, uint32_t e) {
  uint32_t a;
  asm("v_mad_u32_u16 %0, %1, 8, %2 op_sel:[1,0,0,0]" : "=v"(a) : "v"(e), "s"(ts.rel));
  return *(lds_f64 *)(size_t)min(a, ts.kt * 8u);
}

// This lane's run of chunk ch of a row of `slots` padded slots; runs past
// the row read the padding entry, and the header (slot 0) is padding too.
__device__ __forceinline__ void load_run_masked(const uint32_t *__restrict__ row, uint32_t ch, uint32_t slots, int li,
                                                uint32_t pad, uint32_t (&r)[kMaxRun]) {
  const uint32_t q0 = ch * kChunk + uint32_t(li) * kMaxRun;
  if (q0 < slots) {
#pragma unroll
    for (int i = 0; i < kMaxRun; ++i) r[i] = row[q0 + i];
  } else {
#pragma unroll
    for (int i = 0; i < kMaxRun; ++i) r[i] = pad;
  }
  if (q0 == 0u) r[0] = pad;
}

__device__ __forceinline__ double run_sum_tile(const uint32_t (&r)[kMaxRun], const TileState &ts) {
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < kMaxRun; ++i) s = __builtin_fma(double(r[i] & 0xFFFFu), wt_of(ts, r[i]), s);
  return s;
}

// The last step of an S' draw in a tile: in the chunk that holds x (this
// lane's run r, lane sum s, inclusive scan incl, the chunk's terms starting
// at base), the lane whose run holds x and then the entry in it.
__device__ uint32_t walk_finish(const uint32_t (&r)[kMaxRun], double s, double incl, const TileState &ts,
                                double base, double x, int grp, int li, uint32_t *__restrict__ hand) {
  const int sel = run_lane(s, incl, base, x, grp);
  const double start = base + __shfl(incl - s, sel, kGroup);
  if (li == sel) {
#pragma unroll
    for (int i = 0; i < kMaxRun; ++i) hand[i] = r[i];
  }
  __builtin_amdgcn_wave_barrier();
  const uint32_t mine = li < kMaxRun ? hand[li] : 0u;
  const double term = li < kMaxRun ? double(mine & 0xFFFFu) * wt_of(ts, mine) : 0.0;
  return pick_segment(mine >> 16, term, start, x, grp);
}

// tile_walk over two chunks already in registers (runs r, lane sums t).
__device__ uint32_t walk_pair(const uint32_t (&r)[2][kMaxRun], const double (&t)[2], const TileState &ts, double base,
                              double x, int grp, int li, uint32_t *__restrict__ hand) {
  double at = base;
  int pick = -1, last = -1;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const double total = __shfl(row_incl_scan(t[c]), kGroup - 1, kGroup);
    if (pick < 0) {
      if (total > 0.0) {
        last = c;
        at = base;
      }
      if (x < base + total) pick = c;
      else base += total;
    }
  }
  if (pick < 0) {
    pick = last;  // rounding: x at or past the end of the tile's terms
    base = at;
  }
  if (pick < 0) return uint32_t(-1);
  const uint32_t(&rp)[kMaxRun] = pick == 0 ? r[0] : r[1];
  const double sp = pick == 0 ? t[0] : t[1];
  return walk_finish(rp, sp, row_incl_scan(sp), ts, base, x, grp, li, hand);
}

// The S' draw inside one tile: the entry whose segment holds x, the tile's
// terms starting at `base`; chunks [ch0, nch) are walked again in order (the
// others hold no term of the tile).  When
// rounding leaves x past the tile's terms, the last positive term is taken.
__device__ uint32_t tile_walk(const uint32_t *__restrict__ row, uint32_t slots, const TileState &ts, double base,
                              double x, uint32_t pad, int grp, int li, uint32_t *__restrict__ hand, uint32_t ch0,
                              uint32_t nch) {
  uint32_t r[kMaxRun];
  int last_pos = -1;
  double last_base = base;
  uint32_t pick = nch;
  double s = 0.0, incl = 0.0;
  uint32_t rn[kMaxRun];
  load_run_masked(row, ch0, slots, li, pad, rn);
  for (uint32_t ch = ch0; ch < nch; ++ch) {
#pragma unroll
    for (int i = 0; i < kMaxRun; ++i) r[i] = rn[i];
    if (ch + 1 < nch) load_run_masked(row, ch + 1, slots, li, pad, rn);  // the next chunk's loads, in flight meanwhile
    s = run_sum_tile(r, ts);
    incl = row_incl_scan(s);
    const double total = __shfl(incl, kGroup - 1, kGroup);
    if (total > 0.0) {
      last_pos = int(ch);
      last_base = base;
    }
    if (x < base + total) {
      pick = ch;
      break;
    }
    base += total;
  }
  if (pick == nch) {
    // rounding: x at or past the end of the tile's terms
    if (last_pos < 0) return uint32_t(-1);
    pick = uint32_t(last_pos);
    base = last_base;
    load_run_masked(row, pick, slots, li, pad, r);
    s = run_sum_tile(r, ts);
    incl = row_incl_scan(s);
  }
  return walk_finish(r, s, incl, ts, base, x, grp, li, hand);
}


// Fills the tile [base, base + len) of the region's word (zeros elsewhere,
// at K1 and at the padding topic K).  Each thread issues the loads of
// kFillBatch topics (or row entries) before it uses the first, so that a
// fill waits on a few memory latencies rather than one per topic.
constexpr int kFillBatch = 8;
__device__ void fill_tile(const DevState &d, const Params &p, uint32_t v, uint32_t K1, uint32_t base, uint32_t len,
                          uint32_t kt, double *__restrict__ wt, int tid, int nthreads) {
  const uint32_t K = uint32_t(p.K), n = kt + uint32_t(kGroup), nt = uint32_t(nthreads);
  // loads at clamped (always valid) topics; the topics outside the tile get 0
  if (int32_t(v) < p.n_dense) {
    const int32_t *wrow = d.w_dense + size_t(v) * size_t(K);
    uint32_t q0 = uint32_t(tid);
    for (; q0 + (kFillBatch - 1) * nt < n; q0 += kFillBatch * nt) {
      uint32_t cnt[kFillBatch];
      double dn[kFillBatch];
#pragma unroll
      for (int u = 0; u < kFillBatch; ++u) {
        const uint32_t k = min(base + q0 + uint32_t(u) * nt, K - 1u);
        cnt[u] = uint32_t(wrow[k]);
        dn[u] = d.den[k];
      }
#pragma unroll
      for (int u = 0; u < kFillBatch; ++u) {
        const uint32_t q = q0 + uint32_t(u) * nt, k = base + q;
        wt[q] = q < len && k < K && k != K1 ? what(cnt[u], p.beta, dn[u]) : 0.0;
      }
    }
    for (; q0 < n; q0 += nt) {
      const uint32_t k = base + q0;
      wt[q0] = q0 < len && k < K && k != K1 ? what(uint32_t(wrow[k]), p.beta, d.den[k]) : 0.0;
    }
  } else {
    const int s = int(v) - p.n_dense;
    const uint32_t *ents = d.ws_ent + d.ws_cap[s];
    const uint32_t nnz = d.ws_nnz[s];
    uint32_t q0 = uint32_t(tid);
    for (; q0 + (kFillBatch - 1) * nt < n; q0 += kFillBatch * nt) {
      double bd[kFillBatch];
#pragma unroll
      for (int u = 0; u < kFillBatch; ++u) bd[u] = d.bden[min(base + q0 + uint32_t(u) * nt, K - 1u)];
#pragma unroll
      for (int u = 0; u < kFillBatch; ++u) {
        const uint32_t q = q0 + uint32_t(u) * nt, k = base + q;
        wt[q] = q < len && k < K && k != K1 ? bd[u] : 0.0;
      }
    }
    for (; q0 < n; q0 += nt) {
      const uint32_t k = base + q0;
      wt[q0] = q0 < len && k < K && k != K1 ? d.bden[k] : 0.0;
    }
    __syncthreads();
    for (uint32_t q0 = uint32_t(tid); q0 < nnz; q0 += kFillBatch * nt) {
      uint32_t ent[kFillBatch];
#pragma unroll
      for (int u = 0; u < kFillBatch; ++u) ent[u] = ents[min(q0 + uint32_t(u) * nt, nnz - 1u)];
      double dn[kFillBatch];
#pragma unroll
      for (int u = 0; u < kFillBatch; ++u) dn[u] = d.den[min(ent[u] >> 16, K - 1u)];
#pragma unroll
      for (int u = 0; u < kFillBatch; ++u) {
        const uint32_t k = ent[u] >> 16;
        if (q0 + uint32_t(u) * nt < nnz && k >= base && k < base + len && k < K && k != K1)
          wt[k - base] = what(ent[u] & 0xFFFFu, p.beta, dn[u]);
      }
    }
  }
  __syncthreads();
}

// A token's records for one pass of the tiled sampler.
struct TiledTok {
  uint32_t sk, rec, cn;
  uint2 kr;
};

constexpr int kTiledBlock = kTiledThreads;  // threads per workgroup of the tiled sampler (16 waves)
constexpr int kTiledAhead = 2;              // chunks whose loads a group issues together
static_assert(kTiledAhead == 2, "pass 1's walk in registers picks one of two chunks");

__global__ __launch_bounds__(kTiledBlock) void k_sampler_tiled(DevState d, Params p, uint32_t t,
                                                               unsigned long long *__restrict__ stats) {
  extern __shared__ double lds[];
  const int K = p.K;
  const uint32_t kt = uint32_t(p.tile_topics);  // topics per tile, a multiple of kGroup
  const int nb = (K + kGroup - 1) / kGroup;
  double *wt = lds;                                  // [kt + kGroup]
  double *qb = lds + kt + kGroup;                    // [nb + 1]: prefix of alpha*W^' over blocks of kGroup topics
  uint32_t *s_hand = reinterpret_cast<uint32_t *>(qb + nb + 1);  // [kTiledBlock / kGroup * kMaxRun]
  uint32_t *s_reg = s_hand + kTiledBlock / kGroup * kMaxRun;     // [6]: region, flag, list length
  double *s_u = reinterpret_cast<double *>(s_reg + 6);            // [kTiledBlock]: u of the next 16 steps per wave
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = tid / kWave, grp = lane / kGroup, li = lane % kGroup;
  if (blockIdx.x == 0 && tid == 0) stats[ST_MARKS] = 1ull;  // the word-ordered bitmap only
  uint32_t *hand = s_hand + (tid / kGroup) * kMaxRun;
  const uint32_t pad = uint32_t(K) << 16;
  // per-workgroup scratch slices, indexed by the token's place in its region
  double *sc_s = d.ts_s + size_t(blockIdx.x) * size_t(p.max_region);
  uint32_t *sc_c1 = d.ts_c1 + size_t(blockIdx.x) * size_t(p.max_region);
  uint32_t *sc_code = d.ts_code + size_t(blockIdx.x) * size_t(p.max_region);
  TiledRec *sc_list = d.ts_list + size_t(blockIdx.x) * size_t(p.max_region);
  unsigned long long n_sampled = 0, n_after_s = 0, nnz_sum = 0, n_reg = 0, n_dreg = 0, row_bytes = 0;
  const int waves = kTiledBlock / kWave;
  for (;;) {
    if (tid == 0) {
      const uint32_t r = atomicAdd(&d.counters[CNT_SAMPLER], 1u);
      s_reg[3] = int64_t(r) < p.n_regions ? 1u : 0u;
      s_reg[4] = 0u;
      if (s_reg[3]) {
        s_reg[0] = d.region[3 * size_t(r)];
        s_reg[1] = d.region[3 * size_t(r) + 1];
        s_reg[2] = d.region[3 * size_t(r) + 2];
      }
    }
    __syncthreads();
    if (!s_reg[3]) break;
    const uint32_t v = __builtin_amdgcn_readfirstlane(s_reg[0]);
    const uint32_t b = __builtin_amdgcn_readfirstlane(s_reg[1]);
    const uint32_t e = __builtin_amdgcn_readfirstlane(s_reg[2]);
    __syncthreads();  // s_reg is rewritten by the next region's fetch
    n_reg++;
    if (int32_t(v) < p.n_dense) n_dreg++;
    if (b == d.word_off[v])
      row_bytes += int32_t(v) < p.n_dense ? 4ull * uint64_t(K) : 4ull * d.ws_nnz[int(v) - p.n_dense];
    const WordRec rec = d.wrec[v];
    const uint32_t K1 = __builtin_amdgcn_readfirstlane(rec.k1);
    // C1 = D[d][K1] is sought only in the pass whose tile holds topic K1 (that
    // pass reads every chunk with topics of its tile); the other reads 0
    const bool k1_lo = K1 < kt;
    for (int pass = 0; pass < 3; ++pass) {
      const uint32_t tbase = pass == 1 ? kt : 0u;
      const uint32_t tlen = pass == 1 ? uint32_t(K) + 1u - kt : kt;
      fill_tile(d, p, v, K1, tbase, tlen, kt, wt, tid, kTiledBlock);
      const TileState ts{wt, tbase, kt, 0u - tbase * 8u};
      if (pass < 2) {
        // this tile's blocks of the Q' prefix, continuing the previous tile's.
        // Thread i sums blocks i and i + kTiledBlock of the tile (a tile has at
        // most 2 * kTiledBlock blocks), the 16 topics of a block from topic
        // i % 16 on, wrapping, so that the 16 lanes of a row read 16 different
        // LDS bank pairs; the prefix is then a scan per wave, in registers,
        // plus the totals of the waves before, added in wave order
        const int b0 = int(tbase) / kGroup, b1 = min(nb, int(tbase + tlen + kGroup - 1) / kGroup);
        const int nblk = b1 - b0;
        double *s_tot = s_u;  // [2 * waves]; s_u is next written in pass 1's token loop
        // the rotation's start, opaque to the compiler: otherwise it keeps the
        // 16 rotated addresses live (spilled) across the region loop
        uint32_t rot;
        asm volatile("v_mov_b32 %0, %1" : "=v"(rot) : "v"(uint32_t(li)));
        auto block_scan = [&](int blk) {
          double sum = 0.0;
          if (blk < nblk) {
            const double *wb = wt + blk * kGroup;
#pragma unroll
            for (uint32_t i = 0; i < uint32_t(kGroup); ++i)
              sum = __builtin_fma(p.alpha, wb[(i + rot) & uint32_t(kGroup - 1)], sum);
          }
          return wave_incl_scan(sum);
        };
        const double incl0 = block_scan(tid);
        if (lane == kWave - 1) s_tot[wave] = incl0;
        double incl1 = 0.0;
        if (nblk > kTiledBlock) {
          incl1 = block_scan(kTiledBlock + tid);
          if (lane == kWave - 1) s_tot[waves + wave] = incl1;
        }
        __syncthreads();
        double acc = pass == 0 ? 0.0 : qb[b0], own = 0.0;
        for (int w = 0; w < waves; ++w) {
          if (w == wave) own = acc;
          acc += s_tot[w];
        }
        if (tid < nblk) qb[b0 + tid + 1] = own + incl0;
        if (nblk > kTiledBlock) {
          for (int w = 0; w < waves; ++w) {
            if (w == wave) own = acc;
            acc += s_tot[waves + w];
          }
          if (kTiledBlock + tid < nblk) qb[b0 + kTiledBlock + tid + 1] = own + incl1;
        }
        if (pass == 0 && tid == 0) qb[0] = 0.0;
        __syncthreads();
      }
      const uint32_t stride = uint32_t(waves) * 4u;
      if (pass == 2) {
        // the draws pass 1 recorded, in the order it listed them, four per
        // wave at a time; a group's next record is loaded one step ahead
        const uint32_t nl = __builtin_amdgcn_readfirstlane(s_reg[4]);
        TiledRec nrec{};
        if (nl) nrec = sc_list[min(uint32_t(wave) * 4u + uint32_t(grp), nl - 1u)];
        for (uint32_t i0 = uint32_t(wave) * 4u; i0 < nl; i0 += stride) {
          const uint32_t i = i0 + uint32_t(grp);
          const TiledRec tr = nrec;
          if (i0 + stride < nl) nrec = sc_list[min(i + stride, nl - 1u)];
          if (i >= nl) continue;
          const uint32_t j = b + tr.q, code = tr.code, cn = tr.cn;
          const uint32_t *row = d.d_ent + tr.off;
          const double x = tr.x;
          uint32_t topic;
          if ((code & 3u) == 1u) {
            const uint32_t slots = d_row_slots(cn >> 16);
            const double Mm = rec.a1 * (double(cn & 0xFFFFu) + p.alpha);
            const uint32_t sc = code >> 2;
            if (sc < uint32_t(kTiledAhead)) {
              // the tile-0 chunks, 0 to the split chunk, loaded together and
              // walked in registers (a chunk past the split chunk adds nothing)
              uint32_t rb[kTiledAhead][kMaxRun];
              double tb[kTiledAhead];
#pragma unroll
              for (int c = 0; c < kTiledAhead; ++c) load_run_masked(row, uint32_t(c), slots, li, pad, rb[c]);
#pragma unroll
              for (int c = 0; c < kTiledAhead; ++c) tb[c] = run_sum_tile(rb[c], ts);
              topic = walk_pair(rb, tb, ts, Mm, x, grp, li, hand);
            } else {
              topic = tile_walk(row, slots, ts, Mm, x, pad, grp, li, hand, 0u, sc + 1u);
            }
            if (topic == uint32_t(-1)) topic = K1;  // no positive S' term below KT: cannot happen for x in S'
          } else {
            const int lo = int(code >> 2);
            const uint32_t k = uint32_t(lo * kGroup + li);
            const double term = p.alpha * wt[k];
            topic = pick_segment(k, term, tr.keep + qb[lo], x, grp);
          }
          if (li == 0) d.z_w[j] = uint16_t(topic);
        }
        __syncthreads();
        continue;
      }
      // four tokens per wave at a time, one per 16-lane group.  A token's
      // skip word, key and row offset, and its records of pass 0 are loaded
      // one step ahead, while the group works on the previous token (the
      // fp64 record is loaded beside the row's first chunk); pass 0 then
      // loads the row header and first chunk together (the header is slot 0)
      auto tok_load = [&](uint32_t jt) {
        const uint32_t jj = min(jt, e - 1u), qq = jj - b;
        TiledTok o;
        o.sk = d.skip_bits[jj >> 5];
        o.kr = d.wt_kr[jj];
        o.rec = pass == 0 ? 0u : sc_code[qq];  // pass 1: the split chunk
        o.cn = pass == 0 ? 0u : sc_c1[qq];     // pass 1: pass 0's C1 and the row length
        return o;
      };
      TiledTok nxt = tok_load(b + uint32_t(wave) * 4u + uint32_t(grp));
      // pass 1: lane L draws u for the token of group L % 4 at step L / 4 of
      // each block of 16 steps into the wave's slice of LDS
      double *s_uw = s_u + wave * kWave;
      uint32_t step = 0;
      for (uint32_t j0 = b + uint32_t(wave) * 4u; j0 < e; j0 += stride, ++step) {
        const uint32_t j = j0 + uint32_t(grp);
        const uint32_t q = j - b;  // place in the region
        const TiledTok tk = nxt;
        if (j0 + stride < e) nxt = tok_load(j + stride);
        if (pass == 1 && (step & 15u) == 0u) {
          const uint32_t jl = j0 + uint32_t(lane >> 2) * stride + uint32_t(lane & 3);
          s_uw[lane] = uniform_draw(p.seed, t, d.wt_kr[min(jl, e - 1u)].x);
          __builtin_amdgcn_wave_barrier();
        }
        const uint32_t sk = tk.sk;
        const uint2 kr = tk.kr;
        const uint32_t rec0 = tk.rec, cn0 = tk.cn;
        const bool skipped = j < e && ((sk >> (j & 31u)) & 1u);
        if (pass == 0 && skipped && li == 0) d.z_w[j] = uint16_t(K1);  // decided by the step-3 test
        const bool live = j < e && !skipped;
        if (!live) continue;
        const uint32_t *row = d.d_ent + kr.y;
        if (pass == 0) {
          // the first two chunks in full (a row start plus 2 * kChunk slots
          // stays inside the kRowPad slots past the last row), masked below
          static_assert(kTiledAhead * kChunk <= kRowPad, "the speculative chunks stay inside the D array");
          uint32_t r0[kTiledAhead][kMaxRun];
#pragma unroll
          for (int c = 0; c < kTiledAhead; ++c)
#pragma unroll
            for (int i = 0; i < kMaxRun; ++i) r0[c][i] = row[uint32_t(c) * kChunk + uint32_t(li) * kMaxRun + uint32_t(i)];
          const uint32_t nnz = uint32_t(__shfl(int(r0[0][0]), 0, kGroup)) & 0xFFFFu;
          const uint32_t slots = d_row_slots(nnz);
          const uint32_t nch = (slots + kChunk - 1) / kChunk;
          // a lane's run of kMaxRun slots lies wholly inside or past the row
          // (slots is a multiple of 32)
#pragma unroll
          for (int c = 0; c < kTiledAhead; ++c) {
            if (uint32_t(c) * kChunk + uint32_t(li) * kMaxRun >= slots) {
#pragma unroll
              for (int i = 0; i < kMaxRun; ++i) r0[c][i] = pad;
            }
          }
          if (li == 0) r0[0][0] = pad;  // the row header
          // S' over the tile-0 topics and C1, chunk by chunk up to the split
          // chunk; the loads of up to kTiledAhead chunks are issued together
          double s0 = 0.0;
          uint32_t c1 = 0xFFFFFFFFu;
          uint32_t sc = 0;
          bool open = true;
#pragma unroll
          for (int c = 0; c < kTiledAhead; ++c) {
            if (open) {
              if (k1_lo) c1 = run_count_of<kMaxRun>(r0[c], K1, c1);
              sc = uint32_t(c);
              open = sc + 1u < nch && (uint32_t(__shfl(int(r0[c][kMaxRun - 1]), kGroup - 1, kGroup)) >> 16) < kt;
              s0 += run_sum_tile(r0[c], ts);
            }
          }
          for (uint32_t c0 = kTiledAhead; open; c0 += kTiledAhead) {
            uint32_t r[kTiledAhead][kMaxRun];
#pragma unroll
            for (int c = 0; c < kTiledAhead; ++c) load_run_masked(row, c0 + uint32_t(c), slots, li, pad, r[c]);
#pragma unroll
            for (int c = 0; c < kTiledAhead; ++c) {
              if (open) {
                if (k1_lo) c1 = run_count_of<kMaxRun>(r[c], K1, c1);
                sc = c0 + uint32_t(c);
                open = sc + 1u < nch && (uint32_t(__shfl(int(r[c][kMaxRun - 1]), kGroup - 1, kGroup)) >> 16) < kt;
                s0 += run_sum_tile(r[c], ts);
              }
            }
          }
          const double S0 = gsum<kGroup>(s0);
          c1 = gsum_u32<kGroup>(c1 <= 0xFFFFu ? c1 : 0u);
          if (li == 0) {
            sc_s[q] = S0;
            sc_c1[q] = c1 | (nnz << 16);
            sc_code[q] = sc;
          }
        } else {
          const uint32_t sc = rec0;
          const uint32_t nnz = cn0 >> 16;
          const uint32_t slots = d_row_slots(nnz);
          const uint32_t nch = (slots + kChunk - 1) / kChunk;
          // S' over the tile-1 topics, and C1 where pass 0 did not read it,
          // from the split chunk on; the first batch of chunks stays in
          // registers for the draw
          double s1 = 0.0;
          uint32_t c1 = 0xFFFFFFFFu;
          uint32_t rb[kTiledAhead][kMaxRun];
          double tb[kTiledAhead];
#pragma unroll
          for (int c = 0; c < kTiledAhead; ++c) load_run_masked(row, sc + uint32_t(c), slots, li, pad, rb[c]);
#pragma unroll
          for (int c = 0; c < kTiledAhead; ++c) {
            if (!k1_lo) c1 = run_count_of<kMaxRun>(rb[c], K1, c1);
            tb[c] = run_sum_tile(rb[c], ts);
            s1 += tb[c];
          }
          for (uint32_t c0 = sc + kTiledAhead; c0 < nch; c0 += kTiledAhead) {
            uint32_t r[kTiledAhead][kMaxRun];
#pragma unroll
            for (int c = 0; c < kTiledAhead; ++c) load_run_masked(row, c0 + uint32_t(c), slots, li, pad, r[c]);
#pragma unroll
            for (int c = 0; c < kTiledAhead; ++c) {
              if (!k1_lo) c1 = run_count_of<kMaxRun>(r[c], K1, c1);
              s1 += run_sum_tile(r[c], ts);
            }
          }
          const double S1 = gsum<kGroup>(s1);
          const double S0 = sc_s[q];
          // topic K1's entry was sought in one of the two passes, the other read 0
          const uint32_t C1 = max(cn0 & 0xFFFFu, gsum_u32<kGroup>(c1 <= 0xFFFFu ? c1 : 0u));
          const double Mm = rec.a1 * (double(C1) + p.alpha);  // Eq. 7
          const double S = S0 + S1;
          const double x = s_uw[((step & 15u) << 2) | uint32_t(grp)] * ((Mm + S) + rec.qp);
          uint32_t topic = K1, code = 0u;
          double keep = 0.0;
          if (x < Mm) {
            if (li == 0) n_after_s++;
          } else if (x < Mm + S) {
            if (x < Mm + S0) {
              code = 1u | (sc << 2);  // S' draw in tile 0, whose terms end at the split chunk
            } else if (nch - sc <= uint32_t(kTiledAhead)) {
              // every tile-1 chunk is in registers
              const uint32_t k = walk_pair(rb, tb, ts, Mm + S0, x, grp, li, hand);
              if (k == uint32_t(-1)) code = 1u | (sc << 2);  // nothing positive in tile 1: rounding at the tile edge
              else topic = k;
            } else {
              const uint32_t k = tile_walk(row, slots, ts, Mm + S0, x, pad, grp, li, hand, sc, nch);
              if (k == uint32_t(-1)) code = 1u | (sc << 2);  // nothing positive in tile 1: rounding at the tile edge
              else topic = k;
            }
          } else {
            const double qs = Mm + S;
            const double xq = x - qs;
            if (!(xq < qb[nb])) {
              topic = (K1 == uint32_t(K - 1)) ? uint32_t(K - 2) : uint32_t(K - 1);  // last positive segment
            } else {
              // the largest block lo < nb with qb[lo] <= xq, 16 candidates at a time
              int lo = 0, span = nb;
              while (span > 1) {
                const int step = (span + kGroup - 1) / kGroup;
                const int off = li * step;
                const bool ok = off < span && qb[lo + off] <= xq;
                const uint32_t bm = uint32_t(__ballot(ok) >> (grp * kGroup)) & kGroupMask;
                const int best = bm ? 31 - __clz(bm) : 0;
                lo += best * step;
                span = min(step, span - best * step);
              }
              const uint32_t k = uint32_t(lo * kGroup + li);
              if (uint32_t(lo * kGroup) >= kt) {
                const double term = p.alpha * wt[k - kt];
                topic = pick_segment(k, term, qs + qb[lo], x, grp);
              } else {
                code = 2u | (uint32_t(lo) << 2);  // Q' draw in a tile-0 block
                keep = qs;
              }
            }
          }
          if (li == 0) {
            n_sampled++;
            nnz_sum += nnz;
            if (code) {
              TiledRec tr;
              tr.q = q;
              tr.code = code;
              tr.cn = C1 | (nnz << 16);
              tr.off = kr.y;
              tr.x = x;
              tr.keep = keep;
              sc_list[atomicAdd(&s_reg[4], 1u)] = tr;
            } else {
              d.z_w[j] = uint16_t(topic);
            }
          }
        }
      }
      __syncthreads();
    }
  }
  // per-lane counts of group leaders, summed over the wave
  n_sampled = group_sum_u64<kWave>(n_sampled);
  n_after_s = group_sum_u64<kWave>(n_after_s);
  nnz_sum = group_sum_u64<kWave>(nnz_sum);
  if (lane == 0) {
    if (n_sampled) atomicAdd(&stats[ST_SAMPLED], n_sampled);
    if (n_after_s) atomicAdd(&stats[ST_SKIP_AFTER_S], n_after_s);
    if (nnz_sum) atomicAdd(&stats[ST_NNZ], nnz_sum);
  }
  if (tid == 0) {
    if (n_reg) atomicAdd(&stats[ST_REGIONS], n_reg);
    if (n_dreg) atomicAdd(&stats[ST_DENSE_REGIONS], n_dreg);
    if (row_bytes) atomicAdd(&stats[ST_ROW_BYTES], row_bytes);
  }
}

// Rows of split dense words are accumulated with atomics; clear them and T.
__global__ void k_zero_split(DevState d, Params p) {
  const int64_t total = int64_t(p.n_dense) * p.K;
  for (int64_t x = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; x < total; x += int64_t(gridDim.x) * blockDim.x) {
    if (d.split[x / p.K]) d.w_dense[x] = 0;
  }
  for (int64_t k = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; k < p.K; k += int64_t(gridDim.x) * blockDim.x)
    d.T[k] = 0u;
}

constexpr int kHistAhead = 8;  // word-ordered topic loads per thread issued together in the W rebuild

// W rebuild (Sec. 4.3) for K below kWBitsK by one wave per region, the regions dealt
// round-robin over the waves of the grid, with no workgroup barrier per
// region: the region's counts in the wave's LDS table, then the dense row
// written whole (added with atomics when the word is split) or the sparse
// row compacted in ascending topic order, 64 topics per step by ballot; the
// table is cleared as it is read.  T is accumulated per workgroup in LDS and
// added to the device once at the end.
__global__ __launch_bounds__(kBlock) void k_rebuild_w_wave(DevState d, Params p) {
  extern __shared__ uint32_t ldsu[];
  const int K = p.K;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave, tid = threadIdx.x;
  uint32_t *tloc = ldsu;                                  // [K], the workgroup's
  uint32_t *hist = ldsu + size_t(K) * size_t(1 + wave);  // [K], the wave's
  for (int k = tid; k < K; k += kBlock) tloc[k] = 0u;
  for (int k = lane; k < K; k += kWave) hist[k] = 0u;
  __syncthreads();
  uint32_t bad = 0;
  const int64_t nwaves = int64_t(gridDim.x) * (kBlock / kWave);
  for (int64_t r = int64_t(blockIdx.x) * (kBlock / kWave) + wave; r < p.n_regions; r += nwaves) {
    const uint32_t v = d.region[3 * size_t(r)], b = d.region[3 * size_t(r) + 1], e = d.region[3 * size_t(r) + 2];
    for (uint32_t j0 = b + uint32_t(lane); j0 < e; j0 += uint32_t(kHistAhead * kWave)) {
      uint32_t zz[kHistAhead];
#pragma unroll
      for (int u = 0; u < kHistAhead; ++u) zz[u] = uint32_t(u * kWave) < e - j0 ? uint32_t(d.z_w[j0 + u * kWave]) : 0u;
#pragma unroll
      for (int u = 0; u < kHistAhead; ++u) {
        if (uint32_t(u * kWave) < e - j0) {
          if (zz[u] < uint32_t(K)) atomicAdd(&hist[zz[u]], 1u);
          else bad++;
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");  // a wave's LDS accesses run in order
    if (int32_t(v) < p.n_dense) {
      int32_t *wrow = d.w_dense + size_t(v) * size_t(K);
      const bool split = d.split[v] != 0;
      for (int k = lane; k < K; k += kWave) {
        const uint32_t h = hist[k];
        hist[k] = 0u;
        if (h) atomicAdd(&tloc[k], h);
        if (!split) wrow[k] = int32_t(h);
        else if (h) atomicAdd(&wrow[k], int32_t(h));
      }
    } else {
      const int s = int(v) - p.n_dense;
      uint32_t *out = d.ws_ent + d.ws_cap[s];
      uint32_t base = 0;
      for (int k0 = 0; k0 < K; k0 += kWave) {
        const int k = k0 + lane;
        uint32_t h = 0;
        if (k < K) {
          h = hist[k];
          hist[k] = 0u;
        }
        const unsigned long long m = __ballot(h != 0u);
        if (h) {
          atomicAdd(&tloc[k], h);
          const uint32_t rank = __builtin_amdgcn_mbcnt_hi(uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u));
          out[base + rank] = (uint32_t(k) << 16) | h;
        }
        base += uint32_t(__popcll(m));
      }
      if (lane == 0) d.ws_nnz[s] = base;
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
  }
  __syncthreads();
  for (int k = tid; k < K; k += kBlock)
    if (tloc[k]) atomicAdd(&d.T[k], tloc[k]);
  if (bad) atomicAdd(&d.stats[ST_ERRORS], (unsigned long long)bad);
}

// W rebuild for K >= kWBitsK: the touched topics of a region are marked in
// a bitmap, so the work per region follows its tokens, not K.
// Packed: two 16-bit counts per LDS word (every region shorter than 2^16
// tokens), which halves the table (two workgroups per CU at K = 32,768).
// T is left to k_topic_hist and k_topic_reduce: adding each region's counts
// into T with device atomics cost more than the rest of the rebuild.
template <bool Packed>
__global__ __launch_bounds__(kBlock) void k_rebuild_w_bits(DevState d, Params p) {
  extern __shared__ uint32_t ldsu[];
  const int K = p.K;
  const int nw = (K + 31) / 32;
  const int nh = Packed ? (K + 1) / 2 : K;
  uint32_t *hist = ldsu;                              // [nh]: the region's topic counts
  uint32_t *bits = ldsu + nh;                         // [nw]: topics with a nonzero count
  __shared__ uint32_t s_scan[kBlock / kWave];
  const int tid = threadIdx.x;
  uint32_t bad = 0;
  auto count = [&](int k) -> uint32_t { return Packed ? (hist[k >> 1] >> ((k & 1) << 4)) & 0xFFFFu : hist[k]; };
  for (int k = tid; k < nh; k += kBlock) hist[k] = 0u;
  for (int q = tid; q < nw; q += kBlock) bits[q] = 0u;
  __syncthreads();
  // regions dealt round-robin over the workgroups
  for (int64_t r = blockIdx.x; r < p.n_regions; r += gridDim.x) {
    const uint32_t v = d.region[3 * size_t(r)], b = d.region[3 * size_t(r) + 1], e = d.region[3 * size_t(r) + 2];
    // kHistAhead topic loads per thread in flight at once
    for (uint32_t j0 = b + tid; j0 < e; j0 += uint32_t(kHistAhead * kBlock)) {
      uint32_t zz[kHistAhead];
#pragma unroll
      for (int u = 0; u < kHistAhead; ++u) zz[u] = uint32_t(u * kBlock) < e - j0 ? uint32_t(d.z_w[j0 + u * kBlock]) : 0u;
#pragma unroll
      for (int u = 0; u < kHistAhead; ++u) {
        if (uint32_t(u * kBlock) < e - j0) {
          const uint32_t z = zz[u];
          if (z < uint32_t(K)) {
            if (Packed) atomicAdd(&hist[z >> 1], 1u << ((z & 1u) << 4));
            else atomicAdd(&hist[z], 1u);
            atomicOr(&bits[z >> 5], 1u << (z & 31u));
          } else {
            bad++;
          }
        }
      }
    }
    __syncthreads();
    // the touched topics, each thread a contiguous run of bitmap words (ascending)
    const int per = (nw + kBlock - 1) / kBlock;
    const int q0 = min(nw, tid * per), q1 = min(nw, q0 + per);
    if (int32_t(v) < p.n_dense) {
      int32_t *wrow = d.w_dense + size_t(v) * size_t(K);
      if (d.split[v]) {
        for (int q = q0; q < q1; ++q)
          for (uint32_t m = bits[q]; m; m &= m - 1u) {
            const int k = q * 32 + __ffs(m) - 1;
            atomicAdd(&wrow[k], int32_t(count(k)));
          }
      } else {
        for (int k = tid; k < K; k += kBlock) wrow[k] = int32_t(count(k));
      }
    } else {
      const int s = int(v) - p.n_dense;
      uint32_t cnt = 0;
      for (int q = q0; q < q1; ++q) cnt += uint32_t(__popc(bits[q]));
      uint32_t total = 0;
      uint32_t off = block_exclusive_u32(cnt, s_scan, &total);
      uint32_t *out = d.ws_ent + d.ws_cap[s];
      for (int q = q0; q < q1; ++q)
        for (uint32_t m = bits[q]; m; m &= m - 1u) {
          const int k = q * 32 + __ffs(m) - 1;
          out[off++] = (uint32_t(k) << 16) | count(k);
        }
      if (tid == 0) d.ws_nnz[s] = total;
    }
    __syncthreads();  // the non-split dense row reads every hist entry
    for (int q = q0; q < q1; ++q) {
      const uint32_t mq = bits[q];
      // cleared once both counts of a word are read (a word's two topics
      // are in the same bitmap word)
      for (uint32_t m = mq; m; m &= m - 1u) {
        const int k = q * 32 + __ffs(m) - 1;
        hist[Packed ? k >> 1 : k] = 0u;
      }
      bits[q] = 0u;
    }
    __syncthreads();
  }
  if (bad) atomicAdd(&d.stats[ST_ERRORS], (unsigned long long)bad);
}

// T for large K: the histogram of the word-ordered topics.  Each workgroup
// counts a slice of the tokens (8-token aligned, 8 topics a load) in LDS and
// writes its counts to its row of scratch; k_topic_reduce adds the rows into
// T (zeroed by k_zero_split, so out-of-core chunks add up).
constexpr int kHistBlock = 1024;
__global__ __launch_bounds__(kHistBlock) void k_topic_hist(DevState d, Params p, uint32_t *__restrict__ rows) {
  extern __shared__ uint32_t ldsu[];
  const int K = p.K;
  for (int k = threadIdx.x; k < K; k += kHistBlock) ldsu[k] = 0u;
  __syncthreads();
  const int64_t n = p.n, g = blockIdx.x, G = gridDim.x;
  const int64_t b = (n * g / G) & ~int64_t(7), e = g + 1 == G ? n : (n * (g + 1) / G) & ~int64_t(7);
  int64_t j = b + int64_t(threadIdx.x) * 8;
  for (; j + 8 <= e; j += int64_t(kHistBlock) * 8) {
    const uint4 v = *reinterpret_cast<const uint4 *>(d.z_w + j);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t z0 = w[i] & 0xFFFFu, z1 = w[i] >> 16;
      if (z0 < uint32_t(K)) atomicAdd(&ldsu[z0], 1u);
      if (z1 < uint32_t(K)) atomicAdd(&ldsu[z1], 1u);
    }
  }
  for (; j < e; ++j) {  // the slice's last tokens past a whole 8 (at most 7, one thread)
    const uint32_t z = d.z_w[j];
    if (z < uint32_t(K)) atomicAdd(&ldsu[z], 1u);
  }
  __syncthreads();
  uint32_t *row = rows + size_t(g) * size_t(K);
  for (int k = threadIdx.x; k < K; k += kHistBlock) row[k] = ldsu[k];
}

__global__ __launch_bounds__(kBlock) void k_topic_reduce(DevState d, Params p, const uint32_t *__restrict__ rows,
                                                         int G) {
  const int k = int(blockIdx.x) * kBlock + int(threadIdx.x);
  if (k >= p.K) return;
  uint32_t s = 0;
  for (int g = 0; g < G; ++g) s += rows[size_t(g) * size_t(p.K) + size_t(k)];
  if (s) atomicAdd(&d.T[k], s);
}

constexpr int kPre = 2;   // chunks of 64 tokens per document gathered one document ahead
constexpr int kTail = 4;  // chunks of 64 tokens gathered together past the first kPre

// Inclusive prefix sum of a u32 over the 64 lanes of a wave: DPP shifts
// inside each row of 16 lanes (lanes below the shift read 0), then the row
// totals carried across rows.
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v, int lane) {
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x111, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x112, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x114, 0xF, 0xF, true));
  v += uint32_t(__builtin_amdgcn_update_dpp(0, int(v), 0x118, 0xF, 0xF, true));
  const uint32_t r0 = __builtin_amdgcn_readlane(v, 15), r1 = __builtin_amdgcn_readlane(v, 31),
                 r2 = __builtin_amdgcn_readlane(v, 47);
  v += lane >= 16 ? r0 : 0u;
  v += lane >= 32 ? r1 : 0u;
  v += lane >= 48 ? r2 : 0u;
  return v;
}

// The D row of one document from its topic histogram (16-bit counts, two
// per word of hist) and the bitmap of its topics, by one wave: 64 bitmap
// words (2048 topics) per step, one per lane, each lane listing its word's
// topics at its prefix-sum offset, then one lane per listed topic writing the
// packed entry (topic << 16 | count) in ascending topic order.  The two
// topics of a count word share a bitmap word, so both are listed in the same
// step.  The table and the bitmap are left clear; out points at the row's
// first entry, the header (len << 16 | nnz) goes before it and the padding
// entries (topic K, count 0) after the entries.
__device__ __forceinline__ void emit_row(uint32_t *__restrict__ hist, uint32_t *__restrict__ bits, uint16_t *__restrict__ list, int nw,
                         int K, uint32_t *__restrict__ out, uint32_t len, int lane) {
  uint32_t base = 0;
  for (int q0 = 0; q0 < nw; q0 += kWave) {
    const int q = q0 + lane;
    uint32_t m = 0;
    if (q < nw) {
      m = bits[q];
      bits[q] = 0u;
    }
    const uint32_t cnt = uint32_t(__popc(m));
    const uint32_t incl = wave_incl_scan_u32(cnt, lane);
    const uint32_t n = __builtin_amdgcn_readlane(incl, kWave - 1);
    if (n == 0u) continue;
    uint32_t o = incl - cnt;
    while (m) {
      const uint32_t bit = uint32_t(__ffs(m) - 1);
      m &= m - 1u;
      list[o++] = uint16_t(uint32_t(q) * 32u + bit);
    }
    __threadfence_block();
    for (uint32_t j = uint32_t(lane); j < n; j += kWave) {
      const uint32_t z = list[j];
      const uint32_t zn = j + 1u < n ? uint32_t(list[j + 1u]) : 0xFFFFFFFFu;
      const uint32_t w = hist[z >> 1];
      out[base + j] = (z << 16) | ((z & 1u) ? (w >> 16) : (w & 0xFFFFu));
      // clear a count word after its last listed topic has been read
      if ((z & 1u) || zn != z + 1u) hist[z >> 1] = 0u;
    }
    __threadfence_block();
    base += n;
  }
  for (uint32_t q = base + uint32_t(lane); q + 1u < d_row_slots(base); q += kWave) out[q] = uint32_t(K) << 16;
  if (lane == 0) out[-1] = (len << 16) | base;
  __threadfence_block();
}

// The D rows of the heavy documents (longer than kHeavyDoc), one workgroup
// per document, before the workgroup's waves turn to the light documents.
// Each wave gathers topics of its share of the tokens through the inverted
// index into its own histogram and bitmap (so that LDS atomics contend only
// inside a wave), the tables are added into wave 0's (two 16-bit counts per
// word: a document's counts stay below 2^16, so the halves never carry), and
// wave 0 emits the row.  Every table is left clear.
__device__ void heavy_rebuild_d(const DevState &d, const Params &p, uint32_t *__restrict__ lds, uint32_t &bad) {
  __shared__ uint32_t s_next;
  const int K = p.K, half = (K + 1) / 2, nw = (K + 31) / 32;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), nthr = int(blockDim.x), waves = nthr / kWave;
  const size_t words = d_rebuild_lds_words(K);
  uint32_t *hist = lds + size_t(tid / kWave) * words;
  uint32_t *bits = hist + half;
  for (;;) {
    __syncthreads();  // the tables are clear, s_next is free
    if (tid == 0) s_next = atomicAdd(&d.counters[CNT_HEAVY_REBUILD], 1u);
    __syncthreads();
    const uint32_t h = s_next;
    if (h >= uint32_t(p.n_heavy)) break;
    const uint32_t dd = d.heavy_docs[h];
    const uint32_t b = d.doc_off[dd], e = d.doc_off[dd + 1];
    for (uint32_t p0 = b + uint32_t(tid); p0 < e; p0 += uint32_t(4 * nthr)) {
      uint32_t zz[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const uint32_t pp = p0 + uint32_t(c * nthr);
        zz[c] = pp < e ? d.dt_wpos[pp] : 0u;
      }
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (p0 + uint32_t(c * nthr) < e) zz[c] = d.z_w[zz[c]];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (p0 + uint32_t(c * nthr) < e) {
          const uint32_t z = zz[c];
          if (z < uint32_t(K)) {
            atomicAdd(&hist[z >> 1], (z & 1u) ? 0x10000u : 1u);
            atomicOr(&bits[z >> 5], 1u << (z & 31u));
          } else {
            bad++;
          }
        }
      }
    }
    __syncthreads();
    // the other waves' tables added into wave 0's, and cleared
    for (int q = tid; q < half + nw; q += nthr) {
      uint32_t acc = lds[q];
      for (int w = 1; w < waves; ++w) {
        uint32_t *src = lds + size_t(w) * words + q;
        acc = q < half ? acc + *src : acc | *src;
        *src = 0u;
      }
      lds[q] = acc;
    }
    __syncthreads();
    if (tid < kWave)
      emit_row(lds, lds + half, reinterpret_cast<uint16_t *>(lds + half + nw), nw, K, d.d_ent + d.d_cap[dd] + 1u,
               e - b, lane);
  }
  __syncthreads();  // every table is clear again
}

// D rebuild (Sec. 4.3): per document gather the new topics through the
// inverted index (doc order -> word-order slot) into a per-wave LDS table of
// 16-bit counts, marking each touched topic in a bitmap.  The row is then
// emitted in ascending topic order: each lane expands one bitmap word into a
// list of topics at its prefix-sum offset, and one lane per listed topic
// writes the packed entry.  The work per document is K/2048 wave steps plus
// about one per 32 touched topics, so it follows the tokens, not K.
__global__ __launch_bounds__(kBlock) void k_rebuild_d(DevState d, Params p, int light) {
  extern __shared__ uint32_t ldsu[];
  const int K = p.K;
  const int half = (K + 1) / 2, nw = (K + 31) / 32;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  uint32_t *hist = ldsu + size_t(wave) * d_rebuild_lds_words(K);
  uint32_t *bits = hist + half;
  uint16_t *list = reinterpret_cast<uint16_t *>(bits + nw);
  for (int q = lane; q < half; q += kWave) hist[q] = 0u;
  for (int q = lane; q < nw; q += kWave) bits[q] = 0u;
  uint32_t bad = 0;
  // the heavy documents first, each by the whole workgroup (wave 0's tables shared)
  if (p.n_heavy)
    heavy_rebuild_d(d, p, ldsu, bad);
  int part = light ? 0 : kXcds;  // heavy only: the light documents are k_rebuild_d_sort's
  for (;;) {
    uint32_t d0 = 0, d1 = 0;
    if (!next_docs(d.counters + CNT_REBUILD_D, p, part, lane, d0, d1)) break;
    const int nb = int(d1 - d0);
    // the batch's document offsets and D-row offsets, one per lane (loaded
    // here so that no later wait for them also waits for the prefetches)
    const uint32_t b_all = lane <= nb ? d.doc_off[d0 + uint32_t(lane)] : 0u;
    const uint32_t cap_all = lane < nb ? d.d_cap[d0 + uint32_t(lane)] : 0u;
    const uint32_t e_all = uint32_t(__shfl_down(int(b_all), 1, kWave));
    // the batch's light documents moved to the first lanes (a heavy one is a
    // workgroup's, heavy_rebuild_d), so that the loop below has no branch
    // around them: lane j holds begin, end and D-row offset of light document j
    const bool light = lane < nb && e_all - b_all <= kHeavyDoc;
    const unsigned long long lm = __ballot(light);
    const int nd = __popcll(lm);
    const uint32_t below = __builtin_amdgcn_mbcnt_hi(uint32_t(lm >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(lm), 0u));
    const uint32_t target = light ? below : uint32_t(nd) + (uint32_t(lane) - below);  // distinct lanes
    const uint32_t bv = uint32_t(__builtin_amdgcn_ds_permute(int(target * 4u), int(b_all)));
    const uint32_t ev = uint32_t(__builtin_amdgcn_ds_permute(int(target * 4u), int(e_all)));
    const uint32_t capv = uint32_t(__builtin_amdgcn_ds_permute(int(target * 4u), int(cap_all)));
    // pipeline over the first kPre*64 tokens of each document: the
    // word-order slots of document i+3 and the topics of document i+2 are
    // loaded while document i is processed.  Every load is issued (slot
    // indexes past the batch are clamped; lanes past a document's end read
    // slot 0's topic), so the waits count a fixed number of loads and do not
    // drain the pipeline.
    const uint32_t last = uint32_t(p.n - 1);
    auto slots_of = [&](int doc, uint32_t (&w)[kPre]) {
      const uint32_t bn = __builtin_amdgcn_readlane(bv, doc);
#pragma unroll
      for (int c = 0; c < kPre; ++c) w[c] = d.dt_wpos[min(bn + uint32_t(c * kWave + lane), last)];
    };
    auto topics_of = [&](int doc, const uint32_t (&w)[kPre], uint32_t (&z)[kPre]) {
      const uint32_t bn = __builtin_amdgcn_readlane(bv, doc), en = __builtin_amdgcn_readlane(ev, doc);
#pragma unroll
      for (int c = 0; c < kPre; ++c) z[c] = d.z_w[bn + uint32_t(c * kWave + lane) < en ? w[c] : 0u];
    };
    uint32_t zA[kPre], zB[kPre], wC[kPre], wD[kPre];
    slots_of(0, wD);
    topics_of(0, wD, zA);
    slots_of(1, wD);
    topics_of(1, wD, zB);
    slots_of(2, wC);
    for (int i = 0; i < nd; ++i) {
      const uint32_t b = __builtin_amdgcn_readlane(bv, i), e = __builtin_amdgcn_readlane(ev, i);
      uint32_t zv[kPre];
#pragma unroll
      for (int c = 0; c < kPre; ++c) {
        zv[c] = zA[c];
        zA[c] = zB[c];
      }
      slots_of(i + 3, wD);
      topics_of(i + 2, wC, zB);
#pragma unroll
      for (int c = 0; c < kPre; ++c) wC[c] = wD[c];
#pragma unroll
      for (int c = 0; c < kPre; ++c) {
        if (b + uint32_t(c * kWave + lane) < e) {
          const uint32_t z = zv[c];
          if (z < uint32_t(K)) {
            atomicAdd(&hist[z >> 1], (z & 1u) ? 0x10000u : 1u);
            atomicOr(&bits[z >> 5], 1u << (z & 31u));
          } else {
            bad++;
          }
        }
      }
      // the rest of a long document, kTail chunks at a time: all their slot
      // loads, then all their topic gathers, are in flight together
      for (uint32_t p0 = b + uint32_t(kPre * kWave); p0 < e; p0 += uint32_t(kTail * kWave)) {
        uint32_t zt[kTail];
#pragma unroll
        for (int c = 0; c < kTail; ++c) {
          const uint32_t pp = p0 + uint32_t(c * kWave + lane);
          zt[c] = pp < e ? d.dt_wpos[pp] : 0u;
        }
#pragma unroll
        for (int c = 0; c < kTail; ++c) {
          const uint32_t pp = p0 + uint32_t(c * kWave + lane);
          if (pp < e) zt[c] = d.z_w[zt[c]];
        }
#pragma unroll
        for (int c = 0; c < kTail; ++c) {
          if (p0 + uint32_t(c * kWave + lane) < e) {
            const uint32_t z = zt[c];
            if (z < uint32_t(K)) {
              atomicAdd(&hist[z >> 1], (z & 1u) ? 0x10000u : 1u);
              atomicOr(&bits[z >> 5], 1u << (z & 31u));
            } else {
              bad++;
            }
          }
        }
      }
      __threadfence_block();
      // (readlane returns a signed int: the offset is taken back to unsigned,
      // since D has more than 2^31 slots on the largest corpora)
      emit_row(hist, bits, list, nw, K, d.d_ent + uint32_t(__builtin_amdgcn_readlane(capv, i)) + 1u, e - b, lane);
    }
  }
  if (bad) atomicAdd(&d.stats[ST_ERRORS], (unsigned long long)bad);
}

// The D rows of the light documents for large K, one wave per document
// without a table of K counts (which leaves room for two waves per CU at
// K = 32,768): the wave gathers the document's topics into its LDS buffer,
// sorts them (bitonic, ascending; topics >= K are errors and sort last as
// 0xFFFF), and writes one entry per run of equal topics.  The rows are the
// ones emit_row writes: entries in ascending topic order, padding entries
// of topic K, the header (length << 16 | entries).
constexpr int kSortGather = 8;  // slots per lane whose loads are in flight together

// Bitonic sort (ascending) of the P = 64 * E slots of sz in registers: lane l
// holds slots l * E .. l * E + E - 1; compare-exchanges between slots of one
// lane stay in registers, those between lanes exchange by shuffle.  The same
// network as the sort in LDS below, so the same result.
template <int E>
__device__ __forceinline__ void sort_in_registers(uint16_t *__restrict__ sz, int lane) {
  constexpr uint32_t P = uint32_t(E) * uint32_t(kWave);
  uint32_t x[E];
#pragma unroll
  for (int r = 0; r < E; ++r) x[r] = sz[lane * E + r];
#pragma unroll
  for (uint32_t size = 2; size <= P; size <<= 1) {
#pragma unroll
    for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
      if (stride < uint32_t(E)) {
#pragma unroll
        for (int r = 0; r < E; ++r) {
          if ((uint32_t(r) & stride) == 0u) {
            const int q = r | int(stride);
            const bool asc = (uint32_t(lane * E + r) & size) == 0u;
            const uint32_t lo = min(x[r], x[q]), hi = max(x[r], x[q]);
            x[r] = asc ? lo : hi;
            x[q] = asc ? hi : lo;
          }
        }
      } else {
        const int dl = int(stride / uint32_t(E));        // partner lane distance
        const bool upper = (lane & dl) != 0;             // this lane holds the higher slot
        const bool asc = (uint32_t(lane * E) & size) == 0u;
#pragma unroll
        for (int r = 0; r < E; ++r) {
          const uint32_t o = uint32_t(__shfl_xor(int(x[r]), dl, kWave));
          x[r] = (asc != upper) ? min(x[r], o) : max(x[r], o);
        }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < E; ++r) sz[lane * E + r] = uint16_t(x[r]);
}
__global__ __launch_bounds__(kBlock) void k_rebuild_d_sort(DevState d, Params p) {
  extern __shared__ uint32_t ldsu[];
  const int K = p.K;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  uint16_t *sz = reinterpret_cast<uint16_t *>(ldsu) + size_t(wave) * kHeavyDoc;
  uint32_t bad = 0;
  int part = 0;
  for (;;) {
    uint32_t d0 = 0, d1 = 0;
    if (!next_docs(d.counters + CNT_REBUILD_D, p, part, lane, d0, d1)) break;
    for (uint32_t dd = d0; dd < d1; ++dd) {
      const uint32_t b = d.doc_off[dd], len = d.doc_off[dd + 1] - b;
      if (len > uint32_t(kHeavyDoc)) continue;  // a heavy document: k_rebuild_d's
      uint32_t P = kWave;
      while (P < len) P <<= 1;
      // the topics, kSortGather slots per lane at a time (slot loads, then gathers)
      for (uint32_t q0 = 0; q0 < P; q0 += uint32_t(kSortGather * kWave)) {
        uint32_t zz[kSortGather];
#pragma unroll
        for (int c = 0; c < kSortGather; ++c) {
          const uint32_t q = q0 + uint32_t(c * kWave + lane);
          zz[c] = q < len ? d.dt_wpos[b + q] : 0u;
        }
#pragma unroll
        for (int c = 0; c < kSortGather; ++c) {
          const uint32_t q = q0 + uint32_t(c * kWave + lane);
          if (q < len) zz[c] = d.z_w[zz[c]];
        }
#pragma unroll
        for (int c = 0; c < kSortGather; ++c) {
          const uint32_t q = q0 + uint32_t(c * kWave + lane);
          if (q < P) {
            uint32_t z = 0xFFFFu;
            if (q < len) {
              if (zz[c] < uint32_t(K)) z = zz[c];
              else bad++;
            }
            sz[q] = uint16_t(z);
          }
        }
      }
      __threadfence_block();
      // bitonic sort of the P slots, ascending: in registers up to 512 slots
      if (P <= 512u) {
        if (P == 64u) sort_in_registers<1>(sz, lane);
        else if (P == 128u) sort_in_registers<2>(sz, lane);
        else if (P == 256u) sort_in_registers<4>(sz, lane);
        else sort_in_registers<8>(sz, lane);
        __threadfence_block();
      }
      for (uint32_t size = 2; P > 512u && size <= P; size <<= 1) {
        for (uint32_t stride = size >> 1; stride > 0; stride >>= 1) {
          for (uint32_t t = uint32_t(lane); t < P / 2; t += kWave) {
            const uint32_t i = 2 * t - (t & (stride - 1)), j = i + stride;
            const uint32_t a = sz[i], c = sz[j];
            if ((a > c) == ((i & size) == 0)) {
              sz[i] = uint16_t(c);
              sz[j] = uint16_t(a);
            }
          }
          __threadfence_block();
        }
      }
      // entries: a run starts where the topic changes; first the number of
      // entries, then the runs from the last 64 slots to the first, so that
      // each run's end (the next run's start) is known
      uint32_t nnz = 0;
      for (uint32_t q0 = 0; q0 < len; q0 += kWave) {
        const uint32_t i = q0 + uint32_t(lane);
        const uint32_t zi = i < len ? sz[i] : 0xFFFFu, zp = i > 0 && i < len ? sz[i - 1] : 0xFFFFFFFFu;
        nnz += uint32_t(__popcll(__ballot(i < len && zi != 0xFFFFu && zi != zp)));
      }
      uint32_t *out = d.d_ent + d.d_cap[dd] + 1u;
      uint32_t after = nnz, next = len;  // entries and first run start past the current 64 slots
      for (int q0 = int((len - 1u) & ~uint32_t(kWave - 1)); q0 >= 0; q0 -= kWave) {
        const uint32_t i = uint32_t(q0 + lane);
        const uint32_t zi = i < len ? sz[i] : 0xFFFFu, zp = i > 0 && i < len ? sz[i - 1] : 0xFFFFFFFFu;
        const bool start = i < len && zi != zp;
        const unsigned long long sm = __ballot(start), em = __ballot(start && zi != 0xFFFFu);
        const unsigned long long above = lane == kWave - 1 ? 0ull : sm & (~0ull << (lane + 1));
        const uint32_t end = above ? uint32_t(q0) + uint32_t(__ffsll(above) - 1) : next;
        const uint32_t n_here = uint32_t(__popcll(em));
        if (start && zi != 0xFFFFu) {
          const uint32_t below = uint32_t(__popcll(em & ((1ull << lane) - 1ull)));
          out[after - n_here + below] = (zi << 16) | (end - i);
        }
        after -= n_here;
        next = sm ? uint32_t(q0) + uint32_t(__ffsll(sm) - 1) : next;
      }
      for (uint32_t q = nnz + uint32_t(lane); q + 1u < d_row_slots(nnz); q += kWave) out[q] = uint32_t(K) << 16;
      if (lane == 0) out[-1] = (len << 16) | nnz;
      __threadfence_block();
    }
  }
  if (bad) atomicAdd(&d.stats[ST_ERRORS], (unsigned long long)bad);
}

// LLPT terms per region (Sec. 2.2): for every token,
//   log2( (sum_{k in nz(D[d])} D[d][k] W^[v][k] + alpha * sum_k W^[v][k]) / (len(d) + K alpha) ),
// summed in a fixed order so that the result does not depend on the schedule.
__global__ __launch_bounds__(kBlock) void k_loglik(DevState d, Params p) {
  extern __shared__ double lds[];
  const int K = p.K;
  // large K: the row lives in the workgroup's slice of global scratch
  double *wh = p.big_k ? d.wscratch + size_t(blockIdx.x) * size_t(K) : lds;
  __shared__ uint32_t s_reg[3];
  __shared__ int s_valid;
  __shared__ uint32_t s_r;
  __shared__ double s_part[kBlock / kGroup];
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int gid = tid / kGroup, li = lane % kGroup;  // 16 groups per block
  uint32_t cur = 0xFFFFFFFFu;
  double sumw = 0.0;
  const double Kalpha = double(K) * p.alpha;
  for (;;) {
    if (tid == 0) {
      const uint32_t r = atomicAdd(&d.counters[CNT_LOGLIK], 1u);
      s_r = r;
      s_valid = int64_t(r) < p.n_regions;
      if (s_valid) {
        s_reg[0] = d.region[3 * size_t(r)];
        s_reg[1] = d.region[3 * size_t(r) + 1];
        s_reg[2] = d.region[3 * size_t(r) + 2];
      }
    }
    __syncthreads();
    if (!s_valid) break;
    const uint32_t v = s_reg[0], b = s_reg[1], e = s_reg[2], r = s_r;
    if (v != cur) {
      cur = v;
      sumw = d.wrec[v].sumw;
      if (int32_t(v) < p.n_dense) {
        const int32_t *wrow = d.w_dense + size_t(v) * size_t(K);
        for (int k = tid; k < K; k += kBlock) wh[k] = what(uint32_t(wrow[k]), p.beta, d.den[k]);
      } else {
        const int s = int(v) - p.n_dense;
        const uint32_t *ents = d.ws_ent + d.ws_cap[s];
        const uint32_t nnz = d.ws_nnz[s];
        for (int k = tid; k < K; k += kBlock) wh[k] = d.bden[k];
        __syncthreads();
        for (uint32_t q = tid; q < nnz; q += kBlock) {
          const uint32_t ent = ents[q];
          wh[ent >> 16] = what(ent & 0xFFFFu, p.beta, d.den[ent >> 16]);
        }
      }
      __syncthreads();
    }
    double part = 0.0;
    for (uint32_t j = b + uint32_t(gid); j < e; j += kBlock / kGroup) {
      const uint32_t *row = d.d_ent + d.wt_kr[j].y + 1;
      const uint32_t hdr = row[-1];
      const uint32_t nnz = hdr & 0xFFFFu;
      double acc = 0.0;
      for (uint32_t q = li; q < nnz; q += kGroup) {
        const uint32_t ent = row[q];
        acc += double(ent & 0xFFFFu) * wh[ent >> 16];
      }
      const double num = group_sum<kGroup>(acc) + p.alpha * sumw;
      const double len = double(hdr >> 16);
      part += log2(num / (len + Kalpha));
    }
    if (li == 0) s_part[gid] = part;
    __syncthreads();
    if (tid == 0) {
      double s = 0.0;
      for (int q = 0; q < kBlock / kGroup; ++q) s += s_part[q];
      d.ll_part[r] = s;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(kBlock) void k_loglik_reduce(const double *__restrict__ part, int64_t n,
                                                          double *__restrict__ out) {
  __shared__ double red[kBlock / kWave];
  double s = 0.0;
  for (int64_t q = threadIdx.x; q < n; q += kBlock) s += part[q];
  s = block_sum(s, red);
  if (threadIdx.x == 0) out[0] = s;
}

// Total entries of D (for the size query of lda_get_counts).
__global__ void k_sum_nnz(const uint32_t *__restrict__ d_ent, const uint32_t *__restrict__ d_cap, int32_t M,
                          unsigned long long *__restrict__ out) {
  unsigned long long s = 0;
  for (int64_t dd = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; dd < M; dd += int64_t(gridDim.x) * blockDim.x)
    s += d_ent[d_cap[dd]] & 0xFFFFu;
  s = group_sum_u64<kWave>(s);
  if ((threadIdx.x & (kWave - 1)) == 0 && s) atomicAdd(out, s);
}

}  // namespace

// ---------------------------------------------------------- launchers ----

// Dynamic LDS above 64 KB per workgroup has to be requested for the kernel.
template <typename F>
hipError_t allow_lds(F *kernel, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(reinterpret_cast<const void *>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             int(bytes));
}

hipError_t launch_init_topics(const DevState &d, const Params &p, hipStream_t s) {
  const int64_t blocks = std::min<int64_t>((p.n + kBlock - 1) / kBlock, int64_t(p.grid_docs) * 8);
  hipLaunchKernelGGL(k_init_topics, dim3(uint32_t(blocks)), dim3(kBlock), 0, s, d.wt_kr, d.z_w, p.n, p.K, p.seed);
  return hipGetLastError();
}

hipError_t launch_clear_skips(const DevState &d, const Params &p, uint32_t t, hipStream_t s, bool reset_count) {
  const int64_t n = skip_words(p.n);
  const int64_t blocks = std::min<int64_t>((n + kBlock - 1) / kBlock, int64_t(p.grid_docs) * 4);
  hipLaunchKernelGGL(k_clear_skips, dim3(uint32_t(std::max<int64_t>(blocks, 1))), dim3(kBlock), 0, s, d.skip_bits,
                     d.skip_doc, n, n + 64, d.skip_hist, t, reset_count ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_reset_counters(uint32_t *counters, hipStream_t s) {
  hipLaunchKernelGGL(k_reset_counters, dim3(1), dim3(kWave), 0, s, counters);
  return hipGetLastError();
}

hipError_t launch_begin_iteration(const DevState &d, const Params &p, hipStream_t s) {
  hipLaunchKernelGGL(k_begin, dim3((p.K + kBlock - 1) / kBlock), dim3(kBlock), 0, s, d.T, d.den, d.bden, p.K, p.beta,
                     p.vbeta, d.counters, d.stats);
  return hipGetLastError();
}

hipError_t launch_beta_sum(const DevState &d, const Params &p, hipStream_t s) {
  hipLaunchKernelGGL(k_beta_sum, dim3(1), dim3(kBlock), 0, s, d, p);
  return hipGetLastError();
}
hipError_t launch_word_pre(const DevState &d, const Params &p, hipStream_t s) {
  if (p.sparse_pre) {
    // the topic list and the sum of beta/den[k] follow the current T
    size_t bytes = d.topic_tmp_bytes;
    hipError_t err = sort_pairs_u32(d.topic_tmp, bytes, d.T, d.topic_keys, d.topic_iota, d.topic_order, p.K, 32, s);
    if (err != hipSuccess) return err;
    err = launch_beta_sum(d, p, s);
    if (err != hipSuccess) return err;
  }
  // below K = 4,096 a table of K 16-bit counts per wave (at most 32 KB)
  const size_t lds = p.sparse_pre ? 0 : sizeof(uint16_t) * size_t((p.K + 1) & ~1) * (kBlock / kWave);
  const uint32_t grid = uint32_t((p.n_present + kBlock / kWave - 1) / (kBlock / kWave));
  hipLaunchKernelGGL(k_word_pre_wave, dim3(grid), dim3(kBlock), lds, s, d, p);
  return hipGetLastError();
}

hipError_t launch_doc_pass(const DevState &d, const Params &p, uint32_t t, hipStream_t s) {
  const size_t lds = sizeof(uint16_t) * size_t(p.K) * size_t(p.doc_waves);
  const auto kernel = p.key_identity ? k_doc_pass<true> : k_doc_pass<false>;
  hipError_t err = allow_lds(kernel, lds);
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(kernel, dim3(uint32_t(p.grid_docs)), dim3(kWave * p.doc_waves), lds, s, d, p, t, d.stats);
  return hipGetLastError();
}

// The sampler's dynamic LDS for K topics and workgroups of nb threads: the
// W^' row, the Q' block prefix, the per-wave batch slices (u, row offset,
// length, drawn topic, list place; the long-row hand-off) and the region.
size_t sampler_lds_bytes(int K, int nb, bool q_table) {
  const size_t blocks = size_t((K + kGroup - 1) / kGroup);
  const size_t words = size_t(wh_entries(K)) + size_t(q_blocks_padded(int(blocks))) + 1;
  size_t bytes = sizeof(double) * words + size_t(nb) * (sizeof(double) + 2 * sizeof(uint32_t) + sizeof(uint16_t) + 1) +
                 sizeof(uint32_t) * (size_t(nb) / kGroup * kMaxRun + 4);
  if (q_table) bytes += blocks * (kQwStride * sizeof(double) + 1);
  return bytes;
}

// Threads per sampler workgroup for this K: `want` when nonzero, else the
// size with the most resident waves per CU (ties to the smaller).  LDS holds
// the W^ row, so a large K leaves room for few workgroups and larger ones
// keep more waves busy.  0 when the size asked for (or none) fits.
// *q_table: whether the per-topic partial sums of the Q' blocks are kept in
// LDS (q_draw's search instead of its walk; the same draws), which they are
// when they leave the chosen size as many resident waves.
static int sampler_waves(int K, int nb, bool q_table) {
  const size_t lds = sampler_lds_bytes(K, nb, q_table);
  hipError_t err = nb == 256 ? allow_lds(k_sampler, lds) : nb == 512 ? allow_lds(k_sampler_512, lds)
                                                                      : allow_lds(k_sampler_1024, lds);
  int blocks = 0;
  if (err == hipSuccess)
    err = nb == 256 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_sampler, nb, lds)
        : nb == 512 ? hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_sampler_512, nb, lds)
                    : hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_sampler_1024, nb, lds);
  (void)hipGetLastError();
  return err == hipSuccess ? blocks * nb / kWave : 0;
}
int sampler_block(int K, int want, bool *q_table) {
  int best = 0, best_waves = 0;
  const int sizes[3] = {256, 512, 1024};
  for (int q = 0; q < 3; ++q) {
    const int nb = sizes[q];
    if (want && nb != want) continue;
    const int waves = sampler_waves(K, nb, false);
    if (waves > best_waves) {
      best = nb;
      best_waves = waves;
    }
  }
  *q_table = best && sampler_waves(K, best, true) >= best_waves;
  return best;
}

int tiled_topics(int K) { return ((K + 2) / 2 + kGroup - 1) / kGroup * kGroup; }
size_t tiled_lds_bytes(int K, int kt) {
  const size_t nb = size_t((K + kGroup - 1) / kGroup);
  return sizeof(double) * (size_t(kt) + kGroup + nb + 1 + kTiledBlock) +
         sizeof(uint32_t) * (kTiledBlock / kGroup * kMaxRun + 6);
}
hipError_t launch_sampler(const DevState &d, const Params &p, uint32_t t, hipStream_t s) {
  if (p.big_k) {
    // the tile must start at LDS address 0 (wt_of): no static LDS
    static const hipError_t lds_at_0 = [] {
      hipFuncAttributes a;
      const hipError_t e = hipFuncGetAttributes(&a, reinterpret_cast<const void *>(k_sampler_tiled));
      return e != hipSuccess ? e : a.sharedSizeBytes == 0 ? hipSuccess : hipErrorInvalidConfiguration;
    }();
    if (lds_at_0 != hipSuccess) return lds_at_0;
    // a tile's Q' blocks: at most two per thread
    if (p.tile_topics / kGroup + 1 > 2 * kTiledBlock) return hipErrorInvalidValue;
    const size_t lds = tiled_lds_bytes(p.K, p.tile_topics);
    hipError_t err = allow_lds(k_sampler_tiled, lds);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(k_sampler_tiled, dim3(uint32_t(tiled_grid(p))), dim3(kTiledBlock), lds, s, d, p, t, d.stats);
    return hipGetLastError();
  }
  const int nb = p.sampler_block;
  const size_t lds = sampler_lds_bytes(p.K, nb, p.q_table != 0);
  const uint32_t grid = uint32_t(std::max<int64_t>(1, int64_t(p.grid_regions) * kBlock / nb));
  hipError_t err;
  if (p.light_begin == 0) return hipSuccess;  // every region is light
  if (nb == 1024) {
    err = allow_lds(k_sampler_1024, lds);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(k_sampler_1024, dim3(grid), dim3(1024), lds, s, d, p, t, d.stats);
  } else if (nb == 512) {
    err = allow_lds(k_sampler_512, lds);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(k_sampler_512, dim3(grid), dim3(512), lds, s, d, p, t, d.stats);
  } else {
    err = allow_lds(k_sampler, lds);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(k_sampler, dim3(grid), dim3(256), lds, s, d, p, t, d.stats);
  }
  return hipGetLastError();
}

hipError_t launch_sampler_light(const DevState &d, const Params &p, uint32_t t, hipStream_t s) {
  if (p.light_begin >= p.n_regions) return hipSuccess;
  const size_t lds = sampler_lds_bytes(p.K, kWave, p.q_table != 0);
  hipError_t err = allow_lds(k_sampler_light, lds);
  if (err != hipSuccess) return err;
  const int64_t n_light = p.n_regions - p.light_begin;
  const uint32_t grid = uint32_t(std::min<int64_t>(n_light, int64_t(p.grid_regions) * 2));
  hipLaunchKernelGGL(k_sampler_light, dim3(grid), dim3(kWave), lds, s, d, p, t, d.stats);
  return hipGetLastError();
}

hipError_t launch_rebuild(const DevState &d, const Params &p, hipStream_t s) {
  hipError_t err = launch_zero_split(d, p, s);
  if (err == hipSuccess) err = launch_rebuild_w(d, p, s);
  if (err == hipSuccess) err = launch_rebuild_d(d, p, s);
  return err;
}

hipError_t launch_zero_split(const DevState &d, const Params &p, hipStream_t s) {
  const int64_t zb = std::min<int64_t>((int64_t(p.n_dense) * p.K + kBlock - 1) / kBlock + 1, 65536);
  hipLaunchKernelGGL(k_zero_split, dim3(uint32_t(zb)), dim3(kBlock), 0, s, d, p);
  return hipGetLastError();
}

hipError_t launch_rebuild_w(const DevState &d, const Params &p, hipStream_t s) {
  hipError_t err;
  // large K: the bitmap variants, whose work follows the tokens instead of K
  const size_t nwords = size_t((p.K + 31) / 32);
  if (w_bits(p)) {
    // two 16-bit counts per word when every region is shorter than 2^16 tokens
    const bool packed = p.max_region > 0 && p.max_region < 65536;
    const size_t wlds = sizeof(uint32_t) * ((packed ? size_t(p.K + 1) / 2 : size_t(p.K)) + nwords);
    if (packed) {
      err = allow_lds(k_rebuild_w_bits<true>, wlds);
      if (err != hipSuccess) return err;
      hipLaunchKernelGGL(k_rebuild_w_bits<true>, dim3(uint32_t(p.grid_regions)), dim3(kBlock), wlds, s, d, p);
    } else {
      err = allow_lds(k_rebuild_w_bits<false>, wlds);
      if (err != hipSuccess) return err;
      hipLaunchKernelGGL(k_rebuild_w_bits<false>, dim3(uint32_t(p.grid_regions)), dim3(kBlock), wlds, s, d, p);
    }
    if ((err = hipGetLastError()) != hipSuccess) return err;
    // T: per-workgroup histograms in the LLPT kernel's scratch (idle here:
    // loglik_grid_big_k rows of K doubles hold as many rows of K counts)
    if (!d.wscratch) return hipErrorInvalidValue;  // allocated before any rebuild
    const int G = loglik_grid_big_k(p);
    uint32_t *rows = reinterpret_cast<uint32_t *>(d.wscratch);
    err = allow_lds(k_topic_hist, sizeof(uint32_t) * size_t(p.K));
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(k_topic_hist, dim3(uint32_t(G)), dim3(kHistBlock), sizeof(uint32_t) * size_t(p.K), s, d, p,
                       rows);
    if ((err = hipGetLastError()) != hipSuccess) return err;
    hipLaunchKernelGGL(k_topic_reduce, dim3(uint32_t((p.K + kBlock - 1) / kBlock)), dim3(kBlock), 0, s, d, p, rows, G);
  } else {
    // one wave per region: the workgroup's T table and a count table per wave
    const size_t wlds = sizeof(uint32_t) * (1 + kBlock / kWave) * size_t(p.K);
    err = allow_lds(k_rebuild_w_wave, wlds);
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(k_rebuild_w_wave, dim3(uint32_t(p.grid_regions)), dim3(kBlock), wlds, s, d, p);
  }
  return hipGetLastError();
}

hipError_t launch_rebuild_d(const DevState &d, const Params &p, hipStream_t s) {
  hipError_t err;
  const size_t dlds = sizeof(uint32_t) * d_rebuild_lds_words(p.K) * size_t(p.doc_waves);
  err = allow_lds(k_rebuild_d, dlds);
  if (err != hipSuccess) return err;
  // half the document grid (4 workgroups per CU): fewer waves in flight keep
  // a narrower window of documents, whose topic gathers then hit the caches
  // more often
  const uint32_t dgrid = uint32_t(std::max(1, p.grid_docs / 2));
  if (!p.big_k) {
    hipLaunchKernelGGL(k_rebuild_d, dim3(dgrid), dim3(kWave * p.doc_waves), dlds, s, d, p, 1);
    return hipGetLastError();
  }
  // large K: the heavy documents with tables of K counts, the light ones by sorting
  if (p.n_heavy) {
    hipLaunchKernelGGL(k_rebuild_d, dim3(dgrid), dim3(kWave * p.doc_waves), dlds, s, d, p, 0);
    if ((err = hipGetLastError()) != hipSuccess) return err;
  }
  const size_t slds = sizeof(uint16_t) * size_t(kHeavyDoc) * (kBlock / kWave);
  hipLaunchKernelGGL(k_rebuild_d_sort, dim3(uint32_t(p.grid_docs)), dim3(kBlock), slds, s, d, p);
  return hipGetLastError();
}

hipError_t launch_sum_nnz(const DevState &d, const Params &p, unsigned long long *out, hipStream_t s) {
  const int64_t blocks = std::min<int64_t>((int64_t(p.M) + kBlock - 1) / kBlock, 4096);
  hipLaunchKernelGGL(k_sum_nnz, dim3(uint32_t(std::max<int64_t>(blocks, 1))), dim3(kBlock), 0, s, d.d_ent, d.d_cap,
                     p.M, out);
  return hipGetLastError();
}

// ------------------------------------------------- allocation-free LLPT ----
// The scratch of lda_loglik_noalloc: the scheduler counters, the result and
// the per-region partial sums of the LLPT kernels, in one fixed device array
// that every handle on a device shares.  In host code the array's name is not
// a device address: only the address hipGetSymbolAddress returns (one per
// device) may reach a kernel or a copy.
static __device__ __align__(256) unsigned char scratch[kNoAllocHead + sizeof(double) * size_t(LDA_NOALLOC_MAX_REGIONS)];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_addr[kMaxDevices] = {};
}  // namespace

hipError_t noalloc_scratch_address(void **out) {
  *out = nullptr;
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    void *ptr = nullptr;
    err = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return err;
    g_scratch_addr[dev] = ptr;
  }
  *out = g_scratch_addr[dev];
  return hipSuccess;
}

hipError_t launch_loglik_noalloc(DevState d, const Params &p, void *scratch_dev, hipStream_t s) {
  if (p.n_regions > int64_t(LDA_NOALLOC_MAX_REGIONS)) return hipErrorInvalidValue;
  unsigned char *base = static_cast<unsigned char *>(scratch_dev);
  d.counters = reinterpret_cast<uint32_t *>(base);                  // cleared by k_begin
  d.ll_out = reinterpret_cast<double *>(base + kNoAllocResult);      // written by k_loglik_reduce
  d.ll_part = reinterpret_cast<double *>(base + kNoAllocHead);       // one slot per region, each written
  d.stats = nullptr;
  hipError_t err = launch_begin_iteration(d, p, s);
  if (err == hipSuccess) err = launch_word_pre(d, p, s);
  if (err == hipSuccess) err = launch_loglik(d, p, s);
  return err;
}

hipError_t launch_sum_f64(const double *part, int64_t n, double *out, hipStream_t s) {
  hipLaunchKernelGGL(k_loglik_reduce, dim3(1), dim3(kBlock), 0, s, part, n, out);
  return hipGetLastError();
}

hipError_t launch_loglik(const DevState &d, const Params &p, hipStream_t s) {
  const size_t lds = p.big_k ? 0 : sizeof(double) * size_t(p.K);
  hipError_t err0 = allow_lds(k_loglik, lds);
  if (err0 != hipSuccess) return err0;
  // large K: one workgroup per slice of the W^' scratch
  const uint32_t grid = uint32_t(p.big_k ? loglik_grid_big_k(p) : p.grid_regions);
  hipLaunchKernelGGL(k_loglik, dim3(grid), dim3(kBlock), lds, s, d, p);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(k_loglik_reduce, dim3(1), dim3(kBlock), 0, s, d.ll_part, p.n_regions, d.ll_out);
  return hipGetLastError();
}

}  // namespace lda
