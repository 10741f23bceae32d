/*
 * liblda: synchronous collapsed-Gibbs LDA (ESCA) on one AMD Instinct MI355X.
 *
 * Method: arXiv 2007.08725 (ezLDA).  Each iteration draws a new topic for
 * every token from
 *     p(k) ~ (D[d][k] + alpha) * (W[v][k] + beta) / (T[k] + V*beta)     (Sec. 2.2, Eq. 1)
 * against the counts as they stood when the iteration began (the counts
 * include the token itself; the update is applied after every token is drawn,
 * Sec. 4.3).  The draw uses the three-branch split of Sec. 3.2 (Eq. 5) with the
 * S_est skip test (Eq. 6-9), the hybrid dense/sparse word-topic table and
 * inverted index of Sec. 4.2-4.3, and the atomic region scheduler with
 * large-word splitting of Sec. 5.1.
 *
 * Random numbers: Philox4x32-10 (Salmon et al., SC'11), key = seed,
 *   draw of token i at iteration t: counter (i, 0, t, 0), u = ((x0<<32|x1)>>11) * 2^-53
 *   initial topic of token i:       counter (i, 0, 0, 1), z0 = (x0 * K) >> 32
 * where i is the token's index in the caller's input order.  Results are
 * therefore independent of the schedule, the region size and the S_est depth.
 *
 * Conventions for every call:
 *   - Host pointers are caller-owned and borrowed only for the duration of the
 *     call.  All device memory is owned by the handle.
 *   - Every call returns an lda_status; nothing throws across this boundary.
 *     lda_last_error() gives a message for the last failure on a handle.
 *   - A handle is not thread-safe.  All device work runs on the handle's
 *     stream; each call returns after its work has completed.
 *   - After LDA_E_DEVICE the handle is poisoned: later calls return
 *     LDA_E_STATE until lda_destroy.
 */
#ifndef LDA_H
#define LDA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct lda_handle lda_handle;

typedef enum {
  LDA_OK = 0,
  LDA_E_ARG = 1,    /* NULL pointer, bad size, bad id, non-finite or non-positive alpha/beta */
  LDA_E_RANGE = 2,  /* a limit of the 16-bit packed formats or 32-bit positions is exceeded */
  LDA_E_NOMEM = 3,  /* a device or host allocation failed */
  LDA_E_DEVICE = 4, /* a HIP runtime call or kernel failed */
  LDA_E_STATE = 5   /* the handle was poisoned by an earlier device error */
} lda_status;

/* Largest topic count (the paper's largest, Sec. 6): the packed
 * (topic << 16 | count) entries of D and of the sparse rows of W (Sec. 4.2)
 * keep 16 bits per field, and one topic code marks an undrawn token.  Above
 * about 17,000 topics the fp64 word-topic row no longer fits one
 * workgroup's LDS, and the sampler walks it in two tiles. */
#define LDA_MAX_TOPICS 32768
/* Longest document: its per-topic counts must fit 16 bits (Sec. 4.2). */
#define LDA_MAX_DOC_LEN 65535
/* Most chunks of an out-of-core corpus (lda_options.chunks). */
#define LDA_MAX_CHUNKS 256

typedef struct {
  /* hipStream_t to run on; NULL = the handle creates its own stream. */
  void *stream;
  /* Device allocator (for example a caching allocator).  NULL = hipMalloc /
   * hipFree.  dev_free may be NULL only if dev_alloc is NULL. */
  void *(*dev_alloc)(size_t bytes, void *ctx);
  void (*dev_free)(void *ptr, void *ctx);
  void *alloc_ctx;
  /* Depth g of the S_est bound, Eq. 9: 1, 2 or 3 (0 = default 2, Sec. 3.2
   * "Parameter tuning").  Changes which tokens skip the S' scan, never the draw. */
  int32_t g;
  /* Large-word split: tokens per region, Sec. 5.1 (0 = default 10,000). */
  int32_t region_tokens;
  /* Disable the step-3 skip test (every token scans its D row).  Ablation
   * switch; the draws are unchanged. */
  int32_t no_skip;
  /* Hybrid W cutoff, Sec. 4.2: a word is dense when its token count exceeds
   * this (0 = default K; negative = every word dense).  Words with more than
   * 65,535 tokens are always dense (16-bit sparse counts).  Ablation switch;
   * the draws are unchanged. */
  int32_t dense_cutoff;
  /* Two-branch sampling, Sec. 2.2: draw over [S | Q] with no max-topic branch
   * and no skip test (the ablation of Eq. 5).  Same distribution, different
   * canonical order, so different draws for the same u. */
  int32_t two_branch;
  /* Threads per sampler workgroup: 256, 512 or 1024 (0 = the size with the
   * most resident waves per CU for this K; the W^ row of K fp64 values in LDS
   * limits how many workgroups a CU holds).  LDA_E_RANGE if the size asked
   * for does not fit.  Performance switch; the draws are unchanged. */
  int32_t sampler_block;
  /* How the step-3 skip decisions reach the sampler (Sec. 3.3): 0 = chosen
   * per iteration from the previous iteration's skip rate (default); 1 =
   * always a bitmap in word order (one scattered bit per skipped token); 2 =
   * a bitmap in document order (coalesced bits, read by the sampler at each
   * token's key) whenever the input is sorted by document and K fits the
   * regular sampler, else as 1.  Performance switch; the draws are unchanged. */
  int32_t skip_marks;
  /* Steps 2-3 (the per-document C1/C2 pass and the skip test, Sec. 3.3)
   * only save work, and they cost about as much as the sampler work of a
   * tenth of the tokens.  0 (default): they run in every eighth iteration,
   * which measures the skip rate, and in every iteration after one that
   * skipped at least an eighth of the tokens; 1: every iteration.
   * Performance switch; the draws are unchanged (a token not skipped is
   * drawn in full). */
  int32_t always_skip_test;
  /* Out-of-core corpus (Sec. 4.1 and 4.3): 0 or 1 = every per-token array
   * resident on the device (default); C in [2, LDA_MAX_CHUNKS] = the
   * documents are cut into C chunks of near-equal token counts whose
   * per-token arrays (6 bytes a token) live in pinned host memory and stream
   * through two device buffers every iteration, transfers overlapping the
   * previous chunk's work.  W is then dense for every word and kept twice
   * (the snapshot and the next counts), so the draws equal the resident
   * path's.  Needs input sorted by document (LDA_E_ARG otherwise); the
   * per-stage times of lda_iter_stats are 0 (ms_iter is kept). */
  int32_t chunks;
} lda_options;

/* Per-iteration statistics (filled by lda_iterate when requested). */
typedef struct {
  int64_t iteration;     /* t of this iteration */
  double ms_iter;        /* device time of the whole iteration (HIP events) */
  double ms_sampler;     /* device time of the word-major sampler kernel */
  double ms_docpass;     /* device time of the per-document C1/C2 + skip kernel */
  double ms_rebuild;     /* device time of the count rebuild kernels */
  double ms_precompute;  /* device time of the per-topic and per-word precompute */
  int64_t skip_step3;    /* tokens set to K1 by the step-3 test */
  int64_t skip_after_s;  /* tokens drawn as K1 by the second max-topic test */
  int64_t sampled;       /* tokens whose S' was built (not skipped at step 3) */
  int64_t nnz_scanned;   /* D-row entries the sampler read: nnz(D[d]) per sampled token, except one chunk
                          * (at most 128) for a later token of a run of one word in one document whose row
                          * is longer than 511 entries (it draws from the run's first token's sums) */
  int64_t regions;       /* regions handed out by the scheduler */
  int64_t dense_regions; /* of which regions of dense (full-row) words */
  int64_t row_bytes;     /* bytes of W rows the sampler needs: 4*K per dense word, 4*nnz per sparse word */
  int64_t sampler_block; /* threads per sampler workgroup */
  int64_t skip_marks;    /* how step-3 decisions reached the sampler: 1 word-ordered bitmap, 2 document-ordered */
  int64_t skip_test_ran; /* 1 if steps 2-3 ran in this iteration (see always_skip_test), else 0 */
} lda_iter_stats;

/* Count tables in the caller's ids.  Caller-allocated; a call with every array
 * pointer NULL is a size query that fills iteration, M, V, K, n_tokens, nnz_D
 * and nnz_W only. */
typedef struct {
  int64_t iteration; /* completed synchronous iterations */
  int32_t M, V, K;   /* documents (max doc id + 1), vocabulary, topics */
  int64_t n_tokens;
  int64_t nnz_D, nnz_W;
  int32_t *z;        /* [n_tokens] topic of each token, input order */
  int64_t *T;        /* [K] tokens per topic */
  int64_t *D_off;    /* [M+1] CSR offsets of D by doc id */
  int32_t *D_topic;  /* [nnz_D] topics ascending within a doc */
  int32_t *D_count;  /* [nnz_D] */
  int64_t *W_off;    /* [V+1] CSR offsets of W by (caller's) word id */
  int32_t *W_topic;  /* [nnz_W] topics ascending within a word */
  int32_t *W_count;  /* [nnz_W] */
} lda_counts;

/*
 * Build a sampler for the token list <word[i], doc[i]>, i < n_tokens
 * (the token list of Sec. 1), with V words, K topics and priors alpha, beta
 * (Eq. 1; the paper's defaults are alpha = 50/K and beta = 0.01).
 *   word, doc: host arrays of n_tokens ids, any order; word in [0, V),
 *              doc >= 0; M = max doc id + 1 and empty documents are allowed.
 *   seed:      Philox key; the initial topics are drawn from it.
 *   opts:      may be NULL.
 *   out:       receives the handle; stays NULL on failure (nothing leaks).
 * Errors: LDA_E_ARG (NULL pointers, n_tokens <= 0, V <= 0, K < 2,
 * K > LDA_MAX_TOPICS, alpha or beta not finite and > 0, an id out of range,
 * bad options), LDA_E_RANGE (a document longer than LDA_MAX_DOC_LEN, or
 * n_tokens >= 2^32), LDA_E_NOMEM, LDA_E_DEVICE.
 */
lda_status lda_create(const int32_t *word, const int32_t *doc, int64_t n_tokens, int32_t V, int32_t K, double alpha,
                      double beta, uint64_t seed, const lda_options *opts, lda_handle **out);

/*
 * Run n_iters synchronous iterations (sampling then update, Sec. 2.2 and
 * Sec. 4.3).  stats may be NULL, else it points to n_iters records.  One
 * stream synchronisation per call.
 */
lda_status lda_iterate(lda_handle *h, int32_t n_iters, lda_iter_stats *stats);

/* Copy the current assignment and the count tables of Sec. 2.2 to caller
 * memory (see lda_counts): D[d][k] = tokens of document d with topic k, W[v][k]
 * = tokens of word v with topic k, T[k] = sum_v W[v][k]. */
lda_status lda_get_counts(lda_handle *h, lda_counts *out);

/*
 * Log-likelihood per token of the current state, log base 2 (Sec. 2.2,
 * "Evaluation metric"):
 *   (1/N) sum_n log2 sum_k (D[d][k]+alpha)/(len(d)+K*alpha) * (W[v][k]+beta)/(T[k]+V*beta)
 */
lda_status lda_loglik(lda_handle *h, double *llpt);

/*
 * Replace the assignment (input order, values in [0, K)) and the iteration
 * counter, then rebuild D, W and T.  For checkpoint/resume and for tests that
 * start the GPU from a given snapshot.
 */
lda_status lda_set_assignments(lda_handle *h, const int32_t *z, int64_t iteration);

/*
 * lda_loglik for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * computation and the same result, bit for bit, as lda_loglik; its scratch
 * (the per-region partial sums, the scheduler counter and the result) lives in
 * a fixed device array of the library instead of handle memory, so the call
 * itself allocates nothing (no hipMalloc, hipFree or allocating library
 * routine).  The array holds 4 KiB plus 8 B per region (of the largest
 * chunk, with lda_options.chunks), up to LDA_NOALLOC_MAX_REGIONS regions
 * (16 MiB); each device the library runs on keeps its own copy until the
 * process ends.
 *   llpt: host pointer to one double (output).
 * Errors: LDA_E_ARG (llpt NULL), LDA_E_RANGE (the handle's layout has more
 * than LDA_NOALLOC_MAX_REGIONS regions), LDA_E_DEVICE, LDA_E_STATE.
 * Every call on one device shares that device's array, whichever handle makes
 * it: calls that overlap in time on one GPU (other host threads, other
 * streams) race and must be serialised by the caller.
 */
#define LDA_NOALLOC_MAX_REGIONS (1 << 21)
lda_status lda_loglik_noalloc(lda_handle *h, double *llpt);

/* Release every resource of the handle.  NULL is allowed. */
void lda_destroy(lda_handle *h);

/* Message for the last failure on h (or on the last failed lda_create when h
 * is NULL).  Never NULL. */
const char *lda_last_error(const lda_handle *h);

/*
 * Layout description (host only; touches no device).  Relabels words by
 * descending token count (ties by ascending id), marks a word dense when its
 * count exceeds the cutoff (dense_cutoff as in lda_options: 0 = K, Sec. 4.2),
 * and cuts every dense word into regions of at most region_tokens
 * consecutive word-ordered tokens (Sec. 5.1).  Arrays may be NULL; sizes
 * first via the scalar outputs.
 *   relabel[V]      new id of each caller word id (absent words last)
 *   n_present, n_dense, n_regions, n_docs: scalar outputs
 *   word_off[n_present+1]  word-ordered offsets per new id
 *   wt_key[n_tokens]       input index of each word-ordered token
 *   region[3*n_regions]    (new word id, begin, end) per region
 */
lda_status lda_describe_layout(const int32_t *word, const int32_t *doc, int64_t n_tokens, int32_t V, int32_t K,
                               int32_t region_tokens, int32_t dense_cutoff, int32_t *relabel, int32_t *n_present,
                               int32_t *n_dense,
                               int64_t *n_regions, int32_t *n_docs, uint32_t *word_off, uint32_t *wt_key,
                               uint32_t *region);

#ifdef __cplusplus
}
#endif
#endif
