/*
 * LDA oracle: plain, slow, single-threaded CPU reference of one synchronous
 * collapsed-Gibbs (ESCA) iteration with the three-branch decomposition.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load or call this code.  It shares no code
 * with the GPU library and must never serve as a fallback for it.
 *
 * Conventions (all arrays are caller-owned host memory):
 *   n          number of tokens, token i = (word[i], doc[i]) in input order
 *   M, V, K    documents (max doc id + 1), vocabulary size, topics
 *   z          topic per token in input order, 0 <= z < K
 *   counts     D[d][k] (CSR, topics ascending), W[v][k] dense int32, T[k] int64
 * Floating point is IEEE fp64 with no contraction (built -ffp-contract=off).
 */
#ifndef LDA_ORACLE_H
#define LDA_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Philox4x32-10 (Salmon et al., SC'11): 10 rounds of the 4x32 Philox
 * bijection keyed by key[2], applied to the 128-bit counter ctr[4]. */
void ora_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* Uniform draw for token i at iteration t:
 * x = Philox(ctr = (i_lo, i_hi, t, 0), key = (seed_lo, seed_hi)),
 * u = (((x0 << 32) | x1) >> 11) * 2^-53  in [0, 1). */
double ora_uniform(uint64_t seed, uint32_t t, uint64_t i);

/* Initial topic of token i: x = Philox(ctr = (i_lo, i_hi, 0, 1), key = seed),
 * z0 = (x0 * K) >> 32. */
int32_t ora_init_topic(uint64_t seed, uint64_t i, int32_t K);
void ora_init(int64_t n, int32_t K, uint64_t seed, int32_t *z);

/* Count tables from an assignment (Sec. 2.2: D, W and the column sums of W).
 * len[M], doff[M+1], dtop/dcnt (capacity n), W[V*K], T[K]. Returns 0 or an
 * error code (1 bad argument). */
int ora_build_counts(int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V,
                     int32_t K, int64_t *len, int64_t *doff, int32_t *dtop, int32_t *dcnt, int32_t *W, int64_t *T);

/* stats[] slots filled by ora_iterate */
enum {
  ORA_ST_FLAGGED = 0,       /* draws within 1e-9*Z of a CDF edge */
  ORA_ST_SKIP3 = 1,         /* tokens whose step-3 test fires */
  ORA_ST_SEST_VIOL = 2,     /* tokens with S' > S_est*(1+1e-12): must be 0 */
  ORA_ST_SKIP_NOT_K1 = 3,   /* skip fired but the draw is not K1 (unflagged): must be 0 */
  ORA_ST_FALLBACK = 4,      /* x >= Z after rounding: last positive segment */
  ORA_ST_SKIP_AFTER_S = 5,  /* second max-topic test (x < M) fires */
  ORA_ST_NNZ_SCANNED = 6,   /* sum of nnz(D[d]) over tokens not skipped at step 3 */
  ORA_N_STATS = 8
};

/* One synchronous iteration from the snapshot of counts built from z_in.
 *   mode bit 0: 0 = sparse decomposition (scans nz(D[d]), per-word Q' running
 *               sum), 1 = dense brute force (all K topics per token)
 *   mode bit 1: 0 = three-branch canonical order [K1 | S' | Q'] (Eq. 5),
 *               1 = two-branch order [S | Q] of Sec. 2.2 (no max-topic
 *               branch, no skip statistics; the ablation)
 *   g      = depth of the S_est bound used for the skip statistics (1, 2 or 3)
 * If idx is NULL every token i in 0..n-1 is drawn into z_out[i]; otherwise
 * only tokens idx[0..n_sub-1], written to z_out[j], flags[j], Zout[j].
 * flags bit0 = near-boundary draw, bit1 = step-3 skip fired.
 * Zout (nullable) receives the normaliser Z of each drawn token. */
int ora_iterate(int mode, int g, int64_t n, const int32_t *word, const int32_t *doc, int32_t M, int32_t V, int32_t K,
                double alpha, double beta, uint64_t seed, uint32_t t, const int32_t *z_in, int64_t n_sub,
                const int64_t *idx, int32_t *z_out, uint8_t *flags, double *Zout, int64_t *stats);

/* Log-likelihood per token, log base 2, on the counts built from z.
 * mode 0 = sparse form, mode 1 = dense sum over all K topics. */
double ora_llpt(int mode, int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V,
                int32_t K, double alpha, double beta);

/* Per-word quantities of the three-branch method for the counts built from z:
 * K1, K2 (top-2 topic ids, lowest id on ties), a1 >= a2 >= a3 (top-3 values of
 * W^[v]), Qp = sum_{k != K1} alpha*W^[v][k] (ascending running sum). */
int ora_word_stats(int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V,
                   int32_t K, double alpha, double beta, int32_t *K1, int32_t *K2, double *a1, double *a2, double *a3,
                   double *Qp);

/* The third top topic K3 (lowest id among the maxima over k not in {K1, K2};
 * -1 if K < 3) and the fourth top value a4 of W^[v] (0 if K < 4): what the
 * S_est of Eq. 9 uses at depth g = 3. */
int ora_word_top4(int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V,
                  int32_t K, double alpha, double beta, int32_t *K3, double *a4);

/* Draw token i of the snapshot built from z with a given u in [0,1) (test
 * hook for worked examples and exact enumeration).  Returns the topic, or -1
 * on a bad argument; Z and flag as in ora_iterate. */
int32_t ora_draw_given_u(int mode, int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M,
                         int32_t V, int32_t K, double alpha, double beta, int64_t i, double u, double *Z,
                         uint8_t *flag);

/* The normalised word row W^[v][k] = (W[v][k]+beta)/(T[k]+V*beta), Eq. 2. */
int ora_what_row(int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V, int32_t K,
                 double beta, int32_t v, double *out);

/* A counts snapshot kept across calls, so that a caller can draw disjoint
 * token ranges of one iteration from several threads (the draws depend only
 * on (seed, t, i) and the snapshot, so the result does not depend on how the
 * tokens are split).  The code itself is single-threaded and the snapshot is
 * read-only after ora_snapshot_new.
 *   idx == NULL: counts of every word and document (as ora_iterate builds).
 *   idx != NULL: T over every token, but W and D rows only for the words and
 *                documents of tokens idx[0..n_idx): enough to draw exactly
 *                those tokens, in one pass over the corpus.
 *   with_words:  also the per-word quantities (needed by the sparse form and
 *                the LLPT).
 * The word/doc arrays are borrowed and must outlive the snapshot; z is read
 * only during ora_snapshot_new.  Returns 0, 1 (bad argument) or 2 (no memory). */
typedef struct ora_snapshot ora_snapshot;
int ora_snapshot_new(int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V,
                     int32_t K, double alpha, double beta, int with_words, int64_t n_idx, const int64_t *idx,
                     ora_snapshot **out);
/* Draw tokens idx[0..cnt) (idx NULL: tokens first..first+cnt-1) as
 * ora_iterate does; outputs and stats as there, outputs at [0, cnt).
 * Returns 1 for a token the snapshot does not hold. */
int ora_snapshot_draw(const ora_snapshot *s, int mode, int g, uint64_t seed, uint32_t t, int64_t first, int64_t cnt,
                      const int64_t *idx, int32_t *z_out, uint8_t *flags, double *Zout, int64_t *stats);
/* Neumaier-compensated sum (and its compensation) of the LLPT terms of
 * tokens first..first+cnt-1 (sparse form, full snapshot with words). */
int ora_snapshot_llpt(const ora_snapshot *s, int64_t first, int64_t cnt, double *sum, double *comp);
void ora_snapshot_free(ora_snapshot *s);

/* Initial topics of tokens first..first+cnt-1 into z[0..cnt). */
void ora_init_range(int64_t first, int64_t cnt, int32_t K, uint64_t seed, int32_t *z);

#ifdef __cplusplus
}
#endif
#endif
