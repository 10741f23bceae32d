/*
 * LDA oracle: plain single-threaded CPU reference (see lda_oracle.h).
 *
 * TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the
 * benchmark's CPU-baseline leg; never by the GPU library.
 *
 * What it computes, and where the paper defines it (arXiv 2007.08725):
 *   - the ESCA conditional p(k) ~ (D[d][k]+alpha) * W^[v][k],
 *     W^[v][k] = (W[v][k]+beta) / (sum_v W[v][k] + V*beta)      Sec. 2.2, Eq. 1-2
 *     Counts include the token being drawn (no -i exclusion) and are a snapshot
 *     taken at the start of the iteration (synchronous update, Sec. 4.3).
 *   - the three-branch split p = D o W^' + alpha o W^' + (D+alpha) o W^m   Sec. 3.2, Eq. 5
 *     drawn by one forward inverse CDF x = u*Z over the segments
 *       [ K1 | S' terms, topics ascending | Q' terms, topics ascending ]
 *     with a strict "x < running sum" test.  Since Eq. 5 re-splits Eq. 1
 *     exactly, this is a draw from Eq. 1.
 *   - the S_est bound and the step-3 skip test                   Sec. 3.2, Eq. 6-9
 *     (recorded as statistics; it never changes the draw)
 *   - LLPT, log base 2, per token                                 Sec. 2.2, "Evaluation metric"
 * Random numbers come from Philox4x32-10 (Salmon, Moraes, Dror, Shaw:
 * "Parallel Random Numbers: As Easy as 1, 2, 3", SC'11), keyed by the seed and
 * counted by (token index, iteration, domain); the paper only says u ~ U[0,1].
 */
#include "lda_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------ Philox ---- */
/* Round multipliers and Weyl key increments of Philox4x32 (SC'11, Sec. 5). */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void ora_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  uint32_t k0 = key[0], k1 = key[1];
  for (int round = 0; round < 10; round++) {
    uint64_t p0 = (uint64_t)PHILOX_M0 * (uint64_t)x0;
    uint64_t p1 = (uint64_t)PHILOX_M1 * (uint64_t)x2;
    uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
    uint32_t y1 = (uint32_t)p1;
    uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
    uint32_t y3 = (uint32_t)p0;
    x0 = y0;
    x1 = y1;
    x2 = y2;
    x3 = y3;
    k0 += PHILOX_W0;
    k1 += PHILOX_W1;
  }
  out[0] = x0;
  out[1] = x1;
  out[2] = x2;
  out[3] = x3;
}

double ora_uniform(uint64_t seed, uint32_t t, uint64_t i) {
  uint32_t ctr[4] = {(uint32_t)i, (uint32_t)(i >> 32), t, 0u};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t x[4];
  ora_philox4x32_10(ctr, key, x);
  uint64_t bits = ((uint64_t)x[0] << 32) | (uint64_t)x[1];
  return (double)(bits >> 11) * (1.0 / 9007199254740992.0); /* 2^-53 */
}

int32_t ora_init_topic(uint64_t seed, uint64_t i, int32_t K) {
  uint32_t ctr[4] = {(uint32_t)i, (uint32_t)(i >> 32), 0u, 1u};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  uint32_t x[4];
  ora_philox4x32_10(ctr, key, x);
  return (int32_t)(((uint64_t)x[0] * (uint64_t)K) >> 32);
}

void ora_init(int64_t n, int32_t K, uint64_t seed, int32_t *z) {
  for (int64_t i = 0; i < n; i++) z[i] = ora_init_topic(seed, (uint64_t)i, K);
}

/* ------------------------------------------------------------ counts ---- */

static int cmp_i32(const void *a, const void *b) {
  int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
  return (x > y) - (x < y);
}

int ora_build_counts(int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V,
                     int32_t K, int64_t *len, int64_t *doff, int32_t *dtop, int32_t *dcnt, int32_t *W, int64_t *T) {
  if (n < 0 || M < 0 || V <= 0 || K <= 0) return 1;
  for (int64_t i = 0; i < n; i++)
    if (word[i] < 0 || word[i] >= V || doc[i] < 0 || doc[i] >= M || z[i] < 0 || z[i] >= K) return 1;
  memset(len, 0, sizeof(int64_t) * (size_t)M);
  memset(W, 0, sizeof(int32_t) * (size_t)V * (size_t)K);
  memset(T, 0, sizeof(int64_t) * (size_t)K);
  for (int64_t i = 0; i < n; i++) {
    len[doc[i]]++;
    W[(size_t)word[i] * (size_t)K + (size_t)z[i]]++;
    T[z[i]]++;
  }
  /* D rows: gather each document's topics, sort them, run-length encode. */
  int64_t *pos = malloc(sizeof(int64_t) * ((size_t)M + 1));
  int32_t *zt = malloc(sizeof(int32_t) * (size_t)(n > 0 ? n : 1));
  if (!pos || !zt) {
    free(pos);
    free(zt);
    return 2;
  }
  pos[0] = 0;
  for (int32_t d = 0; d < M; d++) pos[d + 1] = pos[d] + len[d];
  for (int64_t i = 0; i < n; i++) zt[pos[doc[i]]++] = z[i];
  int64_t nnz = 0, b = 0;
  for (int32_t d = 0; d < M; d++) {
    int64_t e = b + len[d];
    qsort(zt + b, (size_t)(e - b), sizeof(int32_t), cmp_i32);
    doff[d] = nnz;
    for (int64_t j = b; j < e; j++) {
      if (j == b || zt[j] != zt[j - 1]) {
        dtop[nnz] = zt[j];
        dcnt[nnz] = 0;
        nnz++;
      }
      dcnt[nnz - 1]++;
    }
    b = e;
  }
  doff[M] = nnz;
  free(pos);
  free(zt);
  return 0;
}

/* ------------------------------------------------------- snapshot ctx ---- */

typedef struct ora_snapshot {
  int64_t n;
  const int32_t *word, *doc;
  int32_t M, V, K;
  double alpha, beta;
  /* Rows held: a full snapshot holds every word (row v) and document (row d);
   * a restricted one only those of a token sample, at rows wslot[v] and
   * dslot[d] (-1 = not held).  The counts of the rows it holds are the same. */
  int32_t *wslot, *dslot;
  int32_t nW, nD;
  /* counts snapshot, by row */
  int64_t *len, *doff;
  int32_t *dtop, *dcnt, *W;
  int64_t *T;
  double *den; /* den[k] = T[k] + V*beta */
  /* per-word quantities (sparse form), by row */
  int32_t *K1, *K2, *K3;
  double *a1, *a2, *a3, *a4, *Qp, *Qall, *sumWh;
} snap;

/* Row of word v and of document d in the snapshot (v and d themselves in a
 * full snapshot). */
static inline int64_t wrow(const snap *s, int32_t v) { return s->wslot ? (int64_t)s->wslot[v] : (int64_t)v; }
static inline int64_t drow(const snap *s, int32_t d) { return s->dslot ? (int64_t)s->dslot[d] : (int64_t)d; }

static void snap_free(snap *s) {
  free(s->wslot);
  free(s->dslot);
  free(s->len);
  free(s->doff);
  free(s->dtop);
  free(s->dcnt);
  free(s->W);
  free(s->T);
  free(s->den);
  free(s->K1);
  free(s->K2);
  free(s->K3);
  free(s->a1);
  free(s->a2);
  free(s->a3);
  free(s->a4);
  free(s->Qp);
  free(s->Qall);
  free(s->sumWh);
  memset(s, 0, sizeof(*s));
}

/* W^[v][k], Eq. 1-2, for the word held at row wr: an IEEE fp64 divide (the
 * argmax below depends on it). */
static inline double what(const snap *s, int64_t wr, int32_t k) {
  return ((double)s->W[(size_t)wr * (size_t)s->K + (size_t)k] + s->beta) / s->den[k];
}

static void snap_init(snap *s, int64_t n, const int32_t *word, const int32_t *doc, int32_t M, int32_t V,
                      int32_t K, double alpha, double beta) {
  memset(s, 0, sizeof(*s));
  s->n = n;
  s->word = word;
  s->doc = doc;
  s->M = M;
  s->V = V;
  s->K = K;
  s->alpha = alpha;
  s->beta = beta;
}

/* Counts of every word and document. */
static int snap_counts_full(snap *s, const int32_t *z) {
  const int64_t n = s->n;
  const int32_t M = s->M, V = s->V, K = s->K;
  size_t nn = (size_t)(n > 0 ? n : 1);
  s->nW = V;
  s->nD = M;
  s->len = malloc(sizeof(int64_t) * (size_t)(M > 0 ? M : 1));
  s->doff = malloc(sizeof(int64_t) * ((size_t)M + 1));
  s->dtop = malloc(sizeof(int32_t) * nn);
  s->dcnt = malloc(sizeof(int32_t) * nn);
  s->W = malloc(sizeof(int32_t) * (size_t)V * (size_t)K);
  s->T = malloc(sizeof(int64_t) * (size_t)K);
  if (!s->len || !s->doff || !s->dtop || !s->dcnt || !s->W || !s->T) return 2;
  return ora_build_counts(n, s->word, s->doc, z, M, V, K, s->len, s->doff, s->dtop, s->dcnt, s->W, s->T);
}

/* Counts of the words and documents of tokens idx[0..n_idx) only: T over
 * every token, W rows of those words, D rows of those documents (the same
 * definitions as ora_build_counts, restricted to the rows a sample of draws
 * reads). */
static int snap_counts_sub(snap *s, const int32_t *z, int64_t n_idx, const int64_t *idx) {
  const int64_t n = s->n;
  const int32_t M = s->M, V = s->V, K = s->K;
  const int32_t *word = s->word, *doc = s->doc;
  s->wslot = malloc(sizeof(int32_t) * (size_t)V);
  s->dslot = malloc(sizeof(int32_t) * (size_t)(M > 0 ? M : 1));
  if (!s->wslot || !s->dslot) return 2;
  for (int32_t v = 0; v < V; v++) s->wslot[v] = -1;
  for (int32_t d = 0; d < M; d++) s->dslot[d] = -1;
  for (int64_t j = 0; j < n_idx; j++) {
    const int64_t i = idx[j];
    if (i < 0 || i >= n || word[i] < 0 || word[i] >= V || doc[i] < 0 || doc[i] >= M) return 1;
    if (s->wslot[word[i]] < 0) s->wslot[word[i]] = s->nW++;
    if (s->dslot[doc[i]] < 0) s->dslot[doc[i]] = s->nD++;
  }
  s->W = calloc((size_t)(s->nW > 0 ? s->nW : 1) * (size_t)K, sizeof(int32_t));
  s->T = calloc((size_t)K, sizeof(int64_t));
  s->len = calloc((size_t)(s->nD > 0 ? s->nD : 1), sizeof(int64_t));
  s->doff = malloc(sizeof(int64_t) * ((size_t)s->nD + 1));
  if (!s->W || !s->T || !s->len || !s->doff) return 2;
  /* pass 1: T, the held W rows and the held documents' lengths */
  for (int64_t i = 0; i < n; i++) {
    if (word[i] < 0 || word[i] >= V || doc[i] < 0 || doc[i] >= M || z[i] < 0 || z[i] >= K) return 1;
    s->T[z[i]]++;
    const int32_t wr = s->wslot[word[i]], dr = s->dslot[doc[i]];
    if (wr >= 0) s->W[(size_t)wr * (size_t)K + (size_t)z[i]]++;
    if (dr >= 0) s->len[dr]++;
  }
  /* pass 2: the held documents' topics, then each row sorted and run-length encoded */
  int64_t *pos = malloc(sizeof(int64_t) * ((size_t)s->nD + 1));
  if (!pos) return 2;
  pos[0] = 0;
  for (int32_t r = 0; r < s->nD; r++) pos[r + 1] = pos[r] + s->len[r];
  const int64_t tot = pos[s->nD];
  int32_t *zt = malloc(sizeof(int32_t) * (size_t)(tot > 0 ? tot : 1));
  s->dtop = malloc(sizeof(int32_t) * (size_t)(tot > 0 ? tot : 1));
  s->dcnt = malloc(sizeof(int32_t) * (size_t)(tot > 0 ? tot : 1));
  if (!zt || !s->dtop || !s->dcnt) {
    free(pos);
    free(zt);
    return 2;
  }
  for (int64_t i = 0; i < n; i++) {
    const int32_t dr = s->dslot[doc[i]];
    if (dr >= 0) zt[pos[dr]++] = z[i];
  }
  int64_t nnz = 0, b = 0;
  for (int32_t r = 0; r < s->nD; r++) {
    const int64_t e = b + s->len[r];
    qsort(zt + b, (size_t)(e - b), sizeof(int32_t), cmp_i32);
    s->doff[r] = nnz;
    for (int64_t j = b; j < e; j++) {
      if (j == b || zt[j] != zt[j - 1]) {
        s->dtop[nnz] = zt[j];
        s->dcnt[nnz] = 0;
        nnz++;
      }
      s->dcnt[nnz - 1]++;
    }
    b = e;
  }
  s->doff[s->nD] = nnz;
  free(pos);
  free(zt);
  return 0;
}

/* den[k] and, with with_words, the per-word quantities of every held word. */
static int snap_finish(snap *s, int with_words) {
  const int32_t K = s->K;
  const double alpha = s->alpha;
  s->den = malloc(sizeof(double) * (size_t)K);
  if (!s->den) return 2;
  const double Vbeta = (double)s->V * s->beta;
  for (int32_t k = 0; k < K; k++) s->den[k] = (double)s->T[k] + Vbeta;
  if (!with_words) return 0;
  const size_t nw = (size_t)(s->nW > 0 ? s->nW : 1);
  s->K1 = malloc(sizeof(int32_t) * nw);
  s->K2 = malloc(sizeof(int32_t) * nw);
  s->K3 = malloc(sizeof(int32_t) * nw);
  s->a1 = malloc(sizeof(double) * nw);
  s->a2 = malloc(sizeof(double) * nw);
  s->a3 = malloc(sizeof(double) * nw);
  s->a4 = malloc(sizeof(double) * nw);
  s->Qp = malloc(sizeof(double) * nw);
  s->Qall = malloc(sizeof(double) * nw);
  s->sumWh = malloc(sizeof(double) * nw);
  if (!s->K1 || !s->K2 || !s->K3 || !s->a1 || !s->a2 || !s->a3 || !s->a4 || !s->Qp || !s->Qall || !s->sumWh)
    return 2;
  for (int32_t v = 0; v < s->nW; v++) {
    /* step 1 of the three-branch procedure: top topics of W^[v] (Sec. 3.2).
     * K1 = lowest topic id among the maxima; K2 = lowest id among the maxima
     * over k != K1; K3 = lowest id among the maxima over k not in {K1, K2}
     * (-1 if K < 3), a3 its value (0 if K < 3); a4 = largest value over k not
     * in {K1, K2, K3} (0 if K < 4).  a1 >= a2 >= a3 >= a4 feed the S_est of
     * Eq. 9 for g = 1, 2, 3. */
    int32_t k1 = 0;
    double m1 = what(s, v, 0);
    for (int32_t k = 1; k < K; k++) {
      double w = what(s, v, k);
      if (w > m1) {
        m1 = w;
        k1 = k;
      }
    }
    int32_t k2 = -1;
    double m2 = 0.0;
    for (int32_t k = 0; k < K; k++) {
      if (k == k1) continue;
      double w = what(s, v, k);
      if (k2 < 0 || w > m2) {
        m2 = w;
        k2 = k;
      }
    }
    int32_t k3 = -1;
    double m3 = 0.0;
    for (int32_t k = 0; k < K; k++) {
      if (k == k1 || k == k2) continue;
      double w = what(s, v, k);
      if (k3 < 0 || w > m3) {
        m3 = w;
        k3 = k;
      }
    }
    double m4 = 0.0;
    int have4 = 0;
    for (int32_t k = 0; k < K; k++) {
      if (k == k1 || k == k2 || k == k3) continue;
      double w = what(s, v, k);
      if (!have4 || w > m4) {
        m4 = w;
        have4 = 1;
      }
    }
    /* Q' = sum over k != K1 of alpha*W^[v][k], ascending (Eq. 5, p_q); the
     * two-branch Q sums every k (Sec. 2.2). */
    double q = 0.0, qa = 0.0, sw = 0.0;
    for (int32_t k = 0; k < K; k++) {
      double w = what(s, v, k);
      sw += w;
      qa += alpha * w;
      if (k != k1) q += alpha * w;
    }
    s->K1[v] = k1;
    s->K2[v] = k2;
    s->K3[v] = k3;
    s->a1[v] = m1;
    s->a2[v] = m2;
    s->a3[v] = m3;
    s->a4[v] = m4;
    s->Qp[v] = q;
    s->Qall[v] = qa;
    s->sumWh[v] = sw;
  }
  return 0;
}

static int snap_build(snap *s, int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M,
                      int32_t V, int32_t K, double alpha, double beta, int with_words) {
  snap_init(s, n, word, doc, M, V, K, alpha, beta);
  int rc = snap_counts_full(s, z);
  if (!rc) rc = snap_finish(s, with_words);
  if (rc) snap_free(s);
  return rc;
}

/* Count of topic k in the document held at row dr (0 if absent). */
static int32_t dcount(const snap *s, int64_t dr, int32_t k) {
  for (int64_t e = s->doff[dr]; e < s->doff[dr + 1]; e++)
    if (s->dtop[e] == k) return s->dcnt[e];
  return 0;
}

static const double BOUNDARY_REL = 1e-9;

/* S_est of Eq. 9 for the depth g used by the statistics (g = 1, 2 or 3):
 * the counts of the top topics K2..Kg times their values, and all other
 * tokens of the document times the next value a_{g+1}. */
static double s_est(int g, double a2, double a3, double a4, int32_t C1, int32_t C2, int32_t C3, int64_t len) {
  if (g <= 1) return a2 * (double)(len - C1);
  if (g == 2) return a2 * (double)C2 + a3 * (double)(len - C1 - C2);
  return a2 * (double)C2 + a3 * (double)C3 + a4 * (double)(len - C1 - C2 - C3);
}

/* ------------------------------------------------------- sparse draw ---- */

static int32_t draw_sparse(const snap *s, int g, double u, int64_t i, double *Zo, uint8_t *flag, int64_t *st) {
  const int64_t v = wrow(s, s->word[i]), d = drow(s, s->doc[i]);
  const int32_t K = s->K;
  const double alpha = s->alpha;
  const int32_t K1 = s->K1[v];
  const double a1 = s->a1[v];
  const int64_t b = s->doff[d], e = s->doff[d + 1];
  const int32_t C1 = dcount(s, d, K1), C2 = dcount(s, d, s->K2[v]);
  const int32_t C3 = s->K3[v] >= 0 ? dcount(s, d, s->K3[v]) : 0;

  /* max-topic branch, Eq. 7 */
  const double Mm = a1 * ((double)C1 + alpha);
  /* S' running sum over nz(D[d]) \ {K1}, ascending topics, starting at M */
  double c = Mm, sprime = 0.0;
  for (int64_t j = b; j < e; j++) {
    if (s->dtop[j] == K1) continue;
    double term = (double)s->dcnt[j] * what(s, v, s->dtop[j]);
    c += term;
    sprime += term;
  }
  const double S_end = c;
  const double Z = S_end + s->Qp[v];
  const double x = u * Z;

  /* step-3 statistics: S' <= S_est (Eq. 8-9) and the skip test */
  const double Sest = s_est(g, s->a2[v], s->a3[v], s->a4[v], C1, C2, C3, s->len[d]);
  if (sprime > Sest * (1.0 + 1e-12)) st[ORA_ST_SEST_VIOL]++;
  const int skip3 = u * (Mm + Sest + s->Qp[v]) < Mm;
  if (skip3) st[ORA_ST_SKIP3]++;
  else st[ORA_ST_NNZ_SCANNED] += e - b;

  int32_t pick = -1;
  double lo = 0.0, hi = 0.0;
  if (x < Mm) {
    pick = K1;
    lo = 0.0;
    hi = Mm;
    if (!skip3) st[ORA_ST_SKIP_AFTER_S]++;
  } else {
    double prev = Mm;
    for (int64_t j = b; j < e && pick < 0; j++) {
      if (s->dtop[j] == K1) continue;
      double cur = prev + (double)s->dcnt[j] * what(s, v, s->dtop[j]);
      if (x < cur) {
        pick = s->dtop[j];
        lo = prev;
        hi = cur;
      }
      prev = cur;
    }
  }
  if (pick < 0) {
    /* Q' branch: boundaries S_end + Qcdf[k], Qcdf the per-word running sum */
    double q = 0.0, last_lo = S_end;
    int32_t last = -1;
    for (int32_t k = 0; k < K && pick < 0; k++) {
      if (k == K1) continue;
      const double qb = q;
      q += alpha * what(s, v, k);
      if (x < S_end + q) {
        pick = k;
        lo = S_end + qb;
        hi = S_end + q;
      }
      last = k;
      last_lo = S_end + qb;
    }
    if (pick < 0) {
      /* x >= Z after rounding: the last positive segment */
      pick = last;
      lo = last_lo;
      hi = Z;
      st[ORA_ST_FALLBACK]++;
    }
  }
  const double delta = fmin(x - lo, hi - x);
  uint8_t f = 0;
  if (delta < BOUNDARY_REL * Z) {
    f |= 1;
    st[ORA_ST_FLAGGED]++;
  }
  if (skip3) {
    f |= 2;
    if (pick != K1 && !(f & 1)) st[ORA_ST_SKIP_NOT_K1]++;
  }
  *flag = f;
  if (Zo) *Zo = Z;
  return pick;
}

/* -------------------------------------------------------- dense draw ---- */

static int32_t draw_dense(const snap *s, int g, double u, int64_t i, double *wh, int32_t *Dd, double *Zo,
                          uint8_t *flag, int64_t *st) {
  const int64_t v = wrow(s, s->word[i]), d = drow(s, s->doc[i]);
  const int32_t K = s->K;
  const double alpha = s->alpha;
  for (int32_t k = 0; k < K; k++) {
    Dd[k] = 0;
    wh[k] = what(s, v, k);
  }
  for (int64_t j = s->doff[d]; j < s->doff[d + 1]; j++) Dd[s->dtop[j]] = s->dcnt[j];
  /* K1, K2, K3, a4 recomputed from the dense row */
  int32_t K1 = 0;
  for (int32_t k = 1; k < K; k++)
    if (wh[k] > wh[K1]) K1 = k;
  int32_t K2 = -1;
  for (int32_t k = 0; k < K; k++)
    if (k != K1 && (K2 < 0 || wh[k] > wh[K2])) K2 = k;
  int32_t K3 = -1;
  for (int32_t k = 0; k < K; k++)
    if (k != K1 && k != K2 && (K3 < 0 || wh[k] > wh[K3])) K3 = k;
  double a4 = 0.0;
  int have4 = 0;
  for (int32_t k = 0; k < K; k++)
    if (k != K1 && k != K2 && k != K3 && (!have4 || wh[k] > a4)) {
      a4 = wh[k];
      have4 = 1;
    }
  const double a3 = K3 >= 0 ? wh[K3] : 0.0;
  const double Mm = wh[K1] * ((double)Dd[K1] + alpha);
  double S_end = Mm, sprime = 0.0;
  for (int32_t k = 0; k < K; k++) {
    if (k == K1) continue;
    double term = (double)Dd[k] * wh[k];
    S_end += term;
    sprime += term;
  }
  double Q = 0.0;
  for (int32_t k = 0; k < K; k++)
    if (k != K1) Q += alpha * wh[k];
  const double Z = S_end + Q;
  const double x = u * Z;

  int64_t len = 0;
  for (int32_t k = 0; k < K; k++) len += Dd[k];
  const double Sest = s_est(g, wh[K2], a3, a4, Dd[K1], Dd[K2], K3 >= 0 ? Dd[K3] : 0, len);
  if (sprime > Sest * (1.0 + 1e-12)) st[ORA_ST_SEST_VIOL]++;
  const int skip3 = u * (Mm + Sest + Q) < Mm;
  if (skip3) st[ORA_ST_SKIP3]++;
  else st[ORA_ST_NNZ_SCANNED] += s->doff[d + 1] - s->doff[d];

  int32_t pick = -1;
  double lo = 0.0, hi = 0.0;
  if (x < Mm) {
    pick = K1;
    hi = Mm;
    if (!skip3) st[ORA_ST_SKIP_AFTER_S]++;
  } else {
    double prev = Mm;
    for (int32_t k = 0; k < K && pick < 0; k++) {
      if (k == K1) continue;
      double cur = prev + (double)Dd[k] * wh[k];
      if (x < cur) {
        pick = k;
        lo = prev;
        hi = cur;
      }
      prev = cur;
    }
  }
  if (pick < 0) {
    double q = 0.0, last_lo = S_end;
    int32_t last = -1;
    for (int32_t k = 0; k < K && pick < 0; k++) {
      if (k == K1) continue;
      const double qb = q;
      q += alpha * wh[k];
      if (x < S_end + q) {
        pick = k;
        lo = S_end + qb;
        hi = S_end + q;
      }
      last = k;
      last_lo = S_end + qb;
    }
    if (pick < 0) {
      pick = last;
      lo = last_lo;
      hi = Z;
      st[ORA_ST_FALLBACK]++;
    }
  }
  const double delta = fmin(x - lo, hi - x);
  uint8_t f = 0;
  if (delta < BOUNDARY_REL * Z) {
    f |= 1;
    st[ORA_ST_FLAGGED]++;
  }
  if (skip3) {
    f |= 2;
    if (pick != K1 && !(f & 1)) st[ORA_ST_SKIP_NOT_K1]++;
  }
  *flag = f;
  if (Zo) *Zo = Z;
  return pick;
}

/* ---------------------------------------------------- two-branch draw ---- */
/* The two-branch form of Eq. 1 (Sec. 2.2): p = D o W^ (the S part, over
 * nz(D[d])) + alpha o W^ (the Q part, over every topic), drawn by one
 * forward inverse CDF over [S terms, topics ascending | Q terms, topics
 * ascending] with a strict "x < running sum" test.  There is no max-topic
 * branch and no skip test; this is the ablation of the three-branch split. */

static uint8_t boundary_flag(double x, double lo, double hi, double Z) {
  return fmin(x - lo, hi - x) < BOUNDARY_REL * Z ? 1 : 0;
}

static int32_t draw2_sparse(const snap *s, double u, int64_t i, double *Zo, uint8_t *flag, int64_t *st) {
  const int64_t v = wrow(s, s->word[i]), d = drow(s, s->doc[i]);
  const int32_t K = s->K;
  const double alpha = s->alpha;
  const int64_t b = s->doff[d], e = s->doff[d + 1];
  double S = 0.0;
  for (int64_t j = b; j < e; j++) S += (double)s->dcnt[j] * what(s, v, s->dtop[j]);
  const double Z = S + s->Qall[v];
  const double x = u * Z;
  st[ORA_ST_NNZ_SCANNED] += e - b;
  int32_t pick = -1;
  double lo = 0.0, hi = 0.0, prev = 0.0;
  for (int64_t j = b; j < e && pick < 0; j++) {
    const double cur = prev + (double)s->dcnt[j] * what(s, v, s->dtop[j]);
    if (x < cur) {
      pick = s->dtop[j];
      lo = prev;
      hi = cur;
    }
    prev = cur;
  }
  if (pick < 0) {
    double q = 0.0;
    for (int32_t k = 0; k < K && pick < 0; k++) {
      const double qb = q;
      q += alpha * what(s, v, k);
      if (x < S + q) {
        pick = k;
        lo = S + qb;
        hi = S + q;
      }
    }
    if (pick < 0) {
      /* x >= Z after rounding: the last segment (Q terms are all positive) */
      pick = K - 1;
      lo = S + (q - alpha * what(s, v, K - 1));
      hi = Z;
      st[ORA_ST_FALLBACK]++;
    }
  }
  const uint8_t f = boundary_flag(x, lo, hi, Z);
  if (f) st[ORA_ST_FLAGGED]++;
  *Zo = Z;
  *flag = f;
  return pick;
}

static int32_t draw2_dense(const snap *s, double u, int64_t i, double *wh, int32_t *Dd, double *Zo, uint8_t *flag,
                           int64_t *st) {
  const int64_t v = wrow(s, s->word[i]), d = drow(s, s->doc[i]);
  const int32_t K = s->K;
  const double alpha = s->alpha;
  for (int32_t k = 0; k < K; k++) {
    Dd[k] = 0;
    wh[k] = what(s, v, k);
  }
  for (int64_t j = s->doff[d]; j < s->doff[d + 1]; j++) Dd[s->dtop[j]] = s->dcnt[j];
  double S = 0.0, Q = 0.0;
  for (int32_t k = 0; k < K; k++) S += (double)Dd[k] * wh[k];
  for (int32_t k = 0; k < K; k++) Q += alpha * wh[k];
  const double Z = S + Q;
  const double x = u * Z;
  st[ORA_ST_NNZ_SCANNED] += s->doff[d + 1] - s->doff[d];
  int32_t pick = -1;
  double lo = 0.0, hi = 0.0, prev = 0.0;
  for (int32_t k = 0; k < K && pick < 0; k++) {
    const double cur = prev + (double)Dd[k] * wh[k];
    if (x < cur) {
      pick = k;
      lo = prev;
      hi = cur;
    }
    prev = cur;
  }
  if (pick < 0) {
    double q = 0.0;
    for (int32_t k = 0; k < K && pick < 0; k++) {
      const double qb = q;
      q += alpha * wh[k];
      if (x < S + q) {
        pick = k;
        lo = S + qb;
        hi = S + q;
      }
    }
    if (pick < 0) {
      pick = K - 1;
      lo = S + (q - alpha * wh[K - 1]);
      hi = Z;
      st[ORA_ST_FALLBACK]++;
    }
  }
  const uint8_t f = boundary_flag(x, lo, hi, Z);
  if (f) st[ORA_ST_FLAGGED]++;
  *Zo = Z;
  *flag = f;
  return pick;
}

/* ---------------------------------------------------------- iterate ---- */

/* Draws tokens idx[0..cnt) (or first..first+cnt-1 when idx is NULL) from
 * the snapshot; outputs at [0, cnt).  Statistics are added to st. */
static int draw_tokens(const snap *s, int mode, int g, uint64_t seed, uint32_t t, int64_t first, int64_t cnt,
                       const int64_t *idx, int32_t *z_out, uint8_t *flags, double *Zout, int64_t *st) {
  if (mode < 0 || mode > 3 || g < 1 || g > 3) return 1;
  const int dense = mode & 1, two = mode & 2;
  if (!dense && !s->K1) return 1; /* the sparse form needs the per-word quantities */
  const int32_t K = s->K;
  double *wh = NULL;
  int32_t *Dd = NULL;
  if (dense) {
    wh = malloc(sizeof(double) * (size_t)K);
    Dd = malloc(sizeof(int32_t) * (size_t)K);
    if (!wh || !Dd) {
      free(wh);
      free(Dd);
      return 2;
    }
  }
  int rc = 0;
  for (int64_t j = 0; j < cnt; j++) {
    const int64_t i = idx ? idx[j] : first + j;
    if (i < 0 || i >= s->n || wrow(s, s->word[i]) < 0 || drow(s, s->doc[i]) < 0) {
      rc = 1;
      break;
    }
    double Z;
    uint8_t f;
    const double u = ora_uniform(seed, t, (uint64_t)i);
    int32_t k;
    if (two) k = dense ? draw2_dense(s, u, i, wh, Dd, &Z, &f, st) : draw2_sparse(s, u, i, &Z, &f, st);
    else k = dense ? draw_dense(s, g, u, i, wh, Dd, &Z, &f, st) : draw_sparse(s, g, u, i, &Z, &f, st);
    z_out[j] = k;
    if (flags) flags[j] = f;
    if (Zout) Zout[j] = Z;
  }
  free(wh);
  free(Dd);
  return rc;
}

int ora_iterate(int mode, int g, int64_t n, const int32_t *word, const int32_t *doc, int32_t M, int32_t V, int32_t K,
                double alpha, double beta, uint64_t seed, uint32_t t, const int32_t *z_in, int64_t n_sub,
                const int64_t *idx, int32_t *z_out, uint8_t *flags, double *Zout, int64_t *stats) {
  if (mode < 0 || mode > 3 || g < 1 || g > 3 || K < 2 || !(alpha > 0) || !(beta > 0)) return 1;
  snap s;
  int rc = snap_build(&s, n, word, doc, z_in, M, V, K, alpha, beta, !(mode & 1));
  if (rc) return rc;
  int64_t st[ORA_N_STATS];
  memset(st, 0, sizeof(st));
  rc = draw_tokens(&s, mode, g, seed, t, 0, idx ? n_sub : n, idx, z_out, flags, Zout, st);
  if (stats) memcpy(stats, st, sizeof(st));
  snap_free(&s);
  return rc;
}

/* -------------------------------------------------------------- LLPT ---- */

double ora_llpt(int mode, int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V,
                int32_t K, double alpha, double beta) {
  snap s;
  if (n <= 0 || snap_build(&s, n, word, doc, z, M, V, K, alpha, beta, mode == 0)) return NAN;
  /* Neumaier-compensated sum of the per-token log2 terms */
  double sum = 0.0, comp = 0.0;
  const double Kalpha = (double)K * alpha;
  int32_t *Dd = mode == 1 ? malloc(sizeof(int32_t) * (size_t)K) : NULL;
  for (int64_t i = 0; i < n; i++) {
    const int32_t v = word[i], d = doc[i];
    double term;
    if (mode == 1) {
      for (int32_t k = 0; k < K; k++) Dd[k] = 0;
      for (int64_t j = s.doff[d]; j < s.doff[d + 1]; j++) Dd[s.dtop[j]] = s.dcnt[j];
      double p = 0.0;
      for (int32_t k = 0; k < K; k++) p += (((double)Dd[k] + alpha) / ((double)s.len[d] + Kalpha)) * what(&s, v, k);
      term = log2(p);
    } else {
      double num = 0.0;
      for (int64_t j = s.doff[d]; j < s.doff[d + 1]; j++) num += (double)s.dcnt[j] * what(&s, v, s.dtop[j]);
      num += alpha * s.sumWh[v];
      term = log2(num / ((double)s.len[d] + Kalpha));
    }
    double tsum = sum + term;
    if (fabs(sum) >= fabs(term)) comp += (sum - tsum) + term;
    else comp += (term - tsum) + sum;
    sum = tsum;
  }
  free(Dd);
  snap_free(&s);
  return (sum + comp) / (double)n;
}

int ora_word_stats(int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V,
                   int32_t K, double alpha, double beta, int32_t *K1, int32_t *K2, double *a1, double *a2, double *a3,
                   double *Qp) {
  snap s;
  int rc = snap_build(&s, n, word, doc, z, M, V, K, alpha, beta, 1);
  if (rc) return rc;
  memcpy(K1, s.K1, sizeof(int32_t) * (size_t)V);
  memcpy(K2, s.K2, sizeof(int32_t) * (size_t)V);
  memcpy(a1, s.a1, sizeof(double) * (size_t)V);
  memcpy(a2, s.a2, sizeof(double) * (size_t)V);
  memcpy(a3, s.a3, sizeof(double) * (size_t)V);
  memcpy(Qp, s.Qp, sizeof(double) * (size_t)V);
  snap_free(&s);
  return 0;
}

int ora_word_top4(int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V,
                  int32_t K, double alpha, double beta, int32_t *K3, double *a4) {
  snap s;
  int rc = snap_build(&s, n, word, doc, z, M, V, K, alpha, beta, 1);
  if (rc) return rc;
  memcpy(K3, s.K3, sizeof(int32_t) * (size_t)V);
  memcpy(a4, s.a4, sizeof(double) * (size_t)V);
  snap_free(&s);
  return 0;
}

int32_t ora_draw_given_u(int mode, int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M,
                         int32_t V, int32_t K, double alpha, double beta, int64_t i, double u, double *Z,
                         uint8_t *flag) {
  if (mode < 0 || mode > 3 || K < 2 || i < 0 || i >= n || !(u >= 0.0 && u < 1.0)) return -1;
  const int dense = mode & 1, two = mode & 2;
  snap s;
  if (snap_build(&s, n, word, doc, z, M, V, K, alpha, beta, !dense)) return -1;
  int64_t st[ORA_N_STATS];
  memset(st, 0, sizeof(st));
  int32_t k;
  if (!dense) {
    k = two ? draw2_sparse(&s, u, i, Z, flag, st) : draw_sparse(&s, 2, u, i, Z, flag, st);
  } else {
    double *wh = malloc(sizeof(double) * (size_t)K);
    int32_t *Dd = malloc(sizeof(int32_t) * (size_t)K);
    k = (wh && Dd) ? (two ? draw2_dense(&s, u, i, wh, Dd, Z, flag, st) : draw_dense(&s, 2, u, i, wh, Dd, Z, flag, st))
                   : -1;
    free(wh);
    free(Dd);
  }
  snap_free(&s);
  return k;
}

int ora_what_row(int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V, int32_t K,
                 double beta, int32_t v, double *out) {
  if (v < 0 || v >= V) return 1;
  snap s;
  int rc = snap_build(&s, n, word, doc, z, M, V, K, 1.0, beta, 0);
  if (rc) return rc;
  for (int32_t k = 0; k < K; k++) out[k] = what(&s, v, k);
  snap_free(&s);
  return 0;
}

/* ------------------------------------------------------ snapshot API ---- */

int ora_snapshot_new(int64_t n, const int32_t *word, const int32_t *doc, const int32_t *z, int32_t M, int32_t V,
                     int32_t K, double alpha, double beta, int with_words, int64_t n_idx, const int64_t *idx,
                     ora_snapshot **out) {
  *out = NULL;
  if (n < 0 || M < 0 || V <= 0 || K < 2 || !(alpha > 0) || !(beta > 0) || (idx == NULL && n_idx != 0)) return 1;
  snap *s = malloc(sizeof(snap));
  if (!s) return 2;
  snap_init(s, n, word, doc, M, V, K, alpha, beta);
  int rc = idx ? snap_counts_sub(s, z, n_idx, idx) : snap_counts_full(s, z);
  if (!rc) rc = snap_finish(s, with_words);
  if (rc) {
    snap_free(s);
    free(s);
    return rc;
  }
  *out = s;
  return 0;
}

int ora_snapshot_draw(const ora_snapshot *s, int mode, int g, uint64_t seed, uint32_t t, int64_t first, int64_t cnt,
                      const int64_t *idx, int32_t *z_out, uint8_t *flags, double *Zout, int64_t *stats) {
  if (!s || cnt < 0) return 1;
  int64_t st[ORA_N_STATS];
  memset(st, 0, sizeof(st));
  const int rc = draw_tokens(s, mode, g, seed, t, first, cnt, idx, z_out, flags, Zout, st);
  if (stats) memcpy(stats, st, sizeof(st));
  return rc;
}

int ora_snapshot_llpt(const ora_snapshot *s, int64_t first, int64_t cnt, double *sum_out, double *comp_out) {
  if (!s || !s->sumWh || s->wslot || first < 0 || cnt < 0 || first + cnt > s->n) return 1;
  const double Kalpha = (double)s->K * s->alpha;
  double sum = 0.0, comp = 0.0;
  for (int64_t i = first; i < first + cnt; i++) {
    const int32_t v = s->word[i], d = s->doc[i];
    double num = 0.0;
    for (int64_t j = s->doff[d]; j < s->doff[d + 1]; j++) num += (double)s->dcnt[j] * what(s, v, s->dtop[j]);
    num += s->alpha * s->sumWh[v];
    const double term = log2(num / ((double)s->len[d] + Kalpha));
    const double tsum = sum + term;
    if (fabs(sum) >= fabs(term)) comp += (sum - tsum) + term;
    else comp += (term - tsum) + sum;
    sum = tsum;
  }
  *sum_out = sum;
  *comp_out = comp;
  return 0;
}

void ora_snapshot_free(ora_snapshot *s) {
  if (!s) return;
  snap_free(s);
  free(s);
}

void ora_init_range(int64_t first, int64_t cnt, int32_t K, uint64_t seed, int32_t *z) {
  for (int64_t j = 0; j < cnt; j++) z[j] = ora_init_topic(seed, (uint64_t)(first + j), K);
}
