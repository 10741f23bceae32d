/* The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only):
 * seeded small corpora through every entry point, with the checks that tie
 * the forms together (dense = sparse bit for bit, a restricted snapshot = the
 * full one, count invariants).  Exit status 0 = every check held and the
 * sanitizers found nothing. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "lda_oracle.h"

static uint64_t rs = 88172645463325252ull;
static uint32_t rnd(uint32_t n) {
  rs ^= rs << 13;
  rs ^= rs >> 7;
  rs ^= rs << 17;
  return (uint32_t)(rs % n);
}

#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      return 1;                                                    \
    }                                                              \
  } while (0)

static int one_corpus(int trial) {
  const int32_t M = 1 + (int32_t)rnd(25), V = 1 + (int32_t)rnd(40), K = 2 + (int32_t)rnd(9);
  const int64_t n = 1 + rnd(400);
  int32_t *word = malloc(sizeof(int32_t) * n), *doc = malloc(sizeof(int32_t) * n), *z = malloc(sizeof(int32_t) * n);
  int32_t *za = malloc(sizeof(int32_t) * n), *zb = malloc(sizeof(int32_t) * n);
  uint8_t *fa = malloc(n), *fb = malloc(n);
  double *Za = malloc(sizeof(double) * n), *Zb = malloc(sizeof(double) * n);
  for (int64_t i = 0; i < n; i++) {
    word[i] = (int32_t)rnd((uint32_t)V);
    doc[i] = (int32_t)rnd((uint32_t)M);
  }
  ora_init(n, K, 42 + (uint64_t)trial, z);
  /* counts: sum_k D[d][k] = len(d), sum W = T, sum T = n */
  int64_t *len = malloc(sizeof(int64_t) * M), *doff = malloc(sizeof(int64_t) * (M + 1)), *T = malloc(sizeof(int64_t) * K);
  int32_t *dtop = malloc(sizeof(int32_t) * n), *dcnt = malloc(sizeof(int32_t) * n), *W = malloc(sizeof(int32_t) * V * K);
  CHECK(ora_build_counts(n, word, doc, z, M, V, K, len, doff, dtop, dcnt, W, T) == 0);
  int64_t tot = 0;
  for (int32_t k = 0; k < K; k++) tot += T[k];
  CHECK(tot == n);
  for (int32_t d = 0; d < M; d++) {
    int64_t s = 0;
    for (int64_t e = doff[d]; e < doff[d + 1]; e++) s += dcnt[e];
    CHECK(s == len[d]);
  }
  for (int mode2 = 0; mode2 <= 2; mode2 += 2) {
    for (int g = 1; g <= 3; g++) {
      int64_t sa[8], sb[8];
      CHECK(ora_iterate(0 | mode2, g, n, word, doc, M, V, K, 0.3, 0.05, 7, (uint32_t)trial, z, 0, NULL, za, fa, Za, sa) == 0);
      CHECK(ora_iterate(1 | mode2, g, n, word, doc, M, V, K, 0.3, 0.05, 7, (uint32_t)trial, z, 0, NULL, zb, fb, Zb, sb) == 0);
      for (int64_t i = 0; i < n; i++) CHECK(za[i] == zb[i] && fa[i] == fb[i] && Za[i] == Zb[i]);
      if (!mode2) CHECK(sa[ORA_ST_SEST_VIOL] == 0 && sa[ORA_ST_SKIP_NOT_K1] == 0);
    }
  }
  /* a restricted snapshot holding the rows of every fifth token draws those tokens as the full one does */
  int64_t m = 0, *idx = malloc(sizeof(int64_t) * n);
  for (int64_t i = 0; i < n; i += 5) idx[m++] = i;
  for (int restricted = 0; restricted < 2; restricted++) {
    ora_snapshot *s = NULL;
    CHECK(ora_snapshot_new(n, word, doc, z, M, V, K, 0.3, 0.05, 1, restricted ? m : 0, restricted ? idx : NULL, &s) == 0);
    int64_t st[8];
    CHECK(ora_snapshot_draw(s, 0, 2, 7, 3, 0, m, idx, restricted ? zb : za, restricted ? fb : fa, NULL, st) == 0);
    if (!restricted) {
      double sum = 0, comp = 0;
      CHECK(ora_snapshot_llpt(s, 0, n, &sum, &comp) == 0);
      CHECK(fabs((sum + comp) / (double)n - ora_llpt(0, n, word, doc, z, M, V, K, 0.3, 0.05)) < 1e-12);
    }
    ora_snapshot_free(s);
  }
  for (int64_t j = 0; j < m; j++) CHECK(za[j] == zb[j] && fa[j] == fb[j]);
  const double l0 = ora_llpt(0, n, word, doc, z, M, V, K, 0.3, 0.05), l1 = ora_llpt(1, n, word, doc, z, M, V, K, 0.3, 0.05);
  CHECK(fabs(l0 - l1) <= 1e-12 * (1.0 + fabs(l1)));
  int32_t k3[64];
  double a4[64];
  if (V <= 64) CHECK(ora_word_top4(n, word, doc, z, M, V, K, 0.3, 0.05, k3, a4) == 0);
  double row[16], Zo;
  uint8_t f;
  CHECK(ora_what_row(n, word, doc, z, M, V, K, 0.05, word[0], row) == 0);
  CHECK(ora_draw_given_u(0, n, word, doc, z, M, V, K, 0.3, 0.05, n - 1, 0.5, &Zo, &f) >= 0);
  free(word), free(doc), free(z), free(za), free(zb), free(fa), free(fb), free(Za), free(Zb);
  free(len), free(doff), free(T), free(dtop), free(dcnt), free(W), free(idx);
  return 0;
}

int main(void) {
  for (int trial = 0; trial < 60; trial++)
    if (one_corpus(trial)) {
      fprintf(stderr, "trial %d\n", trial);
      return 1;
    }
  printf("oracle checks passed\n");
  return 0;
}
