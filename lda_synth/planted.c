/*
 * Planted-LDA synthetic corpus generator.
 *
 * This module only produces seeded inputs (token lists of <word, doc>); it
 * contains none of the sampler's arithmetic and is shared by the tests, the
 * benchmark and the oracle's checks.  It stands in for the paper's datasets
 * (PubMed, NYTimes, UMBC; Sec. 6), which are not available.
 *
 * Process (per corpus):
 *   base b_v = (v+1)^-s / H                      (Zipf vocabulary base)
 *   phi_j ~ Dirichlet(eta), eta_v = eta_scale * V * b_v, j < J   (log-space Gamma)
 *   per doc d: theta_d ~ Dirichlet(conc * 1_J) is integrated out and the
 *   topic sequence is drawn from the equivalent Polya urn:
 *       P(z_n = j | z_<n) = (conc + n_j) / (J*conc + n)
 *   w ~ Cat(phi_{z_n}) through a per-topic Walker/Vose alias table.
 *   Word ids are finally passed through a seeded random permutation so that
 *   id order carries no frequency information.
 *
 * Random numbers: xoshiro256** streams seeded through splitmix64 from
 * (seed, stream id).  Stream ids: topic j -> phi; doc d -> its tokens.  The
 * output is therefore independent of the number of threads.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  uint64_t s[4];
} rng_t;

static uint64_t splitmix64(uint64_t *x) {
  uint64_t z = (*x += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static void rng_init(rng_t *r, uint64_t seed, uint64_t stream) {
  uint64_t x = seed * 0xD1342543DE82EF95ull + stream * 0x2545F4914F6CDD1Dull + 0x632BE59BD9B4E019ull;
  for (int i = 0; i < 4; i++) r->s[i] = splitmix64(&x);
}

static inline uint64_t rotl(uint64_t x, int k) { return (x << k) | (x >> (64 - k)); }

static inline uint64_t rng_next(rng_t *r) {
  uint64_t *s = r->s;
  uint64_t res = rotl(s[1] * 5, 7) * 9;
  uint64_t t = s[1] << 17;
  s[2] ^= s[0];
  s[3] ^= s[1];
  s[1] ^= s[2];
  s[0] ^= s[3];
  s[2] ^= t;
  s[3] = rotl(s[3], 45);
  return res;
}

/* uniform on the open interval (0,1) */
static inline double rng_unif(rng_t *r) { return ((double)(rng_next(r) >> 11) + 0.5) * (1.0 / 9007199254740992.0); }

static double rng_normal(rng_t *r) {
  /* Marsaglia polar method */
  for (;;) {
    double a = 2.0 * rng_unif(r) - 1.0, b = 2.0 * rng_unif(r) - 1.0;
    double q = a * a + b * b;
    if (q > 0.0 && q < 1.0) return a * sqrt(-2.0 * log(q) / q);
  }
}

/* log of a Gamma(a, 1) variate: Marsaglia-Tsang (2000) for a >= 1, and the
 * boost Gamma(a) = Gamma(a+1) * U^(1/a) for a < 1, kept in log space so that
 * shapes far below 1 do not underflow. */
static double rng_log_gamma(rng_t *r, double a) {
  if (a < 1.0) return rng_log_gamma(r, a + 1.0) + log(rng_unif(r)) / a;
  double d = a - 1.0 / 3.0, c = 1.0 / sqrt(9.0 * d);
  for (;;) {
    double x = rng_normal(r), v = 1.0 + c * x;
    if (v <= 0.0) continue;
    v = v * v * v;
    double u = rng_unif(r);
    if (log(u) < 0.5 * x * x + d - d * v + d * log(v)) return log(d * v);
  }
}

/* ---------------------------------------------------------------- phi ---- */

typedef struct {
  int V, J, nthreads, tid;
  double s, eta_scale;
  uint64_t seed;
  float *prob;
  uint32_t *alias;
  const uint32_t *perm;
} phi_job;

static void build_alias(int V, const double *p, float *prob, uint32_t *alias, uint32_t *small, uint32_t *large,
                        double *scaled) {
  int ns = 0, nl = 0;
  for (int v = 0; v < V; v++) {
    scaled[v] = p[v] * V;
    if (scaled[v] < 1.0) small[ns++] = v;
    else large[nl++] = v;
  }
  while (ns > 0 && nl > 0) {
    uint32_t sm = small[--ns], lg = large[--nl];
    prob[sm] = (float)scaled[sm];
    alias[sm] = lg;
    scaled[lg] = (scaled[lg] + scaled[sm]) - 1.0;
    if (scaled[lg] < 1.0) small[ns++] = lg;
    else large[nl++] = lg;
  }
  while (nl > 0) {
    uint32_t lg = large[--nl];
    prob[lg] = 1.0f;
    alias[lg] = lg;
  }
  while (ns > 0) {
    uint32_t sm = small[--ns];
    prob[sm] = 1.0f;
    alias[sm] = sm;
  }
}

static void *phi_worker(void *arg) {
  phi_job *jb = (phi_job *)arg;
  int V = jb->V;
  double *base = malloc(sizeof(double) * V);
  double *lg = malloc(sizeof(double) * V);
  double *scaled = malloc(sizeof(double) * V);
  uint32_t *small = malloc(sizeof(uint32_t) * V), *large = malloc(sizeof(uint32_t) * V);
  double H = 0.0;
  for (int v = 0; v < V; v++) {
    base[v] = pow((double)v + 1.0, -jb->s);
    H += base[v];
  }
  for (int v = 0; v < V; v++) base[v] = jb->eta_scale * (double)V * base[v] / H;
  for (int j = jb->tid; j < jb->J; j += jb->nthreads) {
    rng_t r;
    rng_init(&r, jb->seed, 0x100000000ull + (uint64_t)j);
    double mx = -INFINITY;
    for (int v = 0; v < V; v++) {
      /* phi is indexed by permuted word id so that alias slots are final ids */
      double x = rng_log_gamma(&r, base[v]);
      lg[jb->perm[v]] = x;
      if (x > mx) mx = x;
    }
    double sum = 0.0;
    for (int v = 0; v < V; v++) {
      lg[v] = exp(lg[v] - mx);
      sum += lg[v];
    }
    for (int v = 0; v < V; v++) lg[v] /= sum;
    build_alias(V, lg, jb->prob + (size_t)j * V, jb->alias + (size_t)j * V, small, large, scaled);
  }
  free(base);
  free(lg);
  free(scaled);
  free(small);
  free(large);
  return NULL;
}

/* Word-id permutation: Fisher-Yates from stream 0xFFFF0000. */
int synth_perm(int V, uint64_t seed, uint32_t *perm) {
  rng_t r;
  rng_init(&r, seed, 0xFFFF0000ull);
  for (int v = 0; v < V; v++) perm[v] = (uint32_t)v;
  for (int v = V - 1; v > 0; v--) {
    uint64_t j = rng_next(&r) % (uint64_t)(v + 1);
    uint32_t t = perm[v];
    perm[v] = perm[j];
    perm[j] = t;
  }
  return 0;
}

int synth_phi_alias(int V, double s, int J, double eta_scale, uint64_t seed, int nthreads, const uint32_t *perm,
                    float *prob, uint32_t *alias) {
  if (V <= 0 || J <= 0 || nthreads <= 0) return 1;
  pthread_t *th = malloc(sizeof(pthread_t) * nthreads);
  phi_job *jobs = malloc(sizeof(phi_job) * nthreads);
  for (int t = 0; t < nthreads; t++) {
    jobs[t] = (phi_job){V, J, nthreads, t, s, eta_scale, seed, prob, alias, perm};
    pthread_create(&th[t], NULL, phi_worker, &jobs[t]);
  }
  for (int t = 0; t < nthreads; t++) pthread_join(th[t], NULL);
  free(th);
  free(jobs);
  return 0;
}

/* ------------------------------------------------------------- tokens ---- */

typedef struct {
  int64_t n_docs;
  const int32_t *len;
  const int64_t *start;
  int J, V, nthreads, tid;
  double conc;
  const float *prob;
  const uint32_t *alias;
  uint64_t seed;
  int32_t *word, *doc;
  int32_t *topic; /* optional planted topics (may be NULL) */
} tok_job;

static void *tok_worker(void *arg) {
  tok_job *jb = (tok_job *)arg;
  int32_t maxlen = 0;
  for (int64_t d = 0; d < jb->n_docs; d++)
    if (jb->len[d] > maxlen) maxlen = jb->len[d];
  int32_t *zt = malloc(sizeof(int32_t) * (maxlen > 0 ? maxlen : 1));
  const double Jc = (double)jb->J * jb->conc;
  const int64_t chunk = 1024;
  for (int64_t c0 = (int64_t)jb->tid * chunk; c0 < jb->n_docs; c0 += (int64_t)jb->nthreads * chunk) {
    int64_t c1 = c0 + chunk < jb->n_docs ? c0 + chunk : jb->n_docs;
    for (int64_t d = c0; d < c1; d++) {
      rng_t r;
      rng_init(&r, jb->seed, 0x200000000ull + (uint64_t)d);
      int64_t o = jb->start[d];
      for (int32_t n = 0; n < jb->len[d]; n++) {
        int32_t z;
        if (rng_unif(&r) * (Jc + (double)n) < Jc) z = (int32_t)(rng_unif(&r) * jb->J);
        else z = zt[(int32_t)(rng_unif(&r) * n)];
        if (z >= jb->J) z = jb->J - 1;
        zt[n] = z;
        uint64_t x = rng_next(&r);
        uint32_t slot = (uint32_t)(((x >> 32) * (uint64_t)jb->V) >> 32);
        double coin = (double)(x & 0xFFFFFFFFull) * (1.0 / 4294967296.0);
        size_t base = (size_t)z * jb->V;
        int32_t w = coin < (double)jb->prob[base + slot] ? (int32_t)slot : (int32_t)jb->alias[base + slot];
        jb->word[o + n] = w;
        jb->doc[o + n] = (int32_t)d;
        if (jb->topic) jb->topic[o + n] = z;
      }
    }
  }
  free(zt);
  return NULL;
}

/* Tokens of every doc, written doc-sorted at start[d] .. start[d]+len[d]. */
int synth_tokens(int64_t n_docs, const int32_t *len, const int64_t *start, int J, double conc, int V, const float *prob,
                 const uint32_t *alias, uint64_t seed, int nthreads, int32_t *word, int32_t *doc, int32_t *topic) {
  if (n_docs < 0 || J <= 0 || V <= 0 || nthreads <= 0) return 1;
  pthread_t *th = malloc(sizeof(pthread_t) * nthreads);
  tok_job *jobs = malloc(sizeof(tok_job) * nthreads);
  for (int t = 0; t < nthreads; t++) {
    jobs[t] = (tok_job){n_docs, len, start, J, V, nthreads, t, conc, prob, alias, seed, word, doc, topic};
    pthread_create(&th[t], NULL, tok_worker, &jobs[t]);
  }
  for (int t = 0; t < nthreads; t++) pthread_join(th[t], NULL);
  free(th);
  free(jobs);
  return 0;
}
