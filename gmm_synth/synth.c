/*
 * Seeded synthetic inputs for the diagonal-GMM EM hot path.
 *
 * This file holds no arithmetic of the method itself: it only draws the
 * data matrix X, the true mixture it is drawn from, and the random-point
 * initial parameters, so that the GPU path and the CPU checker see the
 * very same fp32 bytes.
 *
 * Random numbers come from Philox4x32-10, the counter-based generator of
 * Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as easy as
 * 1, 2, 3" (SC'11), written here from its published definition (round
 * function, multipliers 0xD2511F53 / 0xCD9E8D57, Weyl key increments
 * 0x9E3779B9 / 0xBB67AE85, ten rounds).  Every draw is addressed by
 * (seed, stream, counter), so any row slice of X can be regenerated on its
 * own without generating the rows before it.
 *
 * Streams (key word 1):
 *   1 = true component means, 2 = true per-dim std devs, 3 = true weights,
 *   4 = rows of X, 5 = random-point initialisation.
 *
 * Normals use the Box-Muller transform (Box & Muller 1958) in fp64.
 * Weights ~ Dirichlet(1, ..., 1) are drawn as normalised Exp(1) variates.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct { uint32_t v[4]; } ctr4;

static inline void mulhilo32(uint32_t a, uint32_t b, uint32_t* hi, uint32_t* lo) {
  uint64_t p = (uint64_t)a * (uint64_t)b;
  *hi = (uint32_t)(p >> 32);
  *lo = (uint32_t)p;
}

/* Philox4x32-10: 10 rounds of the 4x32 round function with key schedule. */
static ctr4 philox4x32_10(ctr4 c, uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    uint32_t hi0, lo0, hi1, lo1;
    mulhilo32(0xD2511F53u, c.v[0], &hi0, &lo0);
    mulhilo32(0xCD9E8D57u, c.v[2], &hi1, &lo1);
    ctr4 n;
    n.v[0] = hi1 ^ c.v[1] ^ k0;
    n.v[1] = lo1;
    n.v[2] = hi0 ^ c.v[3] ^ k1;
    n.v[3] = lo0;
    c = n;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

/* Public for known-answer tests of the generator itself. */
void synth_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  ctr4 c = {{ctr[0], ctr[1], ctr[2], ctr[3]}};
  ctr4 r = philox4x32_10(c, key[0], key[1]);
  memcpy(out, r.v, sizeof(r.v));
}

/* Uniform in the open interval (0, 1) from one 32-bit word. */
static inline double u01(uint32_t w) { return ((double)w + 0.5) * (1.0 / 4294967296.0); }

static inline void draw(uint64_t seed, uint32_t stream, uint64_t a, uint64_t b, uint32_t out[4]) {
  ctr4 c = {{(uint32_t)a, (uint32_t)(a >> 32), (uint32_t)b, (uint32_t)(b >> 32)}};
  uint32_t k0 = (uint32_t)seed ^ (uint32_t)(seed >> 32) * 0x85EBCA6Bu;
  ctr4 r = philox4x32_10(c, k0, stream);
  memcpy(out, r.v, 16);
}

/* Box-Muller pair from two uniforms. */
static inline void box_muller(uint32_t w0, uint32_t w1, double* z0, double* z1) {
  double u1 = u01(w0), u2 = u01(w1);
  double rad = sqrt(-2.0 * log(u1));
  double th = 6.283185307179586476925286766559 * u2;
  *z0 = rad * cos(th);
  *z1 = rad * sin(th);
}

/* Standard normal number j (0-based) of the sequence addressed by (stream, a). */
static double normal_at(uint64_t seed, uint32_t stream, uint64_t a, uint64_t j) {
  uint32_t w[4];
  draw(seed, stream, a, j / 2, w);
  double z0, z1;
  box_muller(w[0], w[1], &z0, &z1);
  return (j & 1) ? z1 : z0;
}

/*
 * True mixture: means[kt*d] ~ N(0, mean_std^2), stds[kt*d] ~ U[std_lo, std_hi],
 * weights[kt] ~ Dirichlet(1).  Outputs are fp64 (rounded to fp32 only in X).
 */
void synth_true_mixture(uint64_t seed, int32_t kt, int32_t d, double mean_std, double std_lo,
                        double std_hi, double* means, double* stds, double* weights) {
  for (int32_t k = 0; k < kt; ++k) {
    for (int32_t j = 0; j < d; ++j) {
      means[(int64_t)k * d + j] = mean_std * normal_at(seed, 1, (uint64_t)k, (uint64_t)j);
      uint32_t w[4];
      draw(seed, 2, (uint64_t)k, (uint64_t)j, w);
      stds[(int64_t)k * d + j] = std_lo + (std_hi - std_lo) * u01(w[0]);
    }
  }
  double tot = 0.0;
  for (int32_t k = 0; k < kt; ++k) {
    uint32_t w[4];
    draw(seed, 3, (uint64_t)k, 0, w);
    weights[k] = -log(u01(w[0]));
    tot += weights[k];
  }
  for (int32_t k = 0; k < kt; ++k) weights[k] /= tot;
}

typedef struct {
  uint64_t seed;
  int64_t row0, row1; /* rows [row0, row1) of the full matrix */
  int32_t d, kt, normalize;
  const double *means, *stds, *cum;
  float* out; /* (row1-row0) x d */
  int32_t* comp;
  double* colsum; /* d, fp64 sums of the fp32 values */
  double* colsq;
} rows_job;

static void* rows_worker(void* p) {
  rows_job* jb = (rows_job*)p;
  const int32_t d = jb->d;
  double* z = (double*)malloc(sizeof(double) * (size_t)d);
  if (jb->colsum) {
    memset(jb->colsum, 0, sizeof(double) * (size_t)d);
    memset(jb->colsq, 0, sizeof(double) * (size_t)d);
  }
  for (int64_t i = jb->row0; i < jb->row1; ++i) {
    uint32_t w[4];
    draw(jb->seed, 4, (uint64_t)i, 0, w);
    double u = u01(w[0]);
    /* component: first k with u < cum[k] (binary search on the cumulative weights) */
    int32_t lo = 0, hi = jb->kt - 1;
    while (lo < hi) {
      int32_t mid = (lo + hi) / 2;
      if (u < jb->cum[mid]) hi = mid; else lo = mid + 1;
    }
    const int32_t c = lo;
    for (int32_t j = 0; j < d; j += 2) {
      draw(jb->seed, 4, (uint64_t)i, 1 + (uint64_t)(j / 4), w);
      int off = (j % 4 == 0) ? 0 : 2;
      double z0, z1;
      box_muller(w[off], w[off + 1], &z0, &z1);
      z[j] = jb->means[(int64_t)c * d + j] + jb->stds[(int64_t)c * d + j] * z0;
      if (j + 1 < d) z[j + 1] = jb->means[(int64_t)c * d + j + 1] + jb->stds[(int64_t)c * d + j + 1] * z1;
    }
    if (jb->normalize) {
      double s = 0.0;
      for (int32_t j = 0; j < d; ++j) s += z[j] * z[j];
      double inv = 1.0 / sqrt(s);
      for (int32_t j = 0; j < d; ++j) z[j] *= inv;
    }
    float* o = jb->out + (i - jb->row0) * (int64_t)d;
    for (int32_t j = 0; j < d; ++j) {
      float v = (float)z[j];
      o[j] = v;
      if (jb->colsum) {
        jb->colsum[j] += (double)v;
        jb->colsq[j] += (double)v * (double)v;
      }
    }
    if (jb->comp) jb->comp[i - jb->row0] = c;
  }
  free(z);
  return NULL;
}

/*
 * Rows [row0, row1) of X (fp32, row-major, (row1-row0) x d), drawn from the
 * true mixture given as fp64 arrays.  comp (optional) receives the true
 * component of each row; colsum / colsq (optional, d each) receive fp64 sums
 * of the fp32 values and of their squares over the slice, combined in a
 * fixed thread order so that the result does not depend on timing.
 * Returns 0 on success.
 */
int synth_rows(uint64_t seed, int64_t row0, int64_t row1, int32_t d, int32_t kt,
               const double* means, const double* stds, const double* weights, int32_t normalize,
               int32_t nthreads, float* out, int32_t* comp, double* colsum, double* colsq) {
  if (row1 < row0 || d <= 0 || kt <= 0) return -1;
  double* cum = (double*)malloc(sizeof(double) * (size_t)kt);
  double acc = 0.0;
  for (int32_t k = 0; k < kt; ++k) { acc += weights[k]; cum[k] = acc; }
  cum[kt - 1] = 2.0; /* guard: u < 1 always lands in the last bucket at worst */
  if (nthreads < 1) nthreads = 1;
  int64_t n = row1 - row0;
  if (n < (int64_t)nthreads * 64) nthreads = (int32_t)(n / 64 > 0 ? n / 64 : 1);
  rows_job* jobs = (rows_job*)calloc((size_t)nthreads, sizeof(rows_job));
  pthread_t* th = (pthread_t*)calloc((size_t)nthreads, sizeof(pthread_t));
  double* part = colsum ? (double*)calloc((size_t)nthreads * 2 * (size_t)d, sizeof(double)) : NULL;
  for (int32_t t = 0; t < nthreads; ++t) {
    rows_job* jb = &jobs[t];
    jb->seed = seed;
    jb->row0 = row0 + n * t / nthreads;
    jb->row1 = row0 + n * (t + 1) / nthreads;
    jb->d = d; jb->kt = kt; jb->normalize = normalize;
    jb->means = means; jb->stds = stds; jb->cum = cum;
    jb->out = out + (jb->row0 - row0) * (int64_t)d;
    jb->comp = comp ? comp + (jb->row0 - row0) : NULL;
    jb->colsum = part ? part + (size_t)t * 2 * d : NULL;
    jb->colsq = part ? part + (size_t)t * 2 * d + d : NULL;
    pthread_create(&th[t], NULL, rows_worker, jb);
  }
  for (int32_t t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  if (colsum) {
    memset(colsum, 0, sizeof(double) * (size_t)d);
    memset(colsq, 0, sizeof(double) * (size_t)d);
    for (int32_t t = 0; t < nthreads; ++t)
      for (int32_t j = 0; j < d; ++j) {
        colsum[j] += part[(size_t)t * 2 * d + j];
        colsq[j] += part[(size_t)t * 2 * d + d + j];
      }
  }
  free(part); free(th); free(jobs); free(cum);
  return 0;
}

/*
 * k distinct row indices in [0, n), the first k positions of a Fisher-Yates
 * shuffle driven by stream 5.  The swaps are kept in a small open-addressing
 * table, so memory is O(k) even when n is 1e8.
 */
int synth_init_rows(uint64_t seed, int64_t n, int32_t k, int64_t* rows) {
  if (k <= 0 || n < k) return -1;
  int64_t cap = 1;
  while (cap < 4 * (int64_t)k) cap <<= 1;
  int64_t* keys = (int64_t*)malloc(sizeof(int64_t) * (size_t)cap);
  int64_t* vals = (int64_t*)malloc(sizeof(int64_t) * (size_t)cap);
  for (int64_t i = 0; i < cap; ++i) keys[i] = -1;
#define SLOT(key) ({ int64_t h_ = (int64_t)(((uint64_t)(key) * 0x9E3779B97F4A7C15ull) & (uint64_t)(cap - 1)); \
                     while (keys[h_] != -1 && keys[h_] != (key)) h_ = (h_ + 1) & (cap - 1); h_; })
  for (int32_t j = 0; j < k; ++j) {
    uint32_t w[4];
    draw(seed, 5, (uint64_t)j, 0, w);
    uint64_t r64 = ((uint64_t)w[1] << 32) | w[0];
    int64_t r = j + (int64_t)(r64 % (uint64_t)(n - j));
    int64_t sj = SLOT(j), sr = SLOT(r);
    int64_t vj = keys[sj] == -1 ? j : vals[sj];
    int64_t vr = keys[sr] == -1 ? r : vals[sr];
    keys[sj] = j; vals[sj] = vr;
    sr = SLOT(r);
    keys[sr] = r; vals[sr] = vj;
    rows[j] = vr;
  }
#undef SLOT
  free(keys); free(vals);
  return 0;
}
