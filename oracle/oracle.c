/*
 * CPU checker for the diagonal-covariance GMM EM iteration: TEST
 * INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the benchmark's
 * CPU-baseline leg use it; the GPU library never calls, links or loads it.
 *
 * Everything is plain fp64 loops over points and components, written from
 * the paper's statement of the model (Sec. 2) with the diagonal covariance
 * the build targets in place of the paper's isotropic sigma_k^2 I:
 *
 *   log-density  l_ik = log pi_k - 1/2 sum_d [ log(2 pi var_kd) + (x_id - mu_kd)^2 / var_kd ]
 *                (the mixture density of Sec. 2 with a diagonal covariance; the
 *                 per-component constant log pi_k - 1/2 sum_d log(2 pi var_kd)
 *                 is evaluated once per component)
 *   normaliser   log Z_i = m_i + log sum_k exp(l_ik - m_i),  m_i = max_k l_ik
 *                (log-sum-exp form of the responsibility denominator, Sec. 2)
 *   responsib.   r_ik = exp(l_ik - log Z_i)                       (Sec. 2)
 *   log-lik.     LL = sum_i log Z_i                                 (Sec. 2)
 *   statistics   N_k = sum_i r_ik            (Eq. Nk)
 *                S_kd = sum_i r_ik x_id     (numerator of Eq. muk)
 *                Q_kd = sum_i r_ik x_id^2   (raw second moment)
 *   M-step       pi_k = N_k / N,  mu_kd = S_kd / N_k   (Eqs. Nk, muk)
 *                var_kd = max(var_floor, sum_i r_ik (x_id - mu_kd)^2 / N_k)
 *                (Eq. sig written per dimension, with the NEW mean, evaluated
 *                 by a second sweep over the data; the floor is this build's
 *                 reading, the paper states none)
 *                dead component (N_k == 0 exactly): keep mu_k and var_k,
 *                set pi_k = 0, so l_ik = -inf from then on.
 *   top-m        components ordered by l_ik, largest first, ties to the
 *                lower index; rank 1 always kept (Sec. 4.2), rank j > 1 kept
 *                iff r_ik > tau (Sec. 4.3); empty slots are -1 / 0.
 *
 * Points are split into a fixed number of contiguous slots (independent of
 * the core count); each slot sums its points in order, and slot partials
 * are added in slot order, so results do not depend on thread timing.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_SLOTS 16

typedef struct {
  int32_t d, k;
  double* mu;    /* k*d */
  double* ivar;  /* k*d, 1/var */
  double* cst;   /* k: log pi_k - 1/2 sum_d log(2 pi var_kd), -inf if pi_k == 0 */
} params;

static const double LOG_2PI = 1.8378770664093454835606594728112;

static void params_init(params* p, int32_t d, int32_t k, const float* w, const float* mu,
                        const float* var) {
  p->d = d; p->k = k;
  p->mu = (double*)malloc(sizeof(double) * (size_t)k * d);
  p->ivar = (double*)malloc(sizeof(double) * (size_t)k * d);
  p->cst = (double*)malloc(sizeof(double) * (size_t)k);
  for (int32_t c = 0; c < k; ++c) {
    double s = 0.0;
    for (int32_t j = 0; j < d; ++j) {
      double v = (double)var[(int64_t)c * d + j];
      p->mu[(int64_t)c * d + j] = (double)mu[(int64_t)c * d + j];
      p->ivar[(int64_t)c * d + j] = 1.0 / v;
      s += LOG_2PI + log(v);
    }
    p->cst[c] = (w[c] > 0.0f) ? log((double)w[c]) - 0.5 * s : -INFINITY;
  }
}

static void params_free(params* p) { free(p->mu); free(p->ivar); free(p->cst); }

/* l[c] for one point, direct form. */
static void logdens(const params* p, const float* x, double* l) {
  const int32_t d = p->d;
  for (int32_t c = 0; c < p->k; ++c) {
    if (p->cst[c] == -INFINITY) { l[c] = -INFINITY; continue; }
    const double* mu = p->mu + (int64_t)c * d;
    const double* iv = p->ivar + (int64_t)c * d;
    double q = 0.0;
    for (int32_t j = 0; j < d; ++j) {
      double t = (double)x[j] - mu[j];
      q += t * t * iv[j];
    }
    l[c] = p->cst[c] - 0.5 * q;
  }
}

/* log Z = max + log sum exp(l - max), the plain two-pass form. */
static double lse(const double* l, int32_t k) {
  double m = -INFINITY;
  for (int32_t c = 0; c < k; ++c) if (l[c] > m) m = l[c];
  if (m == -INFINITY) return -INFINITY;
  double s = 0.0;
  for (int32_t c = 0; c < k; ++c) s += exp(l[c] - m);
  return m + log(s);
}

/* ------------------------------------------------------------------ */
/* Sweep: per slot, accumulate N, S, Q, LL (mode 0) or V about mu2 (mode 1). */

typedef struct {
  const params* p;
  const float* x;
  int64_t i0, i1;
  int mode;
  const double* mu2; /* mode 1: the new means */
  double *nk, *s, *q, *v, ll;
  double* logz;      /* optional per-point log Z (mode 0) */
} sweep_job;

static void* sweep_worker(void* arg) {
  sweep_job* jb = (sweep_job*)arg;
  const params* p = jb->p;
  const int32_t d = p->d, k = p->k;
  double* l = (double*)malloc(sizeof(double) * (size_t)k);
  jb->ll = 0.0;
  for (int64_t i = jb->i0; i < jb->i1; ++i) {
    const float* x = jb->x + i * (int64_t)d;
    logdens(p, x, l);
    double lz = lse(l, k);
    if (jb->mode == 0) {
      jb->ll += lz;
      if (jb->logz) jb->logz[i] = lz;
    }
    for (int32_t c = 0; c < k; ++c) {
      double r = exp(l[c] - lz);
      if (r == 0.0) continue; /* adds nothing to any sum */
      if (jb->mode == 0) {
        jb->nk[c] += r;
        for (int32_t j = 0; j < d; ++j) {
          double xv = (double)x[j];
          jb->s[(int64_t)c * d + j] += r * xv;
          jb->q[(int64_t)c * d + j] += r * xv * xv;
        }
      } else {
        for (int32_t j = 0; j < d; ++j) {
          double t = (double)x[j] - jb->mu2[(int64_t)c * d + j];
          jb->v[(int64_t)c * d + j] += r * t * t;
        }
      }
    }
  }
  free(l);
  return NULL;
}

static void run_sweep(const params* p, const float* x, int64_t n, int mode, const double* mu2,
                      double* nk, double* s, double* q, double* v, double* ll, double* logz,
                      int32_t nthreads) {
  const int32_t d = p->d, k = p->k;
  const size_t kd = (size_t)k * d;
  sweep_job jobs[ORACLE_SLOTS];
  double* buf = (double*)calloc((size_t)ORACLE_SLOTS * (k + 2 * kd), sizeof(double));
  for (int t = 0; t < ORACLE_SLOTS; ++t) {
    sweep_job* jb = &jobs[t];
    memset(jb, 0, sizeof(*jb));
    jb->p = p; jb->x = x; jb->mode = mode; jb->mu2 = mu2; jb->logz = logz;
    jb->i0 = n * t / ORACLE_SLOTS;
    jb->i1 = n * (t + 1) / ORACLE_SLOTS;
    double* b = buf + (size_t)t * (k + 2 * kd);
    jb->nk = b; jb->s = b + k; jb->q = b + k + kd; jb->v = b + k;
  }
  if (nthreads < 1) nthreads = 1;
  if (nthreads > ORACLE_SLOTS) nthreads = ORACLE_SLOTS;
  /* slots are run in waves of nthreads; the slot -> points map is fixed */
  for (int t0 = 0; t0 < ORACLE_SLOTS; t0 += nthreads) {
    pthread_t th[ORACLE_SLOTS];
    int t1 = t0 + nthreads < ORACLE_SLOTS ? t0 + nthreads : ORACLE_SLOTS;
    for (int t = t0; t < t1; ++t) pthread_create(&th[t], NULL, sweep_worker, &jobs[t]);
    for (int t = t0; t < t1; ++t) pthread_join(th[t], NULL);
  }
  for (int t = 0; t < ORACLE_SLOTS; ++t) {
    const sweep_job* jb = &jobs[t];
    if (mode == 0) {
      for (int32_t c = 0; c < k; ++c) nk[c] += jb->nk[c];
      for (size_t e = 0; e < kd; ++e) { s[e] += jb->s[e]; q[e] += jb->q[e]; }
      *ll += jb->ll;
    } else {
      for (size_t e = 0; e < kd; ++e) v[e] += jb->v[e];
    }
  }
  free(buf);
}

/*
 * E-step statistics at parameters (w, mu, var): ADDS N_k, S, Q and LL into
 * the caller's fp64 arrays (so row slices can be summed).  logz (optional)
 * receives log Z_i per point.
 */
void oracle_estep(const float* x, int64_t n, int32_t d, int32_t k, const float* w, const float* mu,
                  const float* var, double* nk, double* s, double* q, double* ll, double* logz,
                  int32_t nthreads) {
  params p;
  params_init(&p, d, k, w, mu, var);
  run_sweep(&p, x, n, 0, NULL, nk, s, q, NULL, ll, logz, nthreads);
  params_free(&p);
}

/*
 * One full EM iteration at Theta_t = (w, mu, var) over all n points:
 * E-step statistics, the M-step of Eqs. Nk / muk / sig (second sweep for the
 * variance about the new mean), the floor and the dead rule.  Writes
 * Theta_{t+1} to (w_out, mu_out, var_out) as fp64, LL(Theta_t) to *ll, and
 * the statistics to nk / s / q (overwritten).
 */
void oracle_iterate(const float* x, int64_t n, int32_t d, int32_t k, const float* w, const float* mu,
                    const float* var, double var_floor, double* w_out, double* mu_out,
                    double* var_out, double* nk, double* s, double* q, double* ll,
                    int32_t nthreads) {
  params p;
  params_init(&p, d, k, w, mu, var);
  const size_t kd = (size_t)k * d;
  memset(nk, 0, sizeof(double) * (size_t)k);
  memset(s, 0, sizeof(double) * kd);
  memset(q, 0, sizeof(double) * kd);
  *ll = 0.0;
  run_sweep(&p, x, n, 0, NULL, nk, s, q, NULL, ll, NULL, nthreads);
  for (int32_t c = 0; c < k; ++c) {
    for (int32_t j = 0; j < d; ++j) {
      size_t e = (size_t)c * d + j;
      mu_out[e] = nk[c] > 0.0 ? s[e] / nk[c] : (double)mu[e];
    }
  }
  double* v = (double*)calloc(kd, sizeof(double));
  run_sweep(&p, x, n, 1, mu_out, NULL, NULL, NULL, v, NULL, NULL, nthreads);
  for (int32_t c = 0; c < k; ++c) {
    w_out[c] = nk[c] / (double)n;
    for (int32_t j = 0; j < d; ++j) {
      size_t e = (size_t)c * d + j;
      if (nk[c] > 0.0) {
        double vv = v[e] / nk[c];
        var_out[e] = vv > var_floor ? vv : var_floor;
      } else {
        var_out[e] = (double)var[e];
      }
    }
  }
  free(v);
  params_free(&p);
}

/* Log-densities l[rows x k] and log Z[rows] of the given rows (fp64). */
void oracle_logdens(const float* x, int64_t n, int32_t d, int32_t k, const float* w,
                    const float* mu, const float* var, double* l, double* logz) {
  params p;
  params_init(&p, d, k, w, mu, var);
  for (int64_t i = 0; i < n; ++i) {
    double* li = l + i * (int64_t)k;
    logdens(&p, x + i * (int64_t)d, li);
    if (logz) logz[i] = lse(li, k);
  }
  params_free(&p);
}

typedef struct {
  const params* p;
  const float* x;
  int64_t i0, i1;
  int32_t m, mr;
  double tau;
  int32_t* idx;
  float* resp;
  int32_t* ridx;  /* optional: top-mr indices per point (no tau rule) */
  double* rresp;  /* optional: their fp64 responsibilities */
} assign_job;

static void* assign_worker(void* arg) {
  assign_job* jb = (assign_job*)arg;
  const params* p = jb->p;
  const int32_t k = p->k;
  double* l = (double*)malloc(sizeof(double) * (size_t)k);
  int32_t top[64];
  for (int64_t i = jb->i0; i < jb->i1; ++i) {
    logdens(p, jb->x + i * (int64_t)p->d, l);
    double lz = lse(l, k);
    int32_t want = jb->m > jb->mr ? jb->m : jb->mr;
    if (want > k) want = k;
    /* selection of the top `want`: larger l first, equal l -> lower index */
    for (int32_t j = 0; j < want; ++j) {
      int32_t best = -1;
      for (int32_t c = 0; c < k; ++c) {
        int taken = 0;
        for (int32_t t = 0; t < j; ++t) if (top[t] == c) { taken = 1; break; }
        if (taken) continue;
        if (best < 0 || l[c] > l[best]) best = c;
      }
      top[j] = best;
    }
    for (int32_t j = 0; j < jb->m; ++j) {
      int64_t o = i * (int64_t)jb->m + j;
      if (j < want && top[j] >= 0) {
        double r = exp(l[top[j]] - lz);
        if (j == 0 || r > jb->tau) { jb->idx[o] = top[j]; jb->resp[o] = (float)r; continue; }
      }
      jb->idx[o] = -1;
      jb->resp[o] = 0.0f;
    }
    if (jb->ridx) {
      for (int32_t j = 0; j < jb->mr; ++j) {
        int64_t o = i * (int64_t)jb->mr + j;
        if (j < want) { jb->ridx[o] = top[j]; jb->rresp[o] = exp(l[top[j]] - lz); }
        else { jb->ridx[o] = -1; jb->rresp[o] = 0.0; }
      }
    }
  }
  free(l);
  return NULL;
}

/*
 * Top-m multi-assignment (Sec. 4.2-4.3).  idx/resp are n*m.  If ridx/rresp
 * are given they receive the top-mr components and their fp64
 * responsibilities without the tau rule (tests use them for margins).
 * m and mr must each be at most 64.
 */
int oracle_assign_topk(const float* x, int64_t n, int32_t d, int32_t k, const float* w,
                       const float* mu, const float* var, int32_t m, double tau, int32_t* idx,
                       float* resp, int32_t mr, int32_t* ridx, double* rresp, int32_t nthreads) {
  if (m < 1 || m > 64 || mr < 0 || mr > 64) return -1;
  params p;
  params_init(&p, d, k, w, mu, var);
  if (nthreads < 1) nthreads = 1;
  if (nthreads > ORACLE_SLOTS) nthreads = ORACLE_SLOTS;
  assign_job jobs[ORACLE_SLOTS];
  pthread_t th[ORACLE_SLOTS];
  for (int t = 0; t < nthreads; ++t) {
    assign_job* jb = &jobs[t];
    jb->p = &p; jb->x = x; jb->m = m; jb->mr = mr; jb->tau = tau;
    jb->i0 = n * t / nthreads; jb->i1 = n * (t + 1) / nthreads;
    jb->idx = idx; jb->resp = resp; jb->ridx = ridx; jb->rresp = rresp;
    pthread_create(&th[t], NULL, assign_worker, jb);
  }
  for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  params_free(&p);
  return 0;
}

/* ------------------------------------------------------------------ */
/*
 * The paper's own model (Sec. 2): isotropic components N(mu_k, var_k I) with
 * one scalar variance per component.  Written on its own from the model,
 * not through the diagonal code above:
 *
 *   log-density  l_ik = log pi_k - D/2 log(2 pi var_k) - ||x_i - mu_k||^2 / (2 var_k)
 *   statistics   N_k = sum_i r_ik,  S_kd = sum_i r_ik x_id,
 *                Q_k = sum_i r_ik ||x_i||^2   (raw, scalar per component)
 *   M-step       pi_k = N_k / N,  mu_k = S_k / N_k                     (Eqs. Nk, muk)
 *                var_k = max(var_floor, sum_i r_ik ||x_i - mu_k||^2 / (D N_k))  (Eq. sig,
 *                the new mean, a second sweep); dead rule as above.
 */
typedef struct {
  int32_t d, k;
  const float* mu;   /* k*d, fp32 as given */
  double* ivar;      /* k: 1 / var_k */
  double* cst;       /* k: log pi_k - D/2 log(2 pi var_k), -inf if pi_k == 0 */
} iso_params;

static void iso_init(iso_params* p, int32_t d, int32_t k, const float* w, const float* mu,
                     const float* var) {
  p->d = d; p->k = k; p->mu = mu;
  p->ivar = (double*)malloc(sizeof(double) * (size_t)k);
  p->cst = (double*)malloc(sizeof(double) * (size_t)k);
  for (int32_t c = 0; c < k; ++c) {
    const double v = (double)var[c];
    p->ivar[c] = 1.0 / v;
    p->cst[c] = (w[c] > 0.0f) ? log((double)w[c]) - 0.5 * (double)d * (LOG_2PI + log(v))
                              : -INFINITY;
  }
}

static void iso_free(iso_params* p) { free(p->ivar); free(p->cst); }

static void iso_logdens(const iso_params* p, const float* x, double* l) {
  for (int32_t c = 0; c < p->k; ++c) {
    if (p->cst[c] == -INFINITY) { l[c] = -INFINITY; continue; }
    const float* mu = p->mu + (int64_t)c * p->d;
    double dist = 0.0;
    for (int32_t j = 0; j < p->d; ++j) {
      const double t = (double)x[j] - (double)mu[j];
      dist += t * t;
    }
    l[c] = p->cst[c] - 0.5 * dist * p->ivar[c];
  }
}

typedef struct {
  const iso_params* p;
  const float* x;
  int64_t i0, i1;
  int mode;              /* 0: N, S, Q, LL; 1: V about mu2 */
  const double* mu2;
  double *nk, *s, *q, *v, ll;
} iso_job;

static void* iso_worker(void* arg) {
  iso_job* jb = (iso_job*)arg;
  const iso_params* p = jb->p;
  const int32_t d = p->d, k = p->k;
  double* l = (double*)malloc(sizeof(double) * (size_t)k);
  jb->ll = 0.0;
  for (int64_t i = jb->i0; i < jb->i1; ++i) {
    const float* x = jb->x + i * (int64_t)d;
    iso_logdens(p, x, l);
    const double lz = lse(l, k);
    if (jb->mode == 0) jb->ll += lz;
    double xx = 0.0;
    for (int32_t j = 0; j < d; ++j) xx += (double)x[j] * (double)x[j];
    for (int32_t c = 0; c < k; ++c) {
      const double r = exp(l[c] - lz);
      if (r == 0.0) continue;
      if (jb->mode == 0) {
        jb->nk[c] += r;
        jb->q[c] += r * xx;
        for (int32_t j = 0; j < d; ++j) jb->s[(int64_t)c * d + j] += r * (double)x[j];
      } else {
        double dist = 0.0;
        for (int32_t j = 0; j < d; ++j) {
          const double t = (double)x[j] - jb->mu2[(int64_t)c * d + j];
          dist += t * t;
        }
        jb->v[c] += r * dist;
      }
    }
  }
  free(l);
  return NULL;
}

static void iso_sweep(const iso_params* p, const float* x, int64_t n, int mode, const double* mu2,
                      double* nk, double* s, double* q, double* v, double* ll, int32_t nthreads) {
  const int32_t d = p->d, k = p->k;
  const size_t kd = (size_t)k * d, per = (size_t)3 * k + kd;
  iso_job jobs[ORACLE_SLOTS];
  double* buf = (double*)calloc((size_t)ORACLE_SLOTS * per, sizeof(double));
  for (int t = 0; t < ORACLE_SLOTS; ++t) {
    iso_job* jb = &jobs[t];
    memset(jb, 0, sizeof(*jb));
    jb->p = p; jb->x = x; jb->mode = mode; jb->mu2 = mu2;
    jb->i0 = n * t / ORACLE_SLOTS;
    jb->i1 = n * (t + 1) / ORACLE_SLOTS;
    double* b = buf + (size_t)t * per;
    jb->nk = b; jb->q = b + k; jb->v = b + 2 * k; jb->s = b + 3 * k;
  }
  if (nthreads < 1) nthreads = 1;
  if (nthreads > ORACLE_SLOTS) nthreads = ORACLE_SLOTS;
  for (int t0 = 0; t0 < ORACLE_SLOTS; t0 += nthreads) {
    pthread_t th[ORACLE_SLOTS];
    int t1 = t0 + nthreads < ORACLE_SLOTS ? t0 + nthreads : ORACLE_SLOTS;
    for (int t = t0; t < t1; ++t) pthread_create(&th[t], NULL, iso_worker, &jobs[t]);
    for (int t = t0; t < t1; ++t) pthread_join(th[t], NULL);
  }
  for (int t = 0; t < ORACLE_SLOTS; ++t) {
    const iso_job* jb = &jobs[t];
    if (mode == 0) {
      for (int32_t c = 0; c < k; ++c) { nk[c] += jb->nk[c]; q[c] += jb->q[c]; }
      for (size_t e = 0; e < kd; ++e) s[e] += jb->s[e];
      *ll += jb->ll;
    } else {
      for (int32_t c = 0; c < k; ++c) v[c] += jb->v[c];
    }
  }
  free(buf);
}

/* Isotropic E-step statistics: ADDS N_k, S (k*d), Q (k) and LL. */
void oracle_iso_estep(const float* x, int64_t n, int32_t d, int32_t k, const float* w,
                      const float* mu, const float* var, double* nk, double* s, double* q,
                      double* ll, int32_t nthreads) {
  iso_params p;
  iso_init(&p, d, k, w, mu, var);
  iso_sweep(&p, x, n, 0, NULL, nk, s, q, NULL, ll, nthreads);
  iso_free(&p);
}

/* One isotropic EM iteration; Theta_{t+1} as fp64, statistics overwritten. */
void oracle_iso_iterate(const float* x, int64_t n, int32_t d, int32_t k, const float* w,
                        const float* mu, const float* var, double var_floor, double* w_out,
                        double* mu_out, double* var_out, double* nk, double* s, double* q,
                        double* ll, int32_t nthreads) {
  iso_params p;
  iso_init(&p, d, k, w, mu, var);
  const size_t kd = (size_t)k * d;
  memset(nk, 0, sizeof(double) * (size_t)k);
  memset(q, 0, sizeof(double) * (size_t)k);
  memset(s, 0, sizeof(double) * kd);
  *ll = 0.0;
  iso_sweep(&p, x, n, 0, NULL, nk, s, q, NULL, ll, nthreads);
  for (int32_t c = 0; c < k; ++c)
    for (int32_t j = 0; j < d; ++j) {
      const size_t e = (size_t)c * d + j;
      mu_out[e] = nk[c] > 0.0 ? s[e] / nk[c] : (double)mu[e];
    }
  double* v = (double*)calloc((size_t)k, sizeof(double));
  iso_sweep(&p, x, n, 1, mu_out, NULL, NULL, NULL, v, NULL, nthreads);
  for (int32_t c = 0; c < k; ++c) {
    w_out[c] = nk[c] / (double)n;
    if (nk[c] > 0.0) {
      const double vv = v[c] / ((double)d * nk[c]);
      var_out[c] = vv > var_floor ? vv : var_floor;
    } else {
      var_out[c] = (double)var[c];
    }
  }
  free(v);
  iso_free(&p);
}

/* ------------------------------------------------------------------ */
/*
 * k-means++ seeding (Arthur and Vassilvitskii, SODA 2007; the initialisation
 * the paper compares with its warm start, Sec. 4.5 and App. C): the first
 * centre is row floor(u_0 N); centre t is drawn with probability
 * proportional to D(x)^2, the squared distance of a row to its nearest chosen
 * centre, by inversion of u_t against the running sum of D^2 over the rows in
 * order: the first row whose running sum exceeds u_t times the total.  The
 * uniforms u are inputs.  When the total is 0 (every row sits on a chosen
 * centre) centre t is row floor(u_t N).
 *
 * margin[t] (optional) is how far the target u_t * total lies inside the
 * picked row's interval [running sum before it, running sum after it],
 * divided by the total; +inf for centre 0 and for a zero total.  A method
 * whose running sums differ from these by rounding alone picks the same row
 * whenever the difference stays below that margin.
 */
static double kpp_dist(const float* x, const float* c, int32_t d) {
  double acc = 0.0;
  for (int32_t j = 0; j < d; ++j) {
    const double t = (double)x[j] - (double)c[j];
    acc += t * t;
  }
  return acc;
}

static int64_t kpp_first(double u, int64_t n) {
  int64_t i = (int64_t)(u * (double)n);
  return i < 0 ? 0 : (i >= n ? n - 1 : i);
}

/* idx[k]: the chosen rows; centers[k*d] (may be NULL): their coordinates;
   margin[k] (may be NULL): see above. */
void oracle_kmeanspp(const float* x, int64_t n, int32_t d, int32_t k, const double* u,
                     int64_t* idx, float* centers, double* margin) {
  double* dist = (double*)malloc(sizeof(double) * (size_t)n);
  for (int64_t i = 0; i < n; ++i) dist[i] = INFINITY;
  for (int32_t t = 0; t < k; ++t) {
    int64_t pick = -1;
    double mg = INFINITY;
    if (t > 0) {
      double total = 0.0;
      for (int64_t i = 0; i < n; ++i) total += dist[i];
      if (total > 0.0) {
        /* the running sum below repeats the total's additions, so it reaches
           the total and, u_t < 1, passes the target at some row */
        const double target = u[t] * total;
        double run = 0.0;
        for (int64_t i = 0; i < n; ++i) {
          const double before = run;
          run += dist[i];
          if (run > target) {
            pick = i;
            mg = fmin(target - before, run - target) / total;
            break;
          }
        }
      }
    }
    if (pick < 0) pick = kpp_first(u[t], n);
    idx[t] = pick;
    if (margin) margin[t] = mg;
    const float* c = x + pick * (int64_t)d;
    if (centers) memcpy(centers + (int64_t)t * d, c, sizeof(float) * (size_t)d);
    for (int64_t i = 0; i < n; ++i) {
      const double dd = kpp_dist(x + i * (int64_t)d, c, d);
      if (dd < dist[i]) dist[i] = dd;
    }
  }
  free(dist);
}

/* ------------------------------------------------------------------ */
/*
 * k-means warm start (the paper's initialisation, Sec. 4.4 and App. C: Lloyd iterations
 * from given centres, then EM from the result).  An iteration assigns every
 * row to its nearest centre (squared Euclidean distance summed in fp64 over
 * the dimensions in order; ties to the lower index) and moves every centre
 * to the mean of its rows (a centre without rows stays).  After n_iters
 * iterations a last assignment gives the mixture the EM starts from, the
 * M-step of Eqs. Nk / muk / sig with hard responsibilities:
 *   pi_k = N_k / N, mu_k = mean of its rows, var_kd = max(var_floor,
 *   sum over its rows (x_d - mu_kd)^2 / N_k) (about the new mean), and for a
 *   centre without rows: pi_k = 0, mu_k its centre, var_k as given.
 * centres [k*d] (in: initial, out: after n_iters iterations), var [k*d] (in:
 * for centres without rows), outputs w_out, mu_out, var_out (fp64) and the
 * final assignment (int32).
 */
static int32_t km_nearest(const float* x, const double* c, int32_t d, int32_t k) {
  int32_t best = 0;
  double bd = INFINITY;
  for (int32_t q = 0; q < k; ++q) {
    double s = 0.0;
    for (int32_t j = 0; j < d; ++j) {
      const double t = (double)x[j] - c[(int64_t)q * d + j];
      s += t * t;
    }
    if (s < bd) { bd = s; best = q; }
  }
  return best;
}

void oracle_kmeans(const float* x, int64_t n, int32_t d, int32_t k, int32_t n_iters,
                   double var_floor, const float* centres_in, const float* var_in, double* centres,
                   double* w_out, double* mu_out, double* var_out, int32_t* assign) {
  const size_t kd = (size_t)k * d;
  double* sum = (double*)malloc(sizeof(double) * kd);
  double* cnt = (double*)malloc(sizeof(double) * (size_t)k);
  for (size_t e = 0; e < kd; ++e) centres[e] = (double)centres_in[e];
  for (int32_t it = 0; it <= n_iters; ++it) {
    for (int64_t i = 0; i < n; ++i) assign[i] = km_nearest(x + i * (int64_t)d, centres, d, k);
    memset(sum, 0, sizeof(double) * kd);
    memset(cnt, 0, sizeof(double) * (size_t)k);
    for (int64_t i = 0; i < n; ++i) {
      const int32_t q = assign[i];
      cnt[q] += 1.0;
      for (int32_t j = 0; j < d; ++j) sum[(int64_t)q * d + j] += (double)x[i * (int64_t)d + j];
    }
    if (it == n_iters) break;    /* the last assignment feeds the mixture below */
    for (int32_t q = 0; q < k; ++q)
      if (cnt[q] > 0.0)
        for (int32_t j = 0; j < d; ++j)
          centres[(int64_t)q * d + j] = (double)(float)(sum[(int64_t)q * d + j] / cnt[q]);
  }
  for (int32_t q = 0; q < k; ++q) {
    w_out[q] = cnt[q] / (double)n;
    for (int32_t j = 0; j < d; ++j) {
      const size_t e = (size_t)q * d + j;
      mu_out[e] = cnt[q] > 0.0 ? sum[e] / cnt[q] : centres[e];
      var_out[e] = 0.0;
    }
  }
  for (int64_t i = 0; i < n; ++i) {
    const int32_t q = assign[i];
    for (int32_t j = 0; j < d; ++j) {
      const double t = (double)x[i * (int64_t)d + j] - mu_out[(int64_t)q * d + j];
      var_out[(int64_t)q * d + j] += t * t;
    }
  }
  for (int32_t q = 0; q < k; ++q)
    for (int32_t j = 0; j < d; ++j) {
      const size_t e = (size_t)q * d + j;
      if (cnt[q] > 0.0) {
        const double v = var_out[e] / cnt[q];
        var_out[e] = v > var_floor ? v : var_floor;
      } else {
        var_out[e] = (double)var_in[e];
      }
    }
  free(sum);
  free(cnt);
}
