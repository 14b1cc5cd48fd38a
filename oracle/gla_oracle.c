/*
 * gla_oracle.c -- CPU fp64 oracle for the gated linear attention (GLA) layer.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, obviously correct
 * definition that the GPU path is checked against.  Only the tests, the smoke
 * check and the benchmark's CPU-baseline leg may load it; the product path
 * never does.  It shares no code, header or constant with the HIP library.
 *
 * What it computes (paper, Sec. 4.1, Eq. 3; per batch row b and head h):
 *
 *     S_0 = S0 (or zero)                         -- initial state (Sec. 2.2)
 *     S_t = Diag(alpha_t) S_{t-1} + k_t^T v_t     -- alpha_t = exp(log_alpha_t)
 *     o_t = q_t S_t
 *
 * with q_t, k_t, log_alpha_t in R^{d_k}, v_t, o_t in R^{d_v} and S_t in
 * R^{d_k x d_v}.  The gate decays the previous state before the outer product
 * of step t is added, so step t itself enters o_t with weight one.
 *
 * The backward is reverse-mode differentiation of exactly that loop
 * (back-propagation through time).  The loss seen from outside is
 *     L = sum_t <o_t, dO_t> + <S_T, dS_T>
 * and, walking t = T..1 with G the gradient w.r.t. S_t:
 *     G      += q_t^T dO_t
 *     dq_t    = S_t dO_t^T
 *     dk_t    = G v_t^T
 *     dv_t    = k_t G
 *     dlogalpha_t[a] = alpha_t[a] * sum_j G[a,j] S_{t-1}[a,j]
 *                      (the direct gate gradient (S_{t-1} (.) dS_t) 1 of
 *                       Sec. 4.3, chained through alpha = exp(log_alpha))
 *     G       = Diag(alpha_t) G                   -- gradient w.r.t. S_{t-1}
 * and dS0 = G at the end.  States are checkpointed every `ckpt` steps and
 * recomputed inside each segment, which bounds memory at long T.
 *
 * Layout: every tensor is contiguous row-major; q, k, log_alpha, dq, dk,
 * dlog_alpha are [BH, T, d_k]; v, o, dO, dv are [BH, T, d_v]; states are
 * [BH, d_k, d_v].  BH is batch*heads flattened (heads are independent).
 * Optional pointers may be NULL (S0, dS_T: zero; S_T, dS0: not wanted).
 * Work is split over host threads by head (and, in the forward, by column
 * block, since the columns of S evolve independently).
 * Return value: 0 on success, -1 on bad arguments, -2 on allocation failure.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int64_t BH, T, K, V;
  const double *q, *k, *v, *la, *S0, *dO, *dST;
  double *o, *ST, *dq, *dk, *dv, *dla, *dS0;
  int64_t ckpt;
  int64_t n_items, col_block;
  int64_t next;             /* next work item, taken under the mutex */
  pthread_mutex_t mu;
  int status;
} job_t;

static int64_t take_item(job_t *J) {
  pthread_mutex_lock(&J->mu);
  int64_t it = J->next < J->n_items ? J->next++ : -1;
  pthread_mutex_unlock(&J->mu);
  return it;
}

/* ---------------------------------------------------------------- forward */

static void fwd_item(job_t *J, int64_t item) {
  const int64_t T = J->T, K = J->K, V = J->V, cb = J->col_block;
  const int64_t nblk = (V + cb - 1) / cb;
  const int64_t h = item / nblk, j0 = (item % nblk) * cb;
  const int64_t w = (j0 + cb <= V) ? cb : V - j0;
  const double *q = J->q + h * T * K, *k = J->k + h * T * K;
  const double *la = J->la + h * T * K, *v = J->v + h * T * V;
  double *o = J->o + h * T * V;
  double *S = (double *)calloc((size_t)(K * w), sizeof(double));
  if (!S) { J->status = -2; return; }
  if (J->S0)
    for (int64_t a = 0; a < K; ++a)
      for (int64_t j = 0; j < w; ++j) S[a * w + j] = J->S0[h * K * V + a * V + j0 + j];
  for (int64_t t = 0; t < T; ++t) {
    const double *vt = v + t * V + j0;
    for (int64_t a = 0; a < K; ++a) {          /* S_t = Diag(alpha_t) S_{t-1} + k_t^T v_t */
      const double al = exp(la[t * K + a]), ka = k[t * K + a];
      double *Sa = S + a * w;
      for (int64_t j = 0; j < w; ++j) Sa[j] = al * Sa[j] + ka * vt[j];
    }
    double *ot = o + t * V + j0;               /* o_t = q_t S_t */
    for (int64_t j = 0; j < w; ++j) ot[j] = 0.0;
    for (int64_t a = 0; a < K; ++a) {
      const double qa = q[t * K + a];
      const double *Sa = S + a * w;
      for (int64_t j = 0; j < w; ++j) ot[j] += qa * Sa[j];
    }
  }
  if (J->ST)
    for (int64_t a = 0; a < K; ++a)
      for (int64_t j = 0; j < w; ++j) J->ST[h * K * V + a * V + j0 + j] = S[a * w + j];
  free(S);
}

static void *fwd_worker(void *arg) {
  job_t *J = (job_t *)arg;
  for (int64_t it; (it = take_item(J)) >= 0;) fwd_item(J, it);
  return NULL;
}

/* --------------------------------------------------------------- backward */

/* One decay-and-add step: dst = Diag(exp(la_t)) src + k_t^T v_t. */
static void step_state(double *dst, const double *src, const double *kt, const double *lat,
                       const double *vt, int64_t K, int64_t V) {
  for (int64_t a = 0; a < K; ++a) {
    const double al = exp(lat[a]), ka = kt[a];
    for (int64_t j = 0; j < V; ++j) dst[a * V + j] = al * src[a * V + j] + ka * vt[j];
  }
}

static void bwd_item(job_t *J, int64_t h) {
  const int64_t T = J->T, K = J->K, V = J->V, ck = J->ckpt, KV = K * V;
  const double *q = J->q + h * T * K, *k = J->k + h * T * K, *la = J->la + h * T * K;
  const double *v = J->v + h * T * V, *dO = J->dO + h * T * V;
  double *dq = J->dq + h * T * K, *dk = J->dk + h * T * K, *dla = J->dla + h * T * K;
  double *dv = J->dv + h * T * V;
  const int64_t nck = (T + ck - 1) / ck;               /* segments [s*ck, min(T,(s+1)*ck)) */
  double *ckp = (double *)calloc((size_t)((nck > 0 ? nck : 1) * KV), sizeof(double)); /* S at segment starts */
  double *seg = (double *)malloc((size_t)((ck + 1) * KV) * sizeof(double));
  double *G = (double *)calloc((size_t)KV, sizeof(double));
  if (!ckp || !seg || !G) { free(ckp); free(seg); free(G); J->status = -2; return; }

  /* Forward pass keeping S_{s*ck} (state before step s*ck+1, 1-based). */
  if (J->S0) memcpy(ckp, J->S0 + h * KV, (size_t)KV * sizeof(double));
  memcpy(seg, ckp, (size_t)KV * sizeof(double));
  for (int64_t s = 0; s < nck; ++s) {
    if (s > 0) memcpy(ckp + s * KV, seg, (size_t)KV * sizeof(double));
    const int64_t t0 = s * ck, t1 = (t0 + ck < T) ? t0 + ck : T;
    for (int64_t t = t0; t < t1; ++t) {
      step_state(seg + KV, seg, k + t * K, la + t * K, v + t * V, K, V);
      memcpy(seg, seg + KV, (size_t)KV * sizeof(double));
    }
  }
  /* seg[0..KV) now holds S_T. */
  if (J->dST) memcpy(G, J->dST + h * KV, (size_t)KV * sizeof(double));

  for (int64_t s = nck - 1; s >= 0; --s) {
    const int64_t t0 = s * ck, t1 = (t0 + ck < T) ? t0 + ck : T, n = t1 - t0;
    /* Recompute seg[m] = state after m steps of this segment, m = 0..n. */
    memcpy(seg, ckp + s * KV, (size_t)KV * sizeof(double));
    for (int64_t m = 0; m < n; ++m)
      step_state(seg + (m + 1) * KV, seg + m * KV, k + (t0 + m) * K, la + (t0 + m) * K,
                 v + (t0 + m) * V, K, V);
    for (int64_t m = n - 1; m >= 0; --m) {
      const int64_t t = t0 + m;
      const double *St = seg + (m + 1) * KV, *Sp = seg + m * KV;
      const double *qt = q + t * K, *kt = k + t * K, *lat = la + t * K;
      const double *vt = v + t * V, *dot = dO + t * V;
      for (int64_t a = 0; a < K; ++a)            /* G += q_t^T dO_t */
        for (int64_t j = 0; j < V; ++j) G[a * V + j] += qt[a] * dot[j];
      for (int64_t a = 0; a < K; ++a) {
        double sq = 0.0, sk = 0.0, sa = 0.0;
        for (int64_t j = 0; j < V; ++j) {
          sq += St[a * V + j] * dot[j];          /* dq_t = S_t dO_t^T     */
          sk += G[a * V + j] * vt[j];            /* dk_t = G v_t^T        */
          sa += G[a * V + j] * Sp[a * V + j];    /* (S_{t-1} (.) G) 1     */
        }
        const double al = exp(lat[a]);
        dq[t * K + a] = sq;
        dk[t * K + a] = sk;
        dla[t * K + a] = al * sa;
      }
      double *dvt = dv + t * V;                  /* dv_t = k_t G */
      for (int64_t j = 0; j < V; ++j) dvt[j] = 0.0;
      for (int64_t a = 0; a < K; ++a)
        for (int64_t j = 0; j < V; ++j) dvt[j] += kt[a] * G[a * V + j];
      for (int64_t a = 0; a < K; ++a) {          /* G = Diag(alpha_t) G */
        const double al = exp(lat[a]);
        for (int64_t j = 0; j < V; ++j) G[a * V + j] *= al;
      }
    }
  }
  if (J->dS0) memcpy(J->dS0 + h * KV, G, (size_t)KV * sizeof(double));
  free(ckp); free(seg); free(G);
}

static void *bwd_worker(void *arg) {
  job_t *J = (job_t *)arg;
  for (int64_t it; (it = take_item(J)) >= 0;) bwd_item(J, it);
  return NULL;
}

static int run(job_t *J, int nthreads, void *(*fn)(void *)) {
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  pthread_t th[256];
  pthread_mutex_init(&J->mu, NULL);
  J->next = 0;
  J->status = 0;
  int started = 0;
  for (int i = 1; i < nthreads; ++i)
    if (pthread_create(&th[started], NULL, fn, J) == 0) ++started;
  fn(J);
  for (int i = 0; i < started; ++i) pthread_join(th[i], NULL);
  pthread_mutex_destroy(&J->mu);
  return J->status;
}

int gla_oracle_fwd(int64_t BH, int64_t T, int64_t K, int64_t V, const double *q,
                   const double *k, const double *v, const double *log_alpha,
                   const double *S0, double *o, double *ST, int nthreads) {
  if (BH < 0 || T < 0 || K <= 0 || V <= 0 || !q || !k || !v || !log_alpha || !o) return -1;
  job_t J;
  memset(&J, 0, sizeof J);
  J.BH = BH; J.T = T; J.K = K; J.V = V;
  J.q = q; J.k = k; J.v = v; J.la = log_alpha; J.S0 = S0; J.o = o; J.ST = ST;
  /* Split columns so that there are at least ~2 items per thread. */
  int64_t nblk = 1;
  while (BH * nblk < 2 * (int64_t)nthreads && V / (nblk * 2) >= 8) nblk *= 2;
  J.col_block = (V + nblk - 1) / nblk;
  J.n_items = BH * ((V + J.col_block - 1) / J.col_block);
  return run(&J, nthreads, fwd_worker);
}

int gla_oracle_bwd(int64_t BH, int64_t T, int64_t K, int64_t V, const double *q,
                   const double *k, const double *v, const double *log_alpha,
                   const double *S0, const double *dO, const double *dST, double *dq,
                   double *dk, double *dv, double *dlog_alpha, double *dS0, int nthreads,
                   int64_t ckpt) {
  if (BH < 0 || T < 0 || K <= 0 || V <= 0 || !q || !k || !v || !log_alpha || !dO || !dq ||
      !dk || !dv || !dlog_alpha)
    return -1;
  job_t J;
  memset(&J, 0, sizeof J);
  J.BH = BH; J.T = T; J.K = K; J.V = V;
  J.q = q; J.k = k; J.v = v; J.la = log_alpha; J.S0 = S0; J.dO = dO; J.dST = dST;
  J.dq = dq; J.dk = dk; J.dv = dv; J.dla = dlog_alpha; J.dS0 = dS0;
  J.ckpt = ckpt > 0 ? ckpt : 64;
  J.n_items = BH;
  return run(&J, nthreads, bwd_worker);
}
