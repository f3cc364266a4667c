/*
 * Comba step recurrence in fp64 -- TEST INFRASTRUCTURE ONLY.
 *
 * This is the plain, slow, token-by-token definition of what the chunk-wise
 * operator computes.  It exists to check the HIP path (tests, smoke check and
 * the CPU baseline of the benchmark) and is never called by the product path.
 * It shares no code with the HIP library.
 *
 * Recurrence (Eq. comba-S, Section 3 "Feedback Parameterization"), written in
 * the transposed state H = S^T in R^{dk x dv} (the orientation the paper's
 * recurrent pseudocode uses, Appendix B.1):
 *
 *     S_t = S_{t-1} (alpha_t I - bt_t k_t k_t^T) + beta_t v_t k_t^T
 *     o_t = S_t (q_t - d k_t)
 *
 * With H = S^T and a_t = H_{t-1}^T k_t this is
 *
 *     delta_t = beta_t v_t - bt_t a_t
 *     H_t     = alpha_t H_{t-1} + k_t delta_t^T
 *     o_t     = H_t^T (q_t - d k_t)                (reads the post-update state)
 *
 * alpha_t = exp(g_t) (g is the log forget gate), bt is the state-feedback
 * strength (tilde beta of Section 3.2; the operator uses bt == beta), d is the
 * per-head output-feedback scalar.
 *
 * The backward is plain reverse-mode differentiation of those three lines
 * (the paper gives no backward); the states needed in reverse order are
 * recomputed from checkpoints taken every CKPT tokens.
 *
 * Layouts: tokens of all sequences are packed along one axis of length Ttot;
 * sequence s covers tokens [cu[s], cu[s+1]).
 *   q, k [Ttot][H][dk]; v, o, dO [Ttot][H][dv]; g, beta, bt [Ttot][H];
 *   d [H]; h0, ht, dht, dh0 [N][H][dk][dv].
 * Work is split into independent (sequence, head) tasks run on a thread pool.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define CKPT 64

typedef struct {
  int nseq, H, dk, dv;
  const int64_t *cu;
  const double *q, *k, *v, *g, *beta, *bt, *d, *h0;
  double *o, *ht;
  /* backward */
  const double *dO, *dht;
  double *dq, *dk_, *dv_, *dg, *dbeta, *dbt, *dd_part, *dh0;
  int next_task; /* shared task counter */
  int failed;
} job_t;

static int take_task(job_t *J) { return __atomic_fetch_add(&J->next_task, 1, __ATOMIC_RELAXED); }

/* One token of the forward recurrence; updates H in place and writes o (may be NULL). */
static void step_forward(const job_t *J, int64_t t, int h, double *Hs, double *a, double *delta,
                         double *o) {
  const int H = J->H, dk = J->dk, dv = J->dv;
  const double *kt = J->k + ((size_t)t * H + h) * dk;
  const double *qt = J->q + ((size_t)t * H + h) * dk;
  const double *vt = J->v + ((size_t)t * H + h) * dv;
  const double alpha = exp(J->g[(size_t)t * H + h]);
  const double beta = J->beta[(size_t)t * H + h];
  const double bt = J->bt[(size_t)t * H + h];
  const double dh = J->d[h];
  for (int j = 0; j < dv; ++j) a[j] = 0.0;
  for (int i = 0; i < dk; ++i) {
    const double ki = kt[i];
    const double *row = Hs + (size_t)i * dv;
    for (int j = 0; j < dv; ++j) a[j] += row[j] * ki;
  }
  for (int j = 0; j < dv; ++j) delta[j] = beta * vt[j] - bt * a[j];
  for (int i = 0; i < dk; ++i) {
    const double ki = kt[i];
    double *row = Hs + (size_t)i * dv;
    for (int j = 0; j < dv; ++j) row[j] = alpha * row[j] + ki * delta[j];
  }
  if (o) {
    for (int j = 0; j < dv; ++j) o[j] = 0.0;
    for (int i = 0; i < dk; ++i) {
      const double qi = qt[i] - dh * kt[i];
      const double *row = Hs + (size_t)i * dv;
      for (int j = 0; j < dv; ++j) o[j] += row[j] * qi;
    }
  }
}

static void *fwd_worker(void *arg) {
  job_t *J = (job_t *)arg;
  const int H = J->H, dk = J->dk, dv = J->dv;
  const size_t S = (size_t)dk * dv;
  double *Hs = (double *)malloc(S * sizeof(double));
  double *a = (double *)malloc((size_t)dv * sizeof(double));
  double *delta = (double *)malloc((size_t)dv * sizeof(double));
  if (!Hs || !a || !delta) {
    J->failed = 1;
    free(Hs); free(a); free(delta);
    return NULL;
  }
  for (;;) {
    int task = take_task(J);
    if (task >= J->nseq * H) break;
    int s = task / H, h = task % H;
    if (J->h0) memcpy(Hs, J->h0 + ((size_t)s * H + h) * S, S * sizeof(double));
    else memset(Hs, 0, S * sizeof(double));
    for (int64_t t = J->cu[s]; t < J->cu[s + 1]; ++t)
      step_forward(J, t, h, Hs, a, delta, J->o ? J->o + ((size_t)t * H + h) * dv : NULL);
    if (J->ht) memcpy(J->ht + ((size_t)s * H + h) * S, Hs, S * sizeof(double));
  }
  free(Hs); free(a); free(delta);
  return NULL;
}

static void *bwd_worker(void *arg) {
  job_t *J = (job_t *)arg;
  const int H = J->H, dk = J->dk, dv = J->dv;
  const size_t S = (size_t)dk * dv;
  double *seg = NULL, *ck = NULL;
  size_t ck_cap = 0;
  double *dH = (double *)malloc(S * sizeof(double));
  double *a = (double *)malloc((size_t)dv * sizeof(double));
  double *delta = (double *)malloc((size_t)dv * sizeof(double));
  double *ddelta = (double *)malloc((size_t)dv * sizeof(double));
  double *qt_ = (double *)malloc((size_t)dk * sizeof(double));
  double *dqt = (double *)malloc((size_t)dk * sizeof(double));
  seg = (double *)malloc((size_t)(CKPT + 1) * S * sizeof(double));
  if (!dH || !a || !delta || !ddelta || !qt_ || !dqt || !seg) { J->failed = 1; goto done; }
  for (;;) {
    int task = take_task(J);
    if (task >= J->nseq * H) break;
    int s = task / H, h = task % H;
    const int64_t t0 = J->cu[s], len = J->cu[s + 1] - J->cu[s];
    const int64_t nck = (len + CKPT - 1) / CKPT;
    if ((size_t)(nck > 0 ? nck : 1) > ck_cap) {
      free(ck);
      ck_cap = (size_t)(nck > 0 ? nck : 1);
      ck = (double *)malloc(ck_cap * S * sizeof(double));
      if (!ck) { J->failed = 1; goto done; }
    }
    /* forward pass: checkpoint the state entering every CKPT-token segment */
    double *Hs = seg; /* scratch state */
    if (J->h0) memcpy(Hs, J->h0 + ((size_t)s * H + h) * S, S * sizeof(double));
    else memset(Hs, 0, S * sizeof(double));
    for (int64_t c = 0; c < nck; ++c) {
      memcpy(ck + (size_t)c * S, Hs, S * sizeof(double));
      int64_t e = (c + 1) * CKPT < len ? (c + 1) * CKPT : len;
      for (int64_t t = t0 + c * CKPT; t < t0 + e; ++t) step_forward(J, t, h, Hs, a, delta, NULL);
    }
    /* dH starts as the gradient of the final state */
    if (J->dht) memcpy(dH, J->dht + ((size_t)s * H + h) * S, S * sizeof(double));
    else memset(dH, 0, S * sizeof(double));
    double dd_acc = 0.0;
    const double dh = J->d[h];
    for (int64_t c = nck - 1; c >= 0; --c) {
      const int64_t sb = c * CKPT;
      const int64_t se = (c + 1) * CKPT < len ? (c + 1) * CKPT : len;
      const int n = (int)(se - sb);
      /* recompute the states of this segment: seg[j] = state before token sb+j */
      memcpy(seg, ck + (size_t)c * S, S * sizeof(double));
      for (int j = 0; j < n; ++j) {
        memcpy(seg + (size_t)(j + 1) * S, seg + (size_t)j * S, S * sizeof(double));
        step_forward(J, t0 + sb + j, h, seg + (size_t)(j + 1) * S, a, delta, NULL);
      }
      for (int j = n - 1; j >= 0; --j) {
        const int64_t t = t0 + sb + j;
        const size_t th = (size_t)t * H + h;
        const double *Hp = seg + (size_t)j * S;       /* H_{t-1} */
        const double *Hc = seg + (size_t)(j + 1) * S; /* H_t */
        const double *kt = J->k + th * dk;
        const double *qt = J->q + th * dk;
        const double *vt = J->v + th * dv;
        const double *dOt = J->dO + th * dv;
        const double alpha = exp(J->g[th]);
        const double beta = J->beta[th], bt = J->bt[th];
        double *dqo = J->dq + th * dk, *dko = J->dk_ + th * dk, *dvo = J->dv_ + th * dv;
        /* o_t = H_t^T qt~ */
        for (int i = 0; i < dk; ++i) qt_[i] = qt[i] - dh * kt[i];
        for (int i = 0; i < dk; ++i) {
          double *row = dH + (size_t)i * dv;
          const double *hrow = Hc + (size_t)i * dv;
          double acc = 0.0;
          for (int jj = 0; jj < dv; ++jj) {
            row[jj] += qt_[i] * dOt[jj];
            acc += hrow[jj] * dOt[jj];
          }
          dqt[i] = acc;
        }
        double kdq = 0.0;
        for (int i = 0; i < dk; ++i) {
          dqo[i] = dqt[i];
          dko[i] = -dh * dqt[i];
          kdq += kt[i] * dqt[i];
        }
        dd_acc -= kdq;
        /* a_t = H_{t-1}^T k_t ; delta_t = beta v_t - bt a_t */
        for (int jj = 0; jj < dv; ++jj) { a[jj] = 0.0; ddelta[jj] = 0.0; }
        for (int i = 0; i < dk; ++i) {
          const double ki = kt[i];
          const double *prow = Hp + (size_t)i * dv;
          const double *drow = dH + (size_t)i * dv;
          for (int jj = 0; jj < dv; ++jj) { a[jj] += prow[jj] * ki; ddelta[jj] += drow[jj] * ki; }
        }
        for (int jj = 0; jj < dv; ++jj) delta[jj] = beta * vt[jj] - bt * a[jj];
        /* H_t = alpha H_{t-1} + k delta^T */
        double dalpha = 0.0;
        for (int i = 0; i < dk; ++i) {
          const double *prow = Hp + (size_t)i * dv;
          const double *drow = dH + (size_t)i * dv;
          double acc_k = 0.0, acc_h = 0.0;
          for (int jj = 0; jj < dv; ++jj) {
            acc_k += drow[jj] * delta[jj];
            dalpha += drow[jj] * prow[jj];
            acc_h += prow[jj] * ddelta[jj];
          }
          dko[i] += acc_k - bt * acc_h; /* second term: through a_t */
        }
        J->dg[th] = alpha * dalpha;
        double db = 0.0, dbt = 0.0;
        for (int jj = 0; jj < dv; ++jj) {
          dvo[jj] = beta * ddelta[jj];
          db += vt[jj] * ddelta[jj];
          dbt -= a[jj] * ddelta[jj];
        }
        J->dbeta[th] = db;
        J->dbt[th] = dbt;
        /* dH_{t-1} = alpha dH_t - bt k_t ddelta^T */
        for (int i = 0; i < dk; ++i) {
          double *row = dH + (size_t)i * dv;
          const double ki = bt * kt[i];
          for (int jj = 0; jj < dv; ++jj) row[jj] = alpha * row[jj] - ki * ddelta[jj];
        }
      }
    }
    if (J->dh0) memcpy(J->dh0 + ((size_t)s * H + h) * S, dH, S * sizeof(double));
    J->dd_part[(size_t)s * H + h] = dd_acc;
  }
done:
  free(dH); free(a); free(delta); free(ddelta); free(qt_); free(dqt); free(seg); free(ck);
  return NULL;
}

static int run_pool(job_t *J, void *(*fn)(void *), int nthreads) {
  if (nthreads < 1) nthreads = 1;
  int ntask = J->nseq * J->H;
  if (nthreads > ntask) nthreads = ntask > 0 ? ntask : 1;
  pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)nthreads);
  if (!th) return -1;
  J->next_task = 0;
  J->failed = 0;
  int started = 0;
  for (int i = 1; i < nthreads; ++i) {
    if (pthread_create(&th[i], NULL, fn, J) != 0) break;
    ++started;
  }
  fn(J);
  for (int i = 1; i <= started; ++i) pthread_join(th[i], NULL);
  free(th);
  return J->failed ? -2 : 0;
}

/* Forward: o [Ttot][H][dv] (may be NULL), ht [N][H][dk][dv] (may be NULL).
 * h0 may be NULL (zero initial state).  Returns 0 on success. */
int oracle_fwd(int nseq, const int64_t *cu, int H, int dk, int dv, const double *q,
               const double *k, const double *v, const double *g, const double *beta,
               const double *bt, const double *d, const double *h0, double *o, double *ht,
               int nthreads) {
  job_t J;
  memset(&J, 0, sizeof(J));
  J.nseq = nseq; J.cu = cu; J.H = H; J.dk = dk; J.dv = dv;
  J.q = q; J.k = k; J.v = v; J.g = g; J.beta = beta; J.bt = bt; J.d = d; J.h0 = h0;
  J.o = o; J.ht = ht;
  return run_pool(&J, fwd_worker, nthreads);
}

/* Backward: gradients of <dO, o> + <dht, ht>.  dO required; dht, h0, dh0 may be NULL.
 * dd_part [N][H] receives per-(sequence, head) partial sums of dd (the caller
 * sums them over sequences in a fixed order).  dbeta is the gradient through
 * the write strength beta, dbt through the feedback strength bt. */
int oracle_bwd(int nseq, const int64_t *cu, int H, int dk, int dv, const double *q,
               const double *k, const double *v, const double *g, const double *beta,
               const double *bt, const double *d, const double *h0, const double *dO,
               const double *dht, double *dq, double *dk_out, double *dv_out, double *dg,
               double *dbeta, double *dbt, double *dd_part, double *dh0, int nthreads) {
  job_t J;
  memset(&J, 0, sizeof(J));
  J.nseq = nseq; J.cu = cu; J.H = H; J.dk = dk; J.dv = dv;
  J.q = q; J.k = k; J.v = v; J.g = g; J.beta = beta; J.bt = bt; J.d = d; J.h0 = h0;
  J.dO = dO; J.dht = dht; J.dq = dq; J.dk_ = dk_out; J.dv_ = dv_out; J.dg = dg;
  J.dbeta = dbeta; J.dbt = dbt; J.dd_part = dd_part; J.dh0 = dh0;
  return run_pool(&J, bwd_worker, nthreads);
}
