/*
 * Gated delta rule: plain fp64 CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the correctness reference that the
 * HIP path is checked against.  Only the tests, the smoke entry and the CPU
 * baseline leg of the benchmark may load it; the product path never does.
 * It shares no code, header or constant with the HIP library.
 *
 * What it computes (Gated DeltaNet, Sec. 3.1, Eq. "gated_delta_rule"):
 *   the paper writes the state as a dv x dk matrix S' with
 *     S'_t = S'_{t-1} ( a_t (I - b_t k_t k_t^T) ) + b_t v_t k_t^T,   o_t = S'_t q_t.
 *   This oracle stores the transpose S = S'^T (dk x dv, row-major), so
 *     S_t = a_t (I - b_t k_t k_t^T) S_{t-1} + b_t k_t v_t^T,        o_t = S_t^T q_t.
 *   It is evaluated token by token in the rank-one "test-time SGD" form the
 *   paper gives in Sec. 3.1 (online-regression view, Table 1 row
 *   "Gated DeltaNet"):
 *     u   = S_{t-1}^T k_t                 (the value the state currently recalls)
 *     r   = v_t - a_t u                   (the correction written back)
 *     S_t = a_t S_{t-1} + b_t k_t r^T
 *   with a_t = exp(log_alpha_t).  The dk x dk transition is never formed.
 *
 * Backward: the vector-Jacobian product of
 *     L = sum_t <dO_t, o_t> + <dS_final, S_L>
 * with respect to q, k, v, beta, log_alpha and the initial state.  The paper
 * gives no backward; the gradient of a smooth map is unique, so the hand
 * derivation below is the definition.  Walking t = L..1 with G = dL/dS_t
 * (initialised to dS_final):
 *     G    += q_t dO_t^T            dq_t = S_t dO_t
 *     r     = v_t - a_t S_{t-1}^T k_t,   y = G^T k_t
 *     dv_t  = b_t y                 dbeta_t = r . y
 *     dlog_alpha_t = <G, S_t - b_t k_t v_t^T>      (= a_t <G, (I - b k k^T) S_{t-1}>)
 *     dk_t  = b_t (G r - a_t S_{t-1} y)
 *     G    <- a_t (G - b_t k_t (k_t^T G))          (dL/dS_{t-1})
 *   and dS_init = G after t = 1.
 *   S_{t-1} and S_t are recomputed segment by segment from checkpoints taken
 *   every `seg` tokens of the forward walk, so memory stays bounded.
 *
 * Sequences: a packed buffer of N sequences given by cu[0..N] (cu[0] = 0,
 * non-decreasing, cu[N] = total tokens).  Every (sequence, head) pair is an
 * independent unit with its own initial state h0[n,h] (or zero); threads
 * own disjoint units, so results do not depend on the thread count.
 *
 * Layouts (contiguous, innermost last): q,k [Ttot,H,dk]; v,o,dO [Ttot,H,dv];
 * beta, log_alpha [Ttot,H]; states [N,H,dk,dv].  All arrays are double.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int N, H, dk, dv, seg;
  const int64_t *cu;
  const double *q, *k, *v, *beta, *log_alpha, *h0;
  /* forward outputs */
  double *o, *ht;
  /* backward inputs / outputs (NULL in a forward-only job) */
  const double *dO, *dht;
  double *dq, *dk_out, *dv_out, *dbeta, *dlog_alpha, *dh0;
  int backward;
  /* work distribution */
  pthread_mutex_t lock;
  long next_unit;
  int failed;
} job_t;

/* one token of the forward recurrence, in place on S (dk x dv);
 * r is scratch for dv doubles. */
static void step_forward(double *S, int dk, int dv, const double *kt,
                         const double *vt, double b, double a, double *r) {
  for (int j = 0; j < dv; ++j) r[j] = 0.0;
  for (int i = 0; i < dk; ++i) {
    const double ki = kt[i];
    const double *Si = S + (size_t)i * dv;
    for (int j = 0; j < dv; ++j) r[j] += Si[j] * ki; /* u = S^T k */
  }
  for (int j = 0; j < dv; ++j) r[j] = vt[j] - a * r[j]; /* r = v - a u */
  for (int i = 0; i < dk; ++i) {
    const double bk = b * kt[i];
    double *Si = S + (size_t)i * dv;
    for (int j = 0; j < dv; ++j) Si[j] = a * Si[j] + bk * r[j];
  }
}

/* o = S^T q */
static void read_out(const double *S, int dk, int dv, const double *qt,
                     double *ot) {
  for (int j = 0; j < dv; ++j) ot[j] = 0.0;
  for (int i = 0; i < dk; ++i) {
    const double qi = qt[i];
    const double *Si = S + (size_t)i * dv;
    for (int j = 0; j < dv; ++j) ot[j] += Si[j] * qi;
  }
}

static int run_unit_forward(job_t *J, int n, int h) {
  const int H = J->H, dk = J->dk, dv = J->dv;
  const size_t SS = (size_t)dk * dv;
  double *S = (double *)malloc(SS * sizeof(double));
  double *r = (double *)malloc((size_t)dv * sizeof(double));
  if (!S || !r) { free(S); free(r); return -1; }
  const size_t unit = (size_t)n * H + h;
  if (J->h0) memcpy(S, J->h0 + unit * SS, SS * sizeof(double));
  else memset(S, 0, SS * sizeof(double));
  for (int64_t t = J->cu[n]; t < J->cu[n + 1]; ++t) {
    const size_t th = (size_t)t * H + h;
    step_forward(S, dk, dv, J->k + th * dk, J->v + th * dv, J->beta[th],
                 exp(J->log_alpha[th]), r);
    read_out(S, dk, dv, J->q + th * dk, J->o + th * dv);
  }
  if (J->ht) memcpy(J->ht + unit * SS, S, SS * sizeof(double));
  free(S); free(r);
  return 0;
}

static int run_unit_backward(job_t *J, int n, int h) {
  const int H = J->H, dk = J->dk, dv = J->dv, seg = J->seg;
  const size_t SS = (size_t)dk * dv;
  const size_t unit = (size_t)n * H + h;
  const int64_t t0 = J->cu[n], L = J->cu[n + 1] - J->cu[n];
  const int64_t nseg = (L + seg - 1) / seg;
  /* checkpoints: state at the start of every segment, plus the final state */
  double *ck = (double *)malloc((size_t)(nseg + 1) * SS * sizeof(double));
  /* states inside one segment: states[j] = S after j tokens of the segment */
  double *states = (double *)malloc((size_t)(seg + 1) * SS * sizeof(double));
  double *G = (double *)malloc(SS * sizeof(double));
  double *r = (double *)malloc((size_t)dv * sizeof(double));
  double *y = (double *)malloc((size_t)dv * sizeof(double));
  double *Gr = (double *)malloc((size_t)dk * sizeof(double));
  double *Sy = (double *)malloc((size_t)dk * sizeof(double));
  if (!ck || !states || !G || !r || !y || !Gr || !Sy) {
    free(ck); free(states); free(G); free(r); free(y); free(Gr); free(Sy);
    return -1;
  }
  /* forward walk, keeping checkpoints (and the outputs, for completeness) */
  double *S = ck;
  if (J->h0) memcpy(S, J->h0 + unit * SS, SS * sizeof(double));
  else memset(S, 0, SS * sizeof(double));
  for (int64_t s = 0; s < nseg; ++s) {
    double *Snext = ck + (size_t)(s + 1) * SS;
    memcpy(Snext, ck + (size_t)s * SS, SS * sizeof(double));
    const int64_t e = (s + 1) * seg < L ? (s + 1) * seg : L;
    for (int64_t t = s * seg; t < e; ++t) {
      const size_t th = (size_t)(t0 + t) * H + h;
      step_forward(Snext, dk, dv, J->k + th * dk, J->v + th * dv, J->beta[th],
                   exp(J->log_alpha[th]), r);
      if (J->o) read_out(Snext, dk, dv, J->q + th * dk, J->o + th * dv);
    }
  }
  if (J->ht) memcpy(J->ht + unit * SS, ck + (size_t)nseg * SS, SS * sizeof(double));

  /* reverse walk */
  if (J->dht) memcpy(G, J->dht + unit * SS, SS * sizeof(double));
  else memset(G, 0, SS * sizeof(double));
  for (int64_t s = nseg - 1; s >= 0; --s) {
    const int64_t b0 = s * seg;
    const int64_t e = (s + 1) * seg < L ? (s + 1) * seg : L;
    memcpy(states, ck + (size_t)s * SS, SS * sizeof(double));
    for (int64_t t = b0; t < e; ++t) {
      const size_t th = (size_t)(t0 + t) * H + h;
      double *Sj = states + (size_t)(t - b0 + 1) * SS;
      memcpy(Sj, Sj - SS, SS * sizeof(double));
      step_forward(Sj, dk, dv, J->k + th * dk, J->v + th * dv, J->beta[th],
                   exp(J->log_alpha[th]), r);
    }
    for (int64_t t = e - 1; t >= b0; --t) {
      const size_t th = (size_t)(t0 + t) * H + h;
      const double *St = states + (size_t)(t - b0 + 1) * SS; /* S_t     */
      const double *Sp = St - SS;                             /* S_{t-1} */
      const double *qt = J->q + th * dk, *kt = J->k + th * dk;
      const double *vt = J->v + th * dv, *dOt = J->dO + th * dv;
      const double b = J->beta[th], a = exp(J->log_alpha[th]);
      /* G += q dO^T ; dq = S_t dO */
      for (int i = 0; i < dk; ++i) {
        double *Gi = G + (size_t)i * dv;
        const double qi = qt[i];
        for (int j = 0; j < dv; ++j) Gi[j] += qi * dOt[j];
      }
      double *dqt = J->dq + th * dk;
      for (int i = 0; i < dk; ++i) {
        const double *Si = St + (size_t)i * dv;
        double acc = 0.0;
        for (int j = 0; j < dv; ++j) acc += Si[j] * dOt[j];
        dqt[i] = acc;
      }
      /* r = v - a S_{t-1}^T k ; y = G^T k */
      for (int j = 0; j < dv; ++j) { r[j] = 0.0; y[j] = 0.0; }
      for (int i = 0; i < dk; ++i) {
        const double ki = kt[i];
        const double *Si = Sp + (size_t)i * dv, *Gi = G + (size_t)i * dv;
        for (int j = 0; j < dv; ++j) { r[j] += Si[j] * ki; y[j] += Gi[j] * ki; }
      }
      for (int j = 0; j < dv; ++j) r[j] = vt[j] - a * r[j];
      double *dvt = J->dv_out + th * dv;
      double db = 0.0;
      for (int j = 0; j < dv; ++j) { dvt[j] = b * y[j]; db += r[j] * y[j]; }
      J->dbeta[th] = db;
      /* dlog_alpha = <G, S_t - b k v^T> */
      double dla = 0.0;
      for (int i = 0; i < dk; ++i) {
        const double *Si = St + (size_t)i * dv, *Gi = G + (size_t)i * dv;
        const double bk = b * kt[i];
        for (int j = 0; j < dv; ++j) dla += Gi[j] * (Si[j] - bk * vt[j]);
      }
      J->dlog_alpha[th] = dla;
      /* dk = b (G r - a S_{t-1} y) */
      for (int i = 0; i < dk; ++i) {
        const double *Si = Sp + (size_t)i * dv, *Gi = G + (size_t)i * dv;
        double gr = 0.0, sy = 0.0;
        for (int j = 0; j < dv; ++j) { gr += Gi[j] * r[j]; sy += Si[j] * y[j]; }
        Gr[i] = gr; Sy[i] = sy;
      }
      double *dkt = J->dk_out + th * dk;
      for (int i = 0; i < dk; ++i) dkt[i] = b * (Gr[i] - a * Sy[i]);
      /* G <- a (G - b k (k^T G)) ; k^T G = y^T */
      for (int i = 0; i < dk; ++i) {
        double *Gi = G + (size_t)i * dv;
        const double bk = b * kt[i];
        for (int j = 0; j < dv; ++j) Gi[j] = a * (Gi[j] - bk * y[j]);
      }
    }
  }
  if (J->dh0) memcpy(J->dh0 + unit * SS, G, SS * sizeof(double));
  free(ck); free(states); free(G); free(r); free(y); free(Gr); free(Sy);
  return 0;
}

static void *worker(void *arg) {
  job_t *J = (job_t *)arg;
  const long total = (long)J->N * J->H;
  for (;;) {
    pthread_mutex_lock(&J->lock);
    const long u = J->next_unit++;
    pthread_mutex_unlock(&J->lock);
    if (u >= total) break;
    const int n = (int)(u / J->H), h = (int)(u % J->H);
    const int rc = J->backward ? run_unit_backward(J, n, h) : run_unit_forward(J, n, h);
    if (rc) {
      pthread_mutex_lock(&J->lock);
      J->failed = 1;
      pthread_mutex_unlock(&J->lock);
    }
  }
  return NULL;
}

static int run_job(job_t *J, int nthreads) {
  if (nthreads < 1) nthreads = 1;
  const long total = (long)J->N * J->H;
  if (nthreads > total) nthreads = (int)(total > 0 ? total : 1);
  pthread_mutex_init(&J->lock, NULL);
  J->next_unit = 0;
  J->failed = 0;
  pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)nthreads);
  if (!th) return -1;
  int started = 0;
  for (int i = 1; i < nthreads; ++i)
    if (pthread_create(&th[started], NULL, worker, J) == 0) ++started;
  /* the calling thread works too */
  worker(J);
  for (int i = 0; i < started; ++i) pthread_join(th[i], NULL);
  free(th);
  pthread_mutex_destroy(&J->lock);
  return J->failed ? -1 : 0;
}

static int check_cu(int N, const int64_t *cu) {
  if (N < 0 || !cu || cu[0] != 0) return -2;
  for (int n = 0; n < N; ++n)
    if (cu[n + 1] < cu[n]) return -2;
  return 0;
}

/* Forward.  h0 and ht may be NULL.  Returns 0 on success. */
int gdn_oracle_fwd(int N, const int64_t *cu, int H, int dk, int dv,
                   const double *q, const double *k, const double *v,
                   const double *beta, const double *log_alpha,
                   const double *h0, double *o, double *ht, int nthreads) {
  if (check_cu(N, cu) || H < 1 || dk < 1 || dv < 1) return -2;
  job_t J;
  memset(&J, 0, sizeof J);
  J.N = N; J.H = H; J.dk = dk; J.dv = dv; J.seg = 64; J.cu = cu;
  J.q = q; J.k = k; J.v = v; J.beta = beta; J.log_alpha = log_alpha; J.h0 = h0;
  J.o = o; J.ht = ht; J.backward = 0;
  return run_job(&J, nthreads);
}

/* Backward (re-runs the forward internally).  o and ht may be NULL; if given
 * they receive the forward outputs.  dht and dh0 may be NULL.  `seg` is the
 * checkpoint spacing in tokens: a memory knob only, the arithmetic is the
 * same for every value.  Returns 0 on success. */
int gdn_oracle_bwd(int N, const int64_t *cu, int H, int dk, int dv,
                   const double *q, const double *k, const double *v,
                   const double *beta, const double *log_alpha,
                   const double *h0, const double *dO, const double *dht,
                   double *o, double *ht, double *dq, double *dk_out,
                   double *dv_out, double *dbeta, double *dlog_alpha,
                   double *dh0, int seg, int nthreads) {
  if (check_cu(N, cu) || H < 1 || dk < 1 || dv < 1 || seg < 1) return -2;
  job_t J;
  memset(&J, 0, sizeof J);
  J.N = N; J.H = H; J.dk = dk; J.dv = dv; J.seg = seg; J.cu = cu;
  J.q = q; J.k = k; J.v = v; J.beta = beta; J.log_alpha = log_alpha; J.h0 = h0;
  J.o = o; J.ht = ht; J.dO = dO; J.dht = dht;
  J.dq = dq; J.dk_out = dk_out; J.dv_out = dv_out; J.dbeta = dbeta;
  J.dlog_alpha = dlog_alpha; J.dh0 = dh0; J.backward = 1;
  return run_job(&J, nthreads);
}
