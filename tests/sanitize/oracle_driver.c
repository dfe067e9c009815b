/* Runs the fp64 oracle (oracle/gdn_oracle.c) on small dense and packed
 * problems, including empty and one-token sequences, under the sanitizers
 * it is built with; checks the return codes and that every output is
 * finite.  Exit status 0 on success. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int gdn_oracle_fwd(int N, const int64_t *cu, int H, int dk, int dv, const double *q,
                   const double *k, const double *v, const double *beta,
                   const double *log_alpha, const double *h0, double *o, double *ht,
                   int nthreads);
int gdn_oracle_bwd(int N, const int64_t *cu, int H, int dk, int dv, const double *q,
                   const double *k, const double *v, const double *beta,
                   const double *log_alpha, const double *h0, const double *dO,
                   const double *dht, double *o, double *ht, double *dq, double *dk_out,
                   double *dv_out, double *dbeta, double *dlog_alpha, double *dh0, int seg,
                   int nthreads);

static uint64_t rng = 88172645463325252ull;
static double uniform(void) { /* xorshift64, in [-1, 1) */
  rng ^= rng << 13;
  rng ^= rng >> 7;
  rng ^= rng << 17;
  return (double)(rng >> 11) / 9007199254740992.0 * 2.0 - 1.0;
}
static double *fill(size_t n, double scale, double offset) {
  double *p = malloc((n ? n : 1) * sizeof(double));
  for (size_t i = 0; i < n; ++i) p[i] = offset + scale * uniform();
  return p;
}
static int finite_all(const double *p, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!isfinite(p[i])) return 0;
  return 1;
}

static int run(int N, const int64_t *cu, int H, int dk, int dv, int with_states, int seg,
               int threads) {
  const size_t T = (size_t)cu[N], rk = T * H * dk, rv = T * H * dv, st = (size_t)N * H * dk * dv;
  double *q = fill(rk, 0.3, 0), *k = fill(rk, 0.3, 0), *v = fill(rv, 1, 0);
  double *beta = fill(T * H, 0.5, 0.5), *la = fill(T * H, 0.05, -0.1);
  double *h0 = with_states ? fill(st, 0.1, 0) : NULL, *dht = with_states ? fill(st, 0.1, 0) : NULL;
  double *dO = fill(rv, 1, 0);
  double *o = fill(rv, 0, 0), *ht = fill(st, 0, 0), *dq = fill(rk, 0, 0), *dkk = fill(rk, 0, 0);
  double *dvv = fill(rv, 0, 0), *db = fill(T * H, 0, 0), *dla = fill(T * H, 0, 0);
  double *dh0 = fill(st, 0, 0);
  int bad = 0;
  if (gdn_oracle_fwd(N, cu, H, dk, dv, q, k, v, beta, la, h0, o, ht, threads) != 0) bad |= 1;
  if (!finite_all(o, rv) || !finite_all(ht, st)) bad |= 2;
  if (gdn_oracle_bwd(N, cu, H, dk, dv, q, k, v, beta, la, h0, dO, dht, o, ht, dq, dkk, dvv, db,
                     dla, with_states ? dh0 : NULL, seg, threads) != 0)
    bad |= 4;
  if (!finite_all(dq, rk) || !finite_all(dkk, rk) || !finite_all(dvv, rv) ||
      !finite_all(db, T * H) || !finite_all(dla, T * H) || !finite_all(dh0, st))
    bad |= 8;
  free(q); free(k); free(v); free(beta); free(la); free(h0); free(dht); free(dO); free(o);
  free(ht); free(dq); free(dkk); free(dvv); free(db); free(dla); free(dh0);
  if (bad) fprintf(stderr, "case N=%d T=%zu H=%d dk=%d dv=%d: failure mask %d\n", N, T, H, dk, dv, bad);
  return bad;
}

int main(void) {
  int bad = 0;
  const int64_t dense[] = {0, 70, 140};
  const int64_t packed[] = {0, 0, 1, 66, 130, 131};
  const int64_t decreasing[] = {0, 5, 3};
  bad |= run(2, dense, 2, 8, 4, 1, 64, 2);
  bad |= run(5, packed, 3, 4, 8, 0, 7, 3);
  bad |= run(5, packed, 1, 16, 16, 1, 1, 1);
  /* argument errors come back as codes, with nothing read */
  if (gdn_oracle_fwd(2, decreasing, 1, 4, 4, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 1) == 0)
    bad |= 16;
  if (gdn_oracle_bwd(2, dense, 1, 4, 4, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL,
                     NULL, NULL, NULL, NULL, NULL, NULL, 0, 1) == 0)
    bad |= 32;
  printf(bad ? "oracle driver: FAILED (%d)\n" : "oracle driver: ok\n", bad);
  return bad ? 1 : 0;
}
