/*
 * Test infrastructure: a driver that exercises the fp64 oracle
 * (tla_oracle.c) on small inputs for a build with the address and
 * undefined-behaviour sanitizers (tests/test_sanitize.py).  Both variants,
 * with and without beta, initial state and final-state gradient, lengths
 * that are and are not multiples of 64 (the backward's checkpoint segment),
 * and one decode step against the forward of one token.  Exits non-zero on a
 * non-finite result or a mismatch.
 */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_fwd(int variant, int B, int T, int H, int K, int V, int E, const double* q,
               const double* k, const double* v, const double* q2, const double* k2,
               const double* g, const double* beta, const double* s0, double* o, double* sf);
int oracle_step(int variant, int N, int H, int K, int V, int E, const double* q, const double* k,
                const double* v, const double* q2, const double* k2, const double* g,
                const double* beta, double* state, double* o);
int oracle_bwd(int variant, int B, int T, int H, int K, int V, int E, const double* q,
               const double* k, const double* v, const double* q2, const double* k2,
               const double* g, const double* beta, const double* s0, const double* dO,
               const double* dSf, double* dq, double* dk, double* dv, double* dq2, double* dk2,
               double* dg, double* dbeta, double* ds0);

static unsigned long long rng = 0x9E3779B97F4A7C15ull;
static double uni(void) { /* xorshift64*, uniform in (-1, 1) */
  rng ^= rng >> 12;
  rng ^= rng << 25;
  rng ^= rng >> 27;
  return (double)((rng * 2685821657736338717ull) >> 11) / 4503599627370496.0 - 1.0;
}
static double* arr(size_t n, double scale, double shift) {
  double* x = (double*)malloc(n * sizeof(double));
  for (size_t i = 0; i < n; ++i) x[i] = shift + scale * uni();
  return x;
}
static int finite_all(const double* x, size_t n) {
  for (size_t i = 0; i < n; ++i)
    if (!isfinite(x[i])) return 0;
  return 1;
}

static int run(int variant, int use_beta, int use_s0, int use_dsf, int B, int T, int H, int K,
               int V, int E) {
  const size_t nt = (size_t)B * T * H, ns = (size_t)B * H * E * K * V;
  double *q = arr(nt * K, 0.3, 0), *k = arr(nt * K, 0.3, 0), *v = arr(nt * V, 1, 0);
  double *q2 = arr(nt * E, 0.5, 0), *k2 = arr(nt * E, 0.5, 0), *g = arr(nt * E, 0.05, -0.1);
  double* beta = use_beta ? arr(nt, 0.4, 0.5) : NULL;
  double* s0 = use_s0 ? arr(ns, 0.02, 0) : NULL;
  double *dO = arr(nt * V, 1, 0), *dsf = use_dsf ? arr(ns, 1, 0) : NULL;
  double *o = arr(nt * V, 0, 0), *sf = arr(ns, 0, 0);
  double *dq = arr(nt * K, 0, 0), *dk = arr(nt * K, 0, 0), *dv = arr(nt * V, 0, 0);
  double *dq2 = arr(nt * E, 0, 0), *dk2 = arr(nt * E, 0, 0), *dg = arr(nt * E, 0, 0);
  double *dbeta = use_beta ? arr(nt, 0, 0) : NULL, *ds0 = arr(ns, 0, 0);
  int bad = 0;
  bad |= oracle_fwd(variant, B, T, H, K, V, E, q, k, v, q2, k2, g, beta, s0, o, sf) != 0;
  bad |= !finite_all(o, nt * V) || !finite_all(sf, ns);
  bad |= oracle_bwd(variant, B, T, H, K, V, E, q, k, v, q2, k2, g, beta, s0, dO, dsf, dq, dk, dv,
                    dq2, dk2, dg, dbeta, ds0) != 0;
  bad |= !finite_all(dq, nt * K) || !finite_all(dk, nt * K) || !finite_all(dv, nt * V) ||
         !finite_all(dq2, nt * E) || !finite_all(dk2, nt * E) || !finite_all(dg, nt * E) ||
         !finite_all(ds0, ns) || (dbeta && !finite_all(dbeta, nt));
  if (T == 1) {  /* one decode step from s0 equals the forward of one token */
    double* st = arr(ns, 0, 0);
    double* od = arr(nt * V, 0, 0);
    for (size_t i = 0; i < ns; ++i) st[i] = s0 ? s0[i] : 0.0;
    bad |= oracle_step(variant, B, H, K, V, E, q, k, v, q2, k2, g, beta, st, od) != 0;
    for (size_t i = 0; i < nt * V; ++i) bad |= fabs(od[i] - o[i]) > 1e-12 * (1 + fabs(o[i]));
    for (size_t i = 0; i < ns; ++i) bad |= fabs(st[i] - sf[i]) > 1e-12 * (1 + fabs(sf[i]));
    free(st);
    free(od);
  }
  double* all[] = {q, k, v, q2, k2, g, beta, s0, dO, dsf, o, sf, dq, dk, dv, dq2, dk2, dg, dbeta, ds0};
  for (size_t i = 0; i < sizeof(all) / sizeof(all[0]); ++i) free(all[i]);
  if (bad)
    fprintf(stderr, "FAIL variant=%d beta=%d s0=%d dsf=%d B=%d T=%d H=%d K=%d V=%d E=%d\n", variant,
            use_beta, use_s0, use_dsf, B, T, H, K, V, E);
  return bad;
}

int main(void) {
  int bad = 0;
  for (int variant = 0; variant < 2; ++variant)
    for (int mask = 0; mask < 8; ++mask) {
      const int use_beta = variant == 1 || (mask & 1), use_s0 = (mask >> 1) & 1, use_dsf = (mask >> 2) & 1;
      bad |= run(variant, use_beta, use_s0, use_dsf, 2, 70, 2, 8, 6, 3);
      bad |= run(variant, use_beta, use_s0, use_dsf, 1, 1, 2, 4, 4, 2);
      bad |= run(variant, use_beta, use_s0, use_dsf, 1, 128, 1, 4, 8, 1);
    }
  puts(bad ? "sanitize check: FAILED" : "sanitize check: ok");
  return bad;
}
