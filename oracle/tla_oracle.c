/*
 * Test infrastructure only: the fp64 CPU oracle for triadic linear attention.
 *
 * Nothing in the product path may link, load or call this file.  Only the
 * tests, the smoke check and the CPU-baseline leg of the benchmark use it.
 *
 * It is the plain definition of the operator, evaluated token by token in
 * double precision, with no chunking, blocking or fusion:
 *
 *   per-slice forgetting   Sbar[e,k,v] = a_t[e] * S_{t-1}[e,k,v]
 *                          (Section 2.4, Eq. forget3; decay before erase)
 *   gated delta rule (GDN) r[v] = sum_{e,k} k2_t[e] k_t[k] Sbar[e,k,v]
 *                          w   = beta_t (v_t - r)        (Eq. gdn3; Alg. 2)
 *   scalar-gated LA (sGLA) w   = beta_t v_t, beta_t = 1 when no beta is given
 *                          (Alg. 2 writes k (x) beta k' (x) v)
 *   write                  S_t = Sbar + k2_t (x) k_t (x) w
 *   read                   o_t[v] = sum_{e,k} q2_t[e] q_t[k] S_t[e,k,v]
 *                          (Eq. la3: the read uses S_t, so token t sees itself)
 *
 * Gates are passed as log-gates g = log a (a = exp g); the per-slice gate
 * a_t[e] multiplies slice e of the state (Eq. forget3).
 *
 * The backward is reverse-mode differentiation of exactly this loop.  States
 * are checkpointed every SEG tokens and each segment is recomputed forward
 * before it is walked in reverse.
 *
 * Layouts (row-major, all double):
 *   q, k    [B][T][H][K]        v, o, dO  [B][T][H][V]
 *   q2, k2, g [B][T][H][E]      beta      [B][T][H]   (may be NULL)
 *   state   [B][H][E][K][V]     (s0 / s_final / dS_final / ds0, NULL = zero)
 * For the single-token step the T axis is absent: q [N][H][K] and so on.
 *
 * Variant codes: 0 = sGLA, 1 = GDN.  Every function returns 0 on success and
 * a negative value on bad arguments or allocation failure.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define SEG 64

static size_t idx_tok(int b, int t, int h, int T, int H, int D) {
  return (((size_t)b * T + t) * H + h) * (size_t)D;
}

/* One token of the recurrence on a single head's state S[E][K][V], in place.
 * w_out receives the written value vector, r_out the retrieval (zero for
 * sGLA), o the read-out. */
static void token_forward(int variant, int K, int V, int E, const double* q,
                          const double* k, const double* v, const double* q2,
                          const double* k2, const double* g, double beta,
                          double* S, double* o, double* w_out, double* r_out) {
  const size_t KV = (size_t)K * V;
  /* decay each slice by its own gate */
  for (int e = 0; e < E; ++e) {
    const double a = exp(g[e]);
    double* Se = S + e * KV;
    for (size_t i = 0; i < KV; ++i) Se[i] *= a;
  }
  /* retrieval under the pair of keys (k, k2) from the decayed state */
  double* r = r_out;
  for (int j = 0; j < V; ++j) r[j] = 0.0;
  if (variant == 1) {
    for (int e = 0; e < E; ++e)
      for (int kk = 0; kk < K; ++kk) {
        const double kap = k2[e] * k[kk];
        const double* row = S + e * KV + (size_t)kk * V;
        for (int j = 0; j < V; ++j) r[j] += kap * row[j];
      }
  }
  double* w = w_out;
  for (int j = 0; j < V; ++j)
    w[j] = (variant == 1) ? beta * (v[j] - r[j]) : beta * v[j];
  /* rank-one write with the joint key k2 (x) k */
  for (int e = 0; e < E; ++e)
    for (int kk = 0; kk < K; ++kk) {
      const double kap = k2[e] * k[kk];
      double* row = S + e * KV + (size_t)kk * V;
      for (int j = 0; j < V; ++j) row[j] += kap * w[j];
    }
  /* read with the joint query q2 (x) q */
  for (int j = 0; j < V; ++j) o[j] = 0.0;
  for (int e = 0; e < E; ++e)
    for (int kk = 0; kk < K; ++kk) {
      const double rho = q2[e] * q[kk];
      const double* row = S + e * KV + (size_t)kk * V;
      for (int j = 0; j < V; ++j) o[j] += rho * row[j];
    }
}

int oracle_fwd(int variant, int B, int T, int H, int K, int V, int E,
               const double* q, const double* k, const double* v,
               const double* q2, const double* k2, const double* g,
               const double* beta, const double* s0, double* o,
               double* s_final) {
  if (B <= 0 || T < 0 || H <= 0 || K <= 0 || V <= 0 || E <= 0) return -1;
  if (variant != 0 && variant != 1) return -1;
  if (variant == 1 && !beta) return -1;
  const size_t S_sz = (size_t)E * K * V;
  int fail = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : fail)
  for (int bh = 0; bh < B * H; ++bh) {
    const int b = bh / H, h = bh % H;
    double* S = (double*)malloc(S_sz * sizeof(double));
    double* w = (double*)malloc((size_t)V * sizeof(double));
    double* r = (double*)malloc((size_t)V * sizeof(double));
    if (!S || !w || !r) {
      free(S); free(w); free(r);
      fail |= 1;
      continue;
    }
    if (s0)
      memcpy(S, s0 + (size_t)bh * S_sz, S_sz * sizeof(double));
    else
      memset(S, 0, S_sz * sizeof(double));
    for (int t = 0; t < T; ++t) {
      const double bt = beta ? beta[((size_t)b * T + t) * H + h] : 1.0;
      token_forward(variant, K, V, E, q + idx_tok(b, t, h, T, H, K),
                    k + idx_tok(b, t, h, T, H, K),
                    v + idx_tok(b, t, h, T, H, V),
                    q2 + idx_tok(b, t, h, T, H, E),
                    k2 + idx_tok(b, t, h, T, H, E),
                    g + idx_tok(b, t, h, T, H, E), bt, S,
                    o + idx_tok(b, t, h, T, H, V), w, r);
    }
    if (s_final) memcpy(s_final + (size_t)bh * S_sz, S, S_sz * sizeof(double));
    free(S); free(w); free(r);
  }
  return fail ? -2 : 0;
}

int oracle_step(int variant, int N, int H, int K, int V, int E,
                const double* q, const double* k, const double* v,
                const double* q2, const double* k2, const double* g,
                const double* beta, double* state, double* o) {
  /* one token per (n, h): a T = 1 forward on the state in place */
  if (N <= 0 || H <= 0 || K <= 0 || V <= 0 || E <= 0) return -1;
  if (variant != 0 && variant != 1) return -1;
  if (variant == 1 && !beta) return -1;
  const size_t S_sz = (size_t)E * K * V;
  int fail = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : fail)
  for (int nh = 0; nh < N * H; ++nh) {
    double* w = (double*)malloc((size_t)V * sizeof(double));
    double* r = (double*)malloc((size_t)V * sizeof(double));
    if (!w || !r) {
      free(w); free(r);
      fail |= 1;
      continue;
    }
    token_forward(variant, K, V, E, q + (size_t)nh * K, k + (size_t)nh * K,
                  v + (size_t)nh * V, q2 + (size_t)nh * E, k2 + (size_t)nh * E,
                  g + (size_t)nh * E, beta ? beta[nh] : 1.0,
                  state + (size_t)nh * S_sz, o + (size_t)nh * V, w, r);
    free(w); free(r);
  }
  return fail ? -2 : 0;
}

/*
 * Reverse-mode backward of oracle_fwd.  dS_final may be NULL (zero).
 * Outputs dq, dk [B][T][H][K]; dv [B][T][H][V]; dq2, dk2, dg [B][T][H][E];
 * dbeta [B][T][H] (written only when beta is given); ds0 [B][H][E][K][V]
 * (may be NULL).  dg is the gradient with respect to the log-gate g.
 */
int oracle_bwd(int variant, int B, int T, int H, int K, int V, int E,
               const double* q, const double* k, const double* v,
               const double* q2, const double* k2, const double* g,
               const double* beta, const double* s0, const double* dO,
               const double* dS_final, double* dq, double* dk, double* dv,
               double* dq2, double* dk2, double* dg, double* dbeta,
               double* ds0) {
  if (B <= 0 || T < 0 || H <= 0 || K <= 0 || V <= 0 || E <= 0) return -1;
  if (variant != 0 && variant != 1) return -1;
  if (variant == 1 && !beta) return -1;
  const size_t S_sz = (size_t)E * K * V;
  const size_t KV = (size_t)K * V;
  const int nseg = (T + SEG - 1) / SEG;
  int fail = 0;
#pragma omp parallel for schedule(dynamic, 1) reduction(| : fail)
  for (int bh = 0; bh < B * H; ++bh) {
    const int b = bh / H, h = bh % H;
    /* ck[j] = state before token j*SEG; seg[i] = state before token t0+i */
    double* ck = (double*)malloc((size_t)(nseg + 1) * S_sz * sizeof(double));
    double* seg = (double*)malloc((size_t)(SEG + 1) * S_sz * sizeof(double));
    double* dS = (double*)malloc(S_sz * sizeof(double));
    double* Sb = (double*)malloc(S_sz * sizeof(double));
    double* tmpo = (double*)malloc((size_t)V * sizeof(double));
    double* w = (double*)malloc((size_t)V * sizeof(double));
    double* r = (double*)malloc((size_t)V * sizeof(double));
    double* dw = (double*)malloc((size_t)V * sizeof(double));
    double* dr = (double*)malloc((size_t)V * sizeof(double));
    double* dkap = (double*)malloc((size_t)E * K * sizeof(double));
    double* drho = (double*)malloc((size_t)E * K * sizeof(double));
    if (!ck || !seg || !dS || !Sb || !tmpo || !w || !r || !dw || !dr || !dkap ||
        !drho) {
      free(ck); free(seg); free(dS); free(Sb); free(tmpo); free(w); free(r);
      free(dw); free(dr); free(dkap); free(drho);
      fail |= 1;
      continue;
    }
    /* forward pass storing segment-start checkpoints */
    if (s0)
      memcpy(ck, s0 + (size_t)bh * S_sz, S_sz * sizeof(double));
    else
      memset(ck, 0, S_sz * sizeof(double));
    memcpy(Sb, ck, S_sz * sizeof(double));
    for (int t = 0; t < T; ++t) {
      const double bt = beta ? beta[((size_t)b * T + t) * H + h] : 1.0;
      token_forward(variant, K, V, E, q + idx_tok(b, t, h, T, H, K),
                    k + idx_tok(b, t, h, T, H, K),
                    v + idx_tok(b, t, h, T, H, V),
                    q2 + idx_tok(b, t, h, T, H, E),
                    k2 + idx_tok(b, t, h, T, H, E),
                    g + idx_tok(b, t, h, T, H, E), bt, Sb, tmpo, w, r);
      if ((t + 1) % SEG == 0)
        memcpy(ck + (size_t)((t + 1) / SEG) * S_sz, Sb, S_sz * sizeof(double));
    }
    /* reverse pass */
    if (dS_final)
      memcpy(dS, dS_final + (size_t)bh * S_sz, S_sz * sizeof(double));
    else
      memset(dS, 0, S_sz * sizeof(double));
    for (int sg = nseg - 1; sg >= 0; --sg) {
      const int t0 = sg * SEG;
      const int t1 = (t0 + SEG < T) ? t0 + SEG : T;
      /* recompute the states of this segment */
      memcpy(seg, ck + (size_t)sg * S_sz, S_sz * sizeof(double));
      for (int t = t0; t < t1; ++t) {
        double* Snext = seg + (size_t)(t - t0 + 1) * S_sz;
        memcpy(Snext, seg + (size_t)(t - t0) * S_sz, S_sz * sizeof(double));
        const double bt = beta ? beta[((size_t)b * T + t) * H + h] : 1.0;
        token_forward(variant, K, V, E, q + idx_tok(b, t, h, T, H, K),
                      k + idx_tok(b, t, h, T, H, K),
                      v + idx_tok(b, t, h, T, H, V),
                      q2 + idx_tok(b, t, h, T, H, E),
                      k2 + idx_tok(b, t, h, T, H, E),
                      g + idx_tok(b, t, h, T, H, E), bt, Snext, tmpo, w, r);
      }
      for (int t = t1 - 1; t >= t0; --t) {
        const double* Sprev = seg + (size_t)(t - t0) * S_sz;   /* S_{t-1} */
        const double* Scur = seg + (size_t)(t - t0 + 1) * S_sz; /* S_t */
        const double* qt = q + idx_tok(b, t, h, T, H, K);
        const double* kt = k + idx_tok(b, t, h, T, H, K);
        const double* vt = v + idx_tok(b, t, h, T, H, V);
        const double* q2t = q2 + idx_tok(b, t, h, T, H, E);
        const double* k2t = k2 + idx_tok(b, t, h, T, H, E);
        const double* gt = g + idx_tok(b, t, h, T, H, E);
        const double* dot = dO + idx_tok(b, t, h, T, H, V);
        const double bt = beta ? beta[((size_t)b * T + t) * H + h] : 1.0;
        double* dqt = dq + idx_tok(b, t, h, T, H, K);
        double* dkt = dk + idx_tok(b, t, h, T, H, K);
        double* dvt = dv + idx_tok(b, t, h, T, H, V);
        double* dq2t = dq2 + idx_tok(b, t, h, T, H, E);
        double* dk2t = dk2 + idx_tok(b, t, h, T, H, E);
        double* dgt = dg + idx_tok(b, t, h, T, H, E);

        /* decayed state Sbar = a (.) S_{t-1} */
        for (int e = 0; e < E; ++e) {
          const double a = exp(gt[e]);
          for (size_t i = 0; i < KV; ++i)
            Sb[e * KV + i] = a * Sprev[e * KV + i];
        }
        /* w and r as in the forward */
        for (int j = 0; j < V; ++j) r[j] = 0.0;
        if (variant == 1)
          for (int e = 0; e < E; ++e)
            for (int kk = 0; kk < K; ++kk) {
              const double kap = k2t[e] * kt[kk];
              const double* row = Sb + e * KV + (size_t)kk * V;
              for (int j = 0; j < V; ++j) r[j] += kap * row[j];
            }
        for (int j = 0; j < V; ++j)
          w[j] = (variant == 1) ? bt * (vt[j] - r[j]) : bt * vt[j];

        /* read o = rho^T S_t: dS += rho do^T, drho = S_t do */
        for (int e = 0; e < E; ++e)
          for (int kk = 0; kk < K; ++kk) {
            const double rho = q2t[e] * qt[kk];
            const double* srow = Scur + e * KV + (size_t)kk * V;
            double* drow = dS + e * KV + (size_t)kk * V;
            double acc = 0.0;
            for (int j = 0; j < V; ++j) {
              drow[j] += rho * dot[j];
              acc += srow[j] * dot[j];
            }
            drho[e * K + kk] = acc;
          }
        for (int kk = 0; kk < K; ++kk) {
          double acc = 0.0;
          for (int e = 0; e < E; ++e) acc += q2t[e] * drho[e * K + kk];
          dqt[kk] = acc;
        }
        for (int e = 0; e < E; ++e) {
          double acc = 0.0;
          for (int kk = 0; kk < K; ++kk) acc += qt[kk] * drho[e * K + kk];
          dq2t[e] = acc;
        }

        /* write S_t = Sbar + kappa w^T: dkappa = dS w, dw = dS^T kappa */
        for (int j = 0; j < V; ++j) dw[j] = 0.0;
        for (int e = 0; e < E; ++e)
          for (int kk = 0; kk < K; ++kk) {
            const double kap = k2t[e] * kt[kk];
            const double* drow = dS + e * KV + (size_t)kk * V;
            double acc = 0.0;
            for (int j = 0; j < V; ++j) {
              acc += drow[j] * w[j];
              dw[j] += kap * drow[j];
            }
            dkap[e * K + kk] = acc;
          }

        /* value path */
        if (variant == 1) {
          double db = 0.0;
          for (int j = 0; j < V; ++j) {
            db += dw[j] * (vt[j] - r[j]);
            dvt[j] = bt * dw[j];
            dr[j] = -bt * dw[j];
          }
          if (dbeta) dbeta[((size_t)b * T + t) * H + h] = db;
          /* r = kappa^T Sbar: dkappa += Sbar dr, dSbar += kappa dr^T */
          for (int e = 0; e < E; ++e)
            for (int kk = 0; kk < K; ++kk) {
              const double kap = k2t[e] * kt[kk];
              const double* sbrow = Sb + e * KV + (size_t)kk * V;
              double* drow = dS + e * KV + (size_t)kk * V;
              double acc = 0.0;
              for (int j = 0; j < V; ++j) {
                acc += sbrow[j] * dr[j];
                drow[j] += kap * dr[j];
              }
              dkap[e * K + kk] += acc;
            }
        } else {
          double db = 0.0;
          for (int j = 0; j < V; ++j) {
            db += dw[j] * vt[j];
            dvt[j] = bt * dw[j];
          }
          if (dbeta && beta) dbeta[((size_t)b * T + t) * H + h] = db;
        }

        /* kappa = k2 (x) k */
        for (int kk = 0; kk < K; ++kk) {
          double acc = 0.0;
          for (int e = 0; e < E; ++e) acc += k2t[e] * dkap[e * K + kk];
          dkt[kk] = acc;
        }
        for (int e = 0; e < E; ++e) {
          double acc = 0.0;
          for (int kk = 0; kk < K; ++kk) acc += kt[kk] * dkap[e * K + kk];
          dk2t[e] = acc;
        }

        /* decay Sbar = a S_{t-1}: dg = a * <S_{t-1}, dSbar> = <Sbar, dSbar>,
           then dS_{t-1} = a dSbar */
        for (int e = 0; e < E; ++e) {
          const double a = exp(gt[e]);
          double acc = 0.0;
          double* drow = dS + e * KV;
          const double* sb = Sb + e * KV;
          for (size_t i = 0; i < KV; ++i) {
            acc += sb[i] * drow[i];
            drow[i] *= a;
          }
          dgt[e] = acc;
        }
      }
    }
    if (ds0) memcpy(ds0 + (size_t)bh * S_sz, dS, S_sz * sizeof(double));
    free(ck); free(seg); free(dS); free(Sb); free(tmpo); free(w); free(r);
    free(dw); free(dr); free(dkap); free(drho);
  }
  return fail ? -2 : 0;
}

/* Threads the OpenMP runtime will use (reported beside oracle timings). */
int oracle_num_threads(void) {
  int n = 1;
#pragma omp parallel
  {
#pragma omp single
    {
#ifdef _OPENMP
      n = omp_get_num_threads();
#endif
    }
  }
  return n;
}
