/*
 * carve_oracle.c -- plain, slow, double-precision CPU reference for the
 * chunked CARVE layer (arXiv 2606.27229).
 *
 * TEST INFRASTRUCTURE ONLY: used by the tests, the smoke check and the
 * CPU-baseline leg of the benchmark.  It shares no code with the HIP path.
 *
 * What is computed (per batch element b and head h, state S in R^{Dv x Dk}):
 *
 *   Chunk c covers tokens [cL, (c+1)L).  At the chunk boundary the state is
 *   frozen, S_hat = S (Sec. 4.2 "folded chunk-boundary state readout": the
 *   content signal is read from the state carried out of chunk c-1, Eq.
 *   content_readout; Alg. carve_fwd).  Then for every token t of the chunk:
 *
 *     F_b = Ub S_hat,  F_w = Uw S_hat                    (Eq. content_readout)
 *     tau_b = tanh(F_b q_t),  tau_w = tanh(F_w q_t)
 *     z_b = bx_t + Vb tau_b,  z_w = wx_t + Vw tau_w       (Eq. erase_gate)
 *     b = sigmoid(z_b),  w = sigmoid(z_w)
 *     alpha = exp(g_t) * (1 - b)        key-axis decay and erase (Eq. carve_state)
 *     e = w * v_t - S k_t               write gate scales v only (Alg. WYChunkDelta
 *                                       step 3: the gate never enters the coupling)
 *     S = S diag(alpha) + beta_t e k_t^T
 *     o_t = S q_t                       read-out after the update (Fig. carve_block,
 *                                       App. linearised cross-attention)
 *
 *   Readings where the paper is silent or inconsistent:
 *     - beta_t (a per-token scalar write strength) multiplies the whole write
 *       term; it is absent from the paper's CARVE equations and beta = 1
 *       recovers them.
 *     - the prediction uses the undecayed previous state (boxed Eq. carve_state).
 *     - chunk 0 folds S0 as well (the paper assumes S0 = 0, where the two
 *       readings coincide; folding S0 is what makes a split call equal a full
 *       call, Table exactness "chunk-by-chunk vs full call").
 *     - 1 - sigmoid(z) is evaluated as sigmoid(-z) (no cancellation).
 */
#include "carve_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* small helpers (scalar math only)                                          */
/* ------------------------------------------------------------------------ */

static double sigm(double z) { return 1.0 / (1.0 + exp(-z)); }

/* softplus(z) = log(1 + e^z), evaluated without overflow. */
static double softplus(double z) {
  if (z > 0.0) return z + log1p(exp(-z));
  return log1p(exp(z));
}

static int check_dims(const cref_dims* d) {
  if (!d) return -1;
  if (d->B <= 0 || d->T <= 0 || d->H <= 0 || d->Dk <= 0 || d->Dv <= 0 || d->R <= 0 || d->L <= 0)
    return -2;
  if (d->T % d->L != 0) return -2;
  return 0;
}

/* offsets of token rows */
static size_t row(const cref_dims* d, int b, int t, int h) {
  return ((size_t)b * d->T + t) * d->H + h;
}
static size_t state_off(const cref_dims* d, int b, int h) {
  return ((size_t)b * d->H + h) * (size_t)d->Dv * d->Dk;
}

/* ------------------------------------------------------------------------ */
/* a tiny thread pool: run job(i) for i in [0, njobs)                        */
/* ------------------------------------------------------------------------ */

typedef void (*job_fn)(void* ctx, int job);
typedef struct {
  job_fn fn;
  void* ctx;
  int njobs;
  int next;
  pthread_mutex_t mu;
} pool_t;

static void* pool_worker(void* arg) {
  pool_t* p = (pool_t*)arg;
  for (;;) {
    pthread_mutex_lock(&p->mu);
    int j = p->next++;
    pthread_mutex_unlock(&p->mu);
    if (j >= p->njobs) break;
    p->fn(p->ctx, j);
  }
  return NULL;
}

static void run_jobs(job_fn fn, void* ctx, int njobs, int nthreads) {
  if (nthreads <= 1 || njobs <= 1) {
    for (int j = 0; j < njobs; ++j) fn(ctx, j);
    return;
  }
  if (nthreads > njobs) nthreads = njobs;
  pool_t p;
  p.fn = fn;
  p.ctx = ctx;
  p.njobs = njobs;
  p.next = 0;
  pthread_mutex_init(&p.mu, NULL);
  pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nthreads);
  int started = 0;
  for (int i = 0; i < nthreads; ++i)
    if (pthread_create(&th[i], NULL, pool_worker, &p) == 0) ++started;
  if (started == 0) pool_worker(&p);
  for (int i = 0; i < started; ++i) pthread_join(th[i], NULL);
  free(th);
  pthread_mutex_destroy(&p.mu);
}

/* ------------------------------------------------------------------------ */
/* shared argument bundle                                                    */
/* ------------------------------------------------------------------------ */

typedef struct {
  const cref_dims* d;
  const double *q, *k, *v, *beta, *g, *bx, *wx, *Ub, *Uw, *Vb, *Vw, *S0;
  double *o, *S_T, *S_chunks, *gate_b, *gate_w;
  /* backward */
  const double *dO, *dS_T;
  double *dq, *dk, *dv, *dbeta, *dg, *dbx, *dwx, *dS0;
  double *pUb, *pUw, *pVb, *pVw; /* per-(b,h) partial parameter gradients */
} args_t;

/* ------------------------------------------------------------------------ */
/* 1. token-serial forward: the definition                                   */
/* ------------------------------------------------------------------------ */

static void serial_job(void* vctx, int job) {
  const args_t* a = (const args_t*)vctx;
  const cref_dims* d = a->d;
  const int Dk = d->Dk, Dv = d->Dv, R = d->R, L = d->L;
  const int b = job / d->H, h = job % d->H;
  const int nch = d->T / L;

  double* S = (double*)calloc((size_t)Dv * Dk, sizeof(double));
  double* Fb = (double*)malloc(sizeof(double) * (size_t)R * Dk);
  double* Fw = (double*)malloc(sizeof(double) * (size_t)R * Dk);
  double* tb = (double*)malloc(sizeof(double) * (size_t)R);
  double* tw = (double*)malloc(sizeof(double) * (size_t)R);
  double* alpha = (double*)malloc(sizeof(double) * (size_t)Dk);
  double* wg = (double*)malloc(sizeof(double) * (size_t)Dv);
  double* e = (double*)malloc(sizeof(double) * (size_t)Dv);

  if (a->S0) memcpy(S, a->S0 + state_off(d, b, h), sizeof(double) * (size_t)Dv * Dk);

  for (int c = 0; c < nch; ++c) {
    /* freeze the chunk-boundary state and fold the down-projections into it */
    if (a->S_chunks)
      memcpy(a->S_chunks + (((size_t)b * d->H + h) * nch + c) * (size_t)Dv * Dk, S,
             sizeof(double) * (size_t)Dv * Dk);
    for (int r = 0; r < R; ++r)
      for (int j = 0; j < Dk; ++j) {
        double sb = 0.0, sw = 0.0;
        for (int i = 0; i < Dv; ++i) {
          sb += a->Ub[(size_t)r * Dv + i] * S[(size_t)i * Dk + j];
          sw += a->Uw[(size_t)r * Dv + i] * S[(size_t)i * Dk + j];
        }
        Fb[(size_t)r * Dk + j] = sb;
        Fw[(size_t)r * Dk + j] = sw;
      }

    for (int t = c * L; t < (c + 1) * L; ++t) {
      const size_t rw = row(d, b, t, h);
      const double* qt = a->q + rw * Dk;
      const double* kt = a->k + rw * Dk;
      const double* vt = a->v + rw * Dv;
      const double* gt = a->g + rw * Dk;
      const double* bxt = a->bx + rw * Dk;
      const double* wxt = a->wx + rw * Dv;
      const double bt = a->beta[rw];

      for (int r = 0; r < R; ++r) {
        double sb = 0.0, sw = 0.0;
        for (int j = 0; j < Dk; ++j) {
          sb += Fb[(size_t)r * Dk + j] * qt[j];
          sw += Fw[(size_t)r * Dk + j] * qt[j];
        }
        tb[r] = tanh(sb);
        tw[r] = tanh(sw);
      }
      for (int j = 0; j < Dk; ++j) {
        double s = 0.0;
        for (int r = 0; r < R; ++r) s += a->Vb[(size_t)j * R + r] * tb[r];
        const double zb = bxt[j] + s;
        alpha[j] = exp(gt[j]) * sigm(-zb);
        if (a->gate_b) a->gate_b[rw * Dk + j] = sigm(zb);
      }
      for (int i = 0; i < Dv; ++i) {
        double s = 0.0;
        for (int r = 0; r < R; ++r) s += a->Vw[(size_t)i * R + r] * tw[r];
        wg[i] = sigm(wxt[i] + s);
        if (a->gate_w) a->gate_w[rw * Dv + i] = wg[i];
      }
      /* prediction error with the undecayed previous state */
      for (int i = 0; i < Dv; ++i) {
        double p = 0.0;
        for (int j = 0; j < Dk; ++j) p += S[(size_t)i * Dk + j] * kt[j];
        e[i] = wg[i] * vt[i] - p;
      }
      for (int i = 0; i < Dv; ++i)
        for (int j = 0; j < Dk; ++j)
          S[(size_t)i * Dk + j] = S[(size_t)i * Dk + j] * alpha[j] + bt * e[i] * kt[j];
      for (int i = 0; i < Dv; ++i) {
        double s = 0.0;
        for (int j = 0; j < Dk; ++j) s += S[(size_t)i * Dk + j] * qt[j];
        a->o[rw * Dv + i] = s;
      }
    }
  }
  if (a->S_T) memcpy(a->S_T + state_off(d, b, h), S, sizeof(double) * (size_t)Dv * Dk);
  free(S); free(Fb); free(Fw); free(tb); free(tw); free(alpha); free(wg); free(e);
}

int cref_fwd_serial(const cref_dims* d, const double* q, const double* k, const double* v,
                    const double* beta, const double* g, const double* bx, const double* wx,
                    const double* Ub, const double* Uw, const double* Vb, const double* Vw,
                    const double* S0, double* o, double* S_T, double* S_chunks,
                    double* gate_b, double* gate_w, int nthreads) {
  int st = check_dims(d);
  if (st) return st;
  if (!q || !k || !v || !beta || !g || !bx || !wx || !Ub || !Uw || !Vb || !Vw || !o) return -1;
  args_t a;
  memset(&a, 0, sizeof(a));
  a.d = d; a.q = q; a.k = k; a.v = v; a.beta = beta; a.g = g; a.bx = bx; a.wx = wx;
  a.Ub = Ub; a.Uw = Uw; a.Vb = Vb; a.Vw = Vw; a.S0 = S0;
  a.o = o; a.S_T = S_T; a.S_chunks = S_chunks; a.gate_b = gate_b; a.gate_w = gate_w;
  run_jobs(serial_job, &a, d->B * d->H, nthreads);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* 2. chunked WY form (Sec. 6.2), plain loops                                */
/*                                                                           */
/* Within a chunk let l_t = g_t - softplus(z_b,t) = log(exp(g_t)(1-b_t)) and */
/* Lam_t = sum_{s<=t} l_s (Eq. gamma_cum in log space, Lam_{-1} = 0).        */
/* With u_t = beta_t (w_t*v_t - S_{t-1} k_t) the recurrence unrolls to       */
/*   S_t = S_hat diag(e^{Lam_t}) + sum_{s<=t} u_s k_s^T diag(e^{Lam_t-Lam_s}) */
/* so (I + A) u = diag(beta)(w*V - Ktil S_hat^T) with                         */
/*   A_ts = beta_t sum_j k_t[j] k_s[j] e^{Lam_{t-1}[j]-Lam_s[j]}   (s < t)     */
/*   Ktil_t = k_t * e^{Lam_{t-1}}                                             */
/* (the coupling of Eq. M_coupling with the retention ratio taken from the    */
/* recurrence itself), solved by forward substitution (Alg. step 5).          */
/* Outputs and the carried state (Alg. steps 6-7 with the intra-chunk decay   */
/* ratios restored):                                                          */
/*   o_t    = S_hat (e^{Lam_t} * q_t) + sum_{s<=t} u_s [k_s . (e^{Lam_t-Lam_s} q_t)] */
/*   S_next = S_hat diag(e^{Lam_{L-1}}) + sum_s u_s (k_s * e^{Lam_{L-1}-Lam_s})^T */
/* Every exponent is a difference Lam_a - Lam_b with a >= b, so it is <= 0.   */
/* ------------------------------------------------------------------------ */

static void chunked_job(void* vctx, int job) {
  const args_t* a = (const args_t*)vctx;
  const cref_dims* d = a->d;
  const int Dk = d->Dk, Dv = d->Dv, R = d->R, L = d->L;
  const int b = job / d->H, h = job % d->H;
  const int nch = d->T / L;

  double* S = (double*)calloc((size_t)Dv * Dk, sizeof(double));
  double* Sn = (double*)malloc(sizeof(double) * (size_t)Dv * Dk);
  double* F = (double*)malloc(sizeof(double) * (size_t)2 * R * Dk); /* [F_b; F_w] */
  double* Lam = (double*)malloc(sizeof(double) * (size_t)L * Dk);
  double* W = (double*)malloc(sizeof(double) * (size_t)L * Dv);   /* write gate */
  double* A = (double*)calloc((size_t)L * L, sizeof(double));
  double* U = (double*)malloc(sizeof(double) * (size_t)L * Dv);
  double* tau = (double*)malloc(sizeof(double) * (size_t)2 * R);

  if (a->S0) memcpy(S, a->S0 + state_off(d, b, h), sizeof(double) * (size_t)Dv * Dk);

  for (int c = 0; c < nch; ++c) {
    const int t0 = c * L;
    if (a->S_chunks)
      memcpy(a->S_chunks + (((size_t)b * d->H + h) * nch + c) * (size_t)Dv * Dk, S,
             sizeof(double) * (size_t)Dv * Dk);
    /* fold: F = [Ub; Uw] S_hat  (2R x Dk) */
    for (int r = 0; r < 2 * R; ++r) {
      const double* Urow = (r < R) ? a->Ub + (size_t)r * Dv : a->Uw + (size_t)(r - R) * Dv;
      for (int j = 0; j < Dk; ++j) {
        double s = 0.0;
        for (int i = 0; i < Dv; ++i) s += Urow[i] * S[(size_t)i * Dk + j];
        F[(size_t)r * Dk + j] = s;
      }
    }
    /* gates and log-retention prefix sums */
    for (int tt = 0; tt < L; ++tt) {
      const size_t rw = row(d, b, t0 + tt, h);
      const double* qt = a->q + rw * Dk;
      for (int r = 0; r < 2 * R; ++r) {
        double s = 0.0;
        for (int j = 0; j < Dk; ++j) s += F[(size_t)r * Dk + j] * qt[j];
        tau[r] = tanh(s);
      }
      for (int j = 0; j < Dk; ++j) {
        double s = 0.0;
        for (int r = 0; r < R; ++r) s += a->Vb[(size_t)j * R + r] * tau[r];
        const double zb = a->bx[rw * Dk + j] + s;
        const double ell = a->g[rw * Dk + j] - softplus(zb);
        Lam[(size_t)tt * Dk + j] = (tt == 0 ? 0.0 : Lam[(size_t)(tt - 1) * Dk + j]) + ell;
        if (a->gate_b) a->gate_b[rw * Dk + j] = sigm(zb);
      }
      for (int i = 0; i < Dv; ++i) {
        double s = 0.0;
        for (int r = 0; r < R; ++r) s += a->Vw[(size_t)i * R + r] * tau[R + r];
        W[(size_t)tt * Dv + i] = sigm(a->wx[rw * Dv + i] + s);
        if (a->gate_w) a->gate_w[rw * Dv + i] = W[(size_t)tt * Dv + i];
      }
    }
    /* coupling A (strictly lower) */
    for (int tt = 0; tt < L; ++tt) {
      const size_t rt = row(d, b, t0 + tt, h);
      for (int ss = 0; ss < tt; ++ss) {
        const size_t rs = row(d, b, t0 + ss, h);
        double s = 0.0;
        for (int j = 0; j < Dk; ++j)
          s += a->k[rt * Dk + j] * a->k[rs * Dk + j] *
               exp(Lam[(size_t)(tt - 1) * Dk + j] - Lam[(size_t)ss * Dk + j]);
        A[(size_t)tt * L + ss] = a->beta[rt] * s;
      }
    }
    /* right-hand sides, then forward substitution u_t = r_t - sum_{s<t} A_ts u_s */
    for (int tt = 0; tt < L; ++tt) {
      const size_t rt = row(d, b, t0 + tt, h);
      for (int i = 0; i < Dv; ++i) {
        double p = 0.0;
        for (int j = 0; j < Dk; ++j) {
          const double lam_prev = (tt == 0) ? 0.0 : Lam[(size_t)(tt - 1) * Dk + j];
          p += S[(size_t)i * Dk + j] * a->k[rt * Dk + j] * exp(lam_prev);
        }
        double rhs = a->beta[rt] * (W[(size_t)tt * Dv + i] * a->v[rt * Dv + i] - p);
        for (int ss = 0; ss < tt; ++ss) rhs -= A[(size_t)tt * L + ss] * U[(size_t)ss * Dv + i];
        U[(size_t)tt * Dv + i] = rhs;
      }
    }
    /* outputs */
    for (int tt = 0; tt < L; ++tt) {
      const size_t rt = row(d, b, t0 + tt, h);
      const double* qt = a->q + rt * Dk;
      for (int i = 0; i < Dv; ++i) {
        double s = 0.0;
        for (int j = 0; j < Dk; ++j)
          s += S[(size_t)i * Dk + j] * qt[j] * exp(Lam[(size_t)tt * Dk + j]);
        a->o[rt * Dv + i] = s;
      }
      for (int ss = 0; ss <= tt; ++ss) {
        const size_t rs = row(d, b, t0 + ss, h);
        double p = 0.0;
        for (int j = 0; j < Dk; ++j)
          p += a->k[rs * Dk + j] * qt[j] *
               exp(Lam[(size_t)tt * Dk + j] - Lam[(size_t)ss * Dk + j]);
        for (int i = 0; i < Dv; ++i) a->o[rt * Dv + i] += p * U[(size_t)ss * Dv + i];
      }
    }
    /* carried state */
    for (int i = 0; i < Dv; ++i)
      for (int j = 0; j < Dk; ++j) {
        const double lam_end = Lam[(size_t)(L - 1) * Dk + j];
        double s = S[(size_t)i * Dk + j] * exp(lam_end);
        for (int ss = 0; ss < L; ++ss) {
          const size_t rs = row(d, b, t0 + ss, h);
          s += U[(size_t)ss * Dv + i] * a->k[rs * Dk + j] *
               exp(lam_end - Lam[(size_t)ss * Dk + j]);
        }
        Sn[(size_t)i * Dk + j] = s;
      }
    memcpy(S, Sn, sizeof(double) * (size_t)Dv * Dk);
  }
  if (a->S_T) memcpy(a->S_T + state_off(d, b, h), S, sizeof(double) * (size_t)Dv * Dk);
  free(S); free(Sn); free(F); free(Lam); free(W); free(A); free(U); free(tau);
}

int cref_fwd_chunked(const cref_dims* d, const double* q, const double* k, const double* v,
                     const double* beta, const double* g, const double* bx, const double* wx,
                     const double* Ub, const double* Uw, const double* Vb, const double* Vw,
                     const double* S0, double* o, double* S_T, double* S_chunks,
                     double* gate_b, double* gate_w, int nthreads) {
  int st = check_dims(d);
  if (st) return st;
  if (!q || !k || !v || !beta || !g || !bx || !wx || !Ub || !Uw || !Vb || !Vw || !o) return -1;
  args_t a;
  memset(&a, 0, sizeof(a));
  a.d = d; a.q = q; a.k = k; a.v = v; a.beta = beta; a.g = g; a.bx = bx; a.wx = wx;
  a.Ub = Ub; a.Uw = Uw; a.Vb = Vb; a.Vw = Vw; a.S0 = S0;
  a.o = o; a.S_T = S_T; a.S_chunks = S_chunks; a.gate_b = gate_b; a.gate_w = gate_w;
  run_jobs(chunked_job, &a, d->B * d->H, nthreads);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* 3. memory-blind baseline: gates from the projections alone                */
/* ------------------------------------------------------------------------ */

static void baseline_job(void* vctx, int job) {
  const args_t* a = (const args_t*)vctx;
  const cref_dims* d = a->d;
  const int Dk = d->Dk, Dv = d->Dv;
  const int b = job / d->H, h = job % d->H;
  double* M = (double*)calloc((size_t)Dv * Dk, sizeof(double));
  double* pred = (double*)malloc(sizeof(double) * (size_t)Dv);
  if (a->S0) memcpy(M, a->S0 + state_off(d, b, h), sizeof(double) * (size_t)Dv * Dk);
  for (int t = 0; t < d->T; ++t) {
    const size_t rw = row(d, b, t, h);
    const double* kt = a->k + rw * Dk;
    for (int i = 0; i < Dv; ++i) {
      double p = 0.0;
      for (int j = 0; j < Dk; ++j) p += M[(size_t)i * Dk + j] * kt[j];
      pred[i] = p;
    }
    for (int i = 0; i < Dv; ++i) {
      const double err = sigm(a->wx[rw * Dv + i]) * a->v[rw * Dv + i] - pred[i];
      for (int j = 0; j < Dk; ++j) {
        const double keep = exp(a->g[rw * Dk + j]) * sigm(-a->bx[rw * Dk + j]);
        M[(size_t)i * Dk + j] = M[(size_t)i * Dk + j] * keep + a->beta[rw] * err * kt[j];
      }
    }
    for (int i = 0; i < Dv; ++i) {
      double s = 0.0;
      for (int j = 0; j < Dk; ++j) s += M[(size_t)i * Dk + j] * a->q[rw * Dk + j];
      a->o[rw * Dv + i] = s;
    }
  }
  if (a->S_T) memcpy(a->S_T + state_off(d, b, h), M, sizeof(double) * (size_t)Dv * Dk);
  free(M); free(pred);
}

int cref_baseline_fwd(const cref_dims* d, const double* q, const double* k, const double* v,
                      const double* beta, const double* g, const double* bx, const double* wx,
                      const double* S0, double* o, double* S_T, int nthreads) {
  int st = check_dims(d);
  if (st) return st;
  if (!q || !k || !v || !beta || !g || !bx || !wx || !o) return -1;
  args_t a;
  memset(&a, 0, sizeof(a));
  a.d = d; a.q = q; a.k = k; a.v = v; a.beta = beta; a.g = g; a.bx = bx; a.wx = wx;
  a.S0 = S0; a.o = o; a.S_T = S_T;
  run_jobs(baseline_job, &a, d->B * d->H, nthreads);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* 4. backward: exact reverse mode of the token-serial forward               */
/*                                                                           */
/* The forward is re-run keeping only the chunk-boundary states; inside each */
/* chunk (processed last to first) the token states are recomputed from that */
/* checkpoint and swept in reverse.  For token t, with dS the gradient with  */
/* respect to S_t:                                                           */
/*   dS += do_t q_t^T ; dq_t = S_t^T do_t                                     */
/*   dalpha = colsum(S_{t-1} * dS) ; dbeta = e . (dS k) ; de = beta dS k      */
/*   dk_t = beta dS^T e - S_{t-1}^T de ; dv = w * de ; dw = v * de            */
/*   dS <- dS diag(alpha) - de k^T                                           */
/*   dg = dalpha * alpha ; dz_b = -dalpha * alpha * b ; dz_w = dw w (1-w)     */
/*   dVb += dz_b tau_b^T ; dVw += dz_w tau_w^T                               */
/*   dY = (V^T dz) (1 - tau^2) ; dF += dY q^T ; dq_t += F^T dY                */
/* and at the first token of the chunk the folded read-out closes the chain  */
/* (the "glue" of App. Alg. megakernel_bwd):                                 */
/*   dUb += dF_b S_hat^T ; dUw += dF_w S_hat^T ; dS += Ub^T dF_b + Uw^T dF_w. */
/* The paper's listing of this backward is internally inconsistent (it puts  */
/* w on the whole prediction error); the steps above are derived directly   */
/* from the forward in this file and checked against finite differences.    */
/* ------------------------------------------------------------------------ */

static void bwd_job(void* vctx, int job) {
  const args_t* a = (const args_t*)vctx;
  const cref_dims* d = a->d;
  const int Dk = d->Dk, Dv = d->Dv, R = d->R, L = d->L;
  const int b = job / d->H, h = job % d->H;
  const int nch = d->T / L;
  const size_t SS = (size_t)Dv * Dk;

  double* ck = (double*)malloc(sizeof(double) * SS * (size_t)nch); /* chunk checkpoints */
  double* St = (double*)malloc(sizeof(double) * SS * (size_t)(L + 1)); /* states in a chunk */
  double* Fb = (double*)malloc(sizeof(double) * (size_t)R * Dk);
  double* Fw = (double*)malloc(sizeof(double) * (size_t)R * Dk);
  double* TB = (double*)malloc(sizeof(double) * (size_t)L * R);
  double* TW = (double*)malloc(sizeof(double) * (size_t)L * R);
  double* BG = (double*)malloc(sizeof(double) * (size_t)L * Dk); /* erase gate */
  double* AL = (double*)malloc(sizeof(double) * (size_t)L * Dk); /* alpha */
  double* WG = (double*)malloc(sizeof(double) * (size_t)L * Dv); /* write gate */
  double* E = (double*)malloc(sizeof(double) * (size_t)L * Dv);  /* prediction error */
  double* dS = (double*)calloc(SS, sizeof(double));
  double* dFb = (double*)malloc(sizeof(double) * (size_t)R * Dk);
  double* dFw = (double*)malloc(sizeof(double) * (size_t)R * Dk);
  double* dal = (double*)malloc(sizeof(double) * (size_t)Dk);
  double* dSk = (double*)malloc(sizeof(double) * (size_t)Dv);
  double* de = (double*)malloc(sizeof(double) * (size_t)Dv);
  double* dzb = (double*)malloc(sizeof(double) * (size_t)Dk);
  double* dzw = (double*)malloc(sizeof(double) * (size_t)Dv);
  double* dYb = (double*)malloc(sizeof(double) * (size_t)R);
  double* dYw = (double*)malloc(sizeof(double) * (size_t)R);
  double* pUb = a->pUb + (size_t)job * R * Dv;
  double* pUw = a->pUw + (size_t)job * R * Dv;
  double* pVb = a->pVb + (size_t)job * Dk * R;
  double* pVw = a->pVw + (size_t)job * Dv * R;
  memset(pUb, 0, sizeof(double) * (size_t)R * Dv);
  memset(pUw, 0, sizeof(double) * (size_t)R * Dv);
  memset(pVb, 0, sizeof(double) * (size_t)Dk * R);
  memset(pVw, 0, sizeof(double) * (size_t)Dv * R);

  /* chunk step: given S_hat (=St[0]) fill St[1..L] and the per-token gate
   * quantities of chunk c.  Same arithmetic as the serial forward. */
#define CHUNK_RECOMPUTE(c)                                                            \
  do {                                                                                \
    const double* Sh = St;                                                            \
    for (int r = 0; r < R; ++r)                                                       \
      for (int j = 0; j < Dk; ++j) {                                                  \
        double sb = 0.0, sw = 0.0;                                                    \
        for (int i = 0; i < Dv; ++i) {                                                \
          sb += a->Ub[(size_t)r * Dv + i] * Sh[(size_t)i * Dk + j];                   \
          sw += a->Uw[(size_t)r * Dv + i] * Sh[(size_t)i * Dk + j];                   \
        }                                                                             \
        Fb[(size_t)r * Dk + j] = sb;                                                  \
        Fw[(size_t)r * Dk + j] = sw;                                                  \
      }                                                                               \
    for (int tt = 0; tt < L; ++tt) {                                                  \
      const size_t rw = row(d, b, (c) * L + tt, h);                                   \
      const double* qt = a->q + rw * Dk;                                              \
      const double* kt = a->k + rw * Dk;                                              \
      const double* Sp = St + (size_t)tt * SS;                                        \
      double* Sx = St + (size_t)(tt + 1) * SS;                                        \
      for (int r = 0; r < R; ++r) {                                                   \
        double sb = 0.0, sw = 0.0;                                                    \
        for (int j = 0; j < Dk; ++j) {                                                \
          sb += Fb[(size_t)r * Dk + j] * qt[j];                                       \
          sw += Fw[(size_t)r * Dk + j] * qt[j];                                       \
        }                                                                             \
        TB[(size_t)tt * R + r] = tanh(sb);                                            \
        TW[(size_t)tt * R + r] = tanh(sw);                                            \
      }                                                                               \
      for (int j = 0; j < Dk; ++j) {                                                  \
        double s = 0.0;                                                               \
        for (int r = 0; r < R; ++r) s += a->Vb[(size_t)j * R + r] * TB[(size_t)tt * R + r]; \
        const double zb = a->bx[rw * Dk + j] + s;                                     \
        BG[(size_t)tt * Dk + j] = sigm(zb);                                           \
        AL[(size_t)tt * Dk + j] = exp(a->g[rw * Dk + j]) * sigm(-zb);                 \
      }                                                                               \
      for (int i = 0; i < Dv; ++i) {                                                  \
        double s = 0.0;                                                               \
        for (int r = 0; r < R; ++r) s += a->Vw[(size_t)i * R + r] * TW[(size_t)tt * R + r]; \
        WG[(size_t)tt * Dv + i] = sigm(a->wx[rw * Dv + i] + s);                       \
      }                                                                               \
      for (int i = 0; i < Dv; ++i) {                                                  \
        double p = 0.0;                                                               \
        for (int j = 0; j < Dk; ++j) p += Sp[(size_t)i * Dk + j] * kt[j];             \
        E[(size_t)tt * Dv + i] = WG[(size_t)tt * Dv + i] * a->v[rw * Dv + i] - p;     \
      }                                                                               \
      for (int i = 0; i < Dv; ++i)                                                    \
        for (int j = 0; j < Dk; ++j)                                                  \
          Sx[(size_t)i * Dk + j] = Sp[(size_t)i * Dk + j] * AL[(size_t)tt * Dk + j] + \
                                   a->beta[rw] * E[(size_t)tt * Dv + i] * kt[j];      \
    }                                                                                 \
  } while (0)

  /* forward sweep: checkpoints only */
  if (a->S0)
    memcpy(St, a->S0 + state_off(d, b, h), sizeof(double) * SS);
  else
    memset(St, 0, sizeof(double) * SS);
  for (int c = 0; c < nch; ++c) {
    memcpy(ck + (size_t)c * SS, St, sizeof(double) * SS);
    CHUNK_RECOMPUTE(c);
    memcpy(St, St + (size_t)L * SS, sizeof(double) * SS);
  }

  if (a->dS_T) memcpy(dS, a->dS_T + state_off(d, b, h), sizeof(double) * SS);

  for (int c = nch - 1; c >= 0; --c) {
    memcpy(St, ck + (size_t)c * SS, sizeof(double) * SS);
    CHUNK_RECOMPUTE(c);
    memset(dFb, 0, sizeof(double) * (size_t)R * Dk);
    memset(dFw, 0, sizeof(double) * (size_t)R * Dk);
    for (int tt = L - 1; tt >= 0; --tt) {
      const size_t rw = row(d, b, c * L + tt, h);
      const double* qt = a->q + rw * Dk;
      const double* kt = a->k + rw * Dk;
      const double* vt = a->v + rw * Dv;
      const double* dot = a->dO + rw * Dv;
      const double* Sp = St + (size_t)tt * SS;
      const double* Sx = St + (size_t)(tt + 1) * SS;
      const double bt = a->beta[rw];
      double* dqt = a->dq + rw * Dk;
      double* dkt = a->dk + rw * Dk;

      /* read-out o_t = S_t q_t */
      for (int i = 0; i < Dv; ++i)
        for (int j = 0; j < Dk; ++j) dS[(size_t)i * Dk + j] += dot[i] * qt[j];
      for (int j = 0; j < Dk; ++j) {
        double s = 0.0;
        for (int i = 0; i < Dv; ++i) s += Sx[(size_t)i * Dk + j] * dot[i];
        dqt[j] = s;
      }
      /* S_t = S_{t-1} diag(alpha) + beta e k^T */
      for (int j = 0; j < Dk; ++j) {
        double s = 0.0;
        for (int i = 0; i < Dv; ++i) s += Sp[(size_t)i * Dk + j] * dS[(size_t)i * Dk + j];
        dal[j] = s;
      }
      double dbt = 0.0;
      for (int i = 0; i < Dv; ++i) {
        double s = 0.0;
        for (int j = 0; j < Dk; ++j) s += dS[(size_t)i * Dk + j] * kt[j];
        dSk[i] = s;
        de[i] = bt * s;
        dbt += E[(size_t)tt * Dv + i] * s;
      }
      a->dbeta[rw] = dbt;
      for (int j = 0; j < Dk; ++j) {
        double s1 = 0.0, s2 = 0.0;
        for (int i = 0; i < Dv; ++i) {
          s1 += dS[(size_t)i * Dk + j] * E[(size_t)tt * Dv + i];
          s2 += Sp[(size_t)i * Dk + j] * de[i];
        }
        dkt[j] = bt * s1 - s2;
      }
      /* e = w*v - S_{t-1} k */
      for (int i = 0; i < Dv; ++i) {
        const double w = WG[(size_t)tt * Dv + i];
        a->dv[rw * Dv + i] = w * de[i];
        const double dw = vt[i] * de[i];
        dzw[i] = dw * w * (1.0 - w);
        a->dwx[rw * Dv + i] = dzw[i];
      }
      for (int i = 0; i < Dv; ++i)
        for (int j = 0; j < Dk; ++j)
          dS[(size_t)i * Dk + j] = dS[(size_t)i * Dk + j] * AL[(size_t)tt * Dk + j] - de[i] * kt[j];
      /* alpha = exp(g) sigmoid(-z_b) */
      for (int j = 0; j < Dk; ++j) {
        const double al = AL[(size_t)tt * Dk + j];
        a->dg[rw * Dk + j] = dal[j] * al;
        dzb[j] = -dal[j] * al * BG[(size_t)tt * Dk + j];
        a->dbx[rw * Dk + j] = dzb[j];
      }
      /* z = x + V tau ; tau = tanh(F q) */
      for (int j = 0; j < Dk; ++j)
        for (int r = 0; r < R; ++r) pVb[(size_t)j * R + r] += dzb[j] * TB[(size_t)tt * R + r];
      for (int i = 0; i < Dv; ++i)
        for (int r = 0; r < R; ++r) pVw[(size_t)i * R + r] += dzw[i] * TW[(size_t)tt * R + r];
      for (int r = 0; r < R; ++r) {
        double sb = 0.0, sw = 0.0;
        for (int j = 0; j < Dk; ++j) sb += a->Vb[(size_t)j * R + r] * dzb[j];
        for (int i = 0; i < Dv; ++i) sw += a->Vw[(size_t)i * R + r] * dzw[i];
        const double tbv = TB[(size_t)tt * R + r], twv = TW[(size_t)tt * R + r];
        dYb[r] = sb * (1.0 - tbv * tbv);
        dYw[r] = sw * (1.0 - twv * twv);
      }
      for (int r = 0; r < R; ++r)
        for (int j = 0; j < Dk; ++j) {
          dFb[(size_t)r * Dk + j] += dYb[r] * qt[j];
          dFw[(size_t)r * Dk + j] += dYw[r] * qt[j];
        }
      for (int j = 0; j < Dk; ++j) {
        double s = 0.0;
        for (int r = 0; r < R; ++r)
          s += Fb[(size_t)r * Dk + j] * dYb[r] + Fw[(size_t)r * Dk + j] * dYw[r];
        dqt[j] += s;
      }
    }
    /* glue: F = U S_hat with S_hat = St[0] */
    for (int r = 0; r < R; ++r)
      for (int i = 0; i < Dv; ++i) {
        double sb = 0.0, sw = 0.0;
        for (int j = 0; j < Dk; ++j) {
          sb += dFb[(size_t)r * Dk + j] * St[(size_t)i * Dk + j];
          sw += dFw[(size_t)r * Dk + j] * St[(size_t)i * Dk + j];
        }
        pUb[(size_t)r * Dv + i] += sb;
        pUw[(size_t)r * Dv + i] += sw;
      }
    for (int i = 0; i < Dv; ++i)
      for (int j = 0; j < Dk; ++j) {
        double s = 0.0;
        for (int r = 0; r < R; ++r)
          s += a->Ub[(size_t)r * Dv + i] * dFb[(size_t)r * Dk + j] +
               a->Uw[(size_t)r * Dv + i] * dFw[(size_t)r * Dk + j];
        dS[(size_t)i * Dk + j] += s;
      }
  }
  if (a->dS0) memcpy(a->dS0 + state_off(d, b, h), dS, sizeof(double) * SS);
#undef CHUNK_RECOMPUTE
  free(ck); free(St); free(Fb); free(Fw); free(TB); free(TW); free(BG); free(AL); free(WG);
  free(E); free(dS); free(dFb); free(dFw); free(dal); free(dSk); free(de); free(dzb);
  free(dzw); free(dYb); free(dYw);
}

int cref_bwd(const cref_dims* d, const double* q, const double* k, const double* v,
             const double* beta, const double* g, const double* bx, const double* wx,
             const double* Ub, const double* Uw, const double* Vb, const double* Vw,
             const double* S0, const double* dO, const double* dS_T,
             double* dq, double* dk, double* dv, double* dbeta, double* dg,
             double* dbx, double* dwx, double* dUb, double* dUw, double* dVb,
             double* dVw, double* dS0, int nthreads) {
  int st = check_dims(d);
  if (st) return st;
  if (!q || !k || !v || !beta || !g || !bx || !wx || !Ub || !Uw || !Vb || !Vw || !dO || !dq ||
      !dk || !dv || !dbeta || !dg || !dbx || !dwx || !dUb || !dUw || !dVb || !dVw)
    return -1;
  const int nj = d->B * d->H;
  const int R = d->R, Dk = d->Dk, Dv = d->Dv;
  args_t a;
  memset(&a, 0, sizeof(a));
  a.d = d; a.q = q; a.k = k; a.v = v; a.beta = beta; a.g = g; a.bx = bx; a.wx = wx;
  a.Ub = Ub; a.Uw = Uw; a.Vb = Vb; a.Vw = Vw; a.S0 = S0;
  a.dO = dO; a.dS_T = dS_T; a.dq = dq; a.dk = dk; a.dv = dv; a.dbeta = dbeta; a.dg = dg;
  a.dbx = dbx; a.dwx = dwx; a.dS0 = dS0;
  a.pUb = (double*)malloc(sizeof(double) * (size_t)nj * R * Dv);
  a.pUw = (double*)malloc(sizeof(double) * (size_t)nj * R * Dv);
  a.pVb = (double*)malloc(sizeof(double) * (size_t)nj * Dk * R);
  a.pVw = (double*)malloc(sizeof(double) * (size_t)nj * Dv * R);
  run_jobs(bwd_job, &a, nj, nthreads);
  /* parameters are shared by all heads: reduce the partials in (b,h) order */
  memset(dUb, 0, sizeof(double) * (size_t)R * Dv);
  memset(dUw, 0, sizeof(double) * (size_t)R * Dv);
  memset(dVb, 0, sizeof(double) * (size_t)Dk * R);
  memset(dVw, 0, sizeof(double) * (size_t)Dv * R);
  for (int jb = 0; jb < nj; ++jb) {
    for (size_t x = 0; x < (size_t)R * Dv; ++x) {
      dUb[x] += a.pUb[(size_t)jb * R * Dv + x];
      dUw[x] += a.pUw[(size_t)jb * R * Dv + x];
    }
    for (size_t x = 0; x < (size_t)Dk * R; ++x) dVb[x] += a.pVb[(size_t)jb * Dk * R + x];
    for (size_t x = 0; x < (size_t)Dv * R; ++x) dVw[x] += a.pVw[(size_t)jb * Dv * R + x];
  }
  free(a.pUb); free(a.pUw); free(a.pVb); free(a.pVw);
  return 0;
}

/* ------------------------------------------------------------------------ */
/* key-axis decay gate computed from its raw logit (Sec. decay_gate)        */
/* ------------------------------------------------------------------------ */

/* g = -exp(A) * softplus(f + tau) per key channel (Eq. decay_gate), with the
 * learned log-amplitudes A and biases tau of head h shared by every token. */
int cref_decay_gate(const cref_dims* d, const double* f, const double* A, const double* tau, double* g) {
  int st = check_dims(d);
  if (st) return st;
  if (!f || !A || !tau || !g) return -1;
  for (int b = 0; b < d->B; ++b)
    for (int t = 0; t < d->T; ++t)
      for (int h = 0; h < d->H; ++h) {
        const size_t r = row(d, b, t, h) * d->Dk;
        for (int j = 0; j < d->Dk; ++j) {
          const size_t p = (size_t)h * d->Dk + j;
          g[r + j] = -exp(A[p]) * softplus(f[r + j] + tau[p]);
        }
      }
  return 0;
}

/* Reverse mode of cref_decay_gate for an incoming gradient dg:
 *   dg/df = dg/dtau = -exp(A) * sigmoid(f + tau)   (d softplus(z)/dz = sigmoid(z))
 *   dg/dA = g
 * df is per token; dA and dtau are summed over batch and tokens in the
 * order b, t (overwritten, not accumulated). */
int cref_decay_gate_bwd(const cref_dims* d, const double* f, const double* A, const double* tau,
                        const double* dg, double* df, double* dA, double* dtau) {
  int st = check_dims(d);
  if (st) return st;
  if (!f || !A || !tau || !dg || !df || !dA || !dtau) return -1;
  const size_t np = (size_t)d->H * d->Dk;
  for (size_t p = 0; p < np; ++p) dA[p] = dtau[p] = 0.0;
  for (int b = 0; b < d->B; ++b)
    for (int t = 0; t < d->T; ++t)
      for (int h = 0; h < d->H; ++h) {
        const size_t r = row(d, b, t, h) * d->Dk;
        for (int j = 0; j < d->Dk; ++j) {
          const size_t p = (size_t)h * d->Dk + j;
          const double z = f[r + j] + tau[p];
          const double ea = exp(A[p]);
          const double g = -ea * softplus(z);
          const double dfz = dg[r + j] * (-ea * sigm(z));
          df[r + j] = dfz;
          dtau[p] += dfz;
          dA[p] += dg[r + j] * g;
        }
      }
  return 0;
}
