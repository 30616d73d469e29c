/*
 * bcjr_oracle.c -- plain fp64 CPU oracle.  TEST INFRASTRUCTURE ONLY: the
 * product path never links or calls it (see bcjr_oracle.h).
 *
 * Everything is written from the definitions, state by state, with no
 * grouping of states, no tiling and no reordering beyond what the equations
 * state:
 *   - the trellis (paper Sec. 3.1): next(s, b) = ((s << k) | b) & (S - 1);
 *   - the local field h_t(s) = -(w_t - c(s))^2 / (2T) (Sec. 3.3, Eq. boltzmann);
 *   - the forward / backward partition functions and their linear
 *     recursions through the transfer matrix T_{s->s'} = 1[next(s, .) = s']
 *     (Sec. 3.4, Eqs. alpha, beta and the two recursions that follow them),
 *     carried in the log domain (Sec. 3.4, "Numerical stability");
 *   - the marginal p_T(s_t = s) = alpha_t(s) beta_t(s) / Z_T and
 *     Z_T = sum_s alpha_t(s) beta_t(s) (Eq. marginal);
 *   - the soft codeword  sum_s c(s) p_T(s_t = s)  (Eqs. soft-codeword,
 *     softcode-final);
 *   - the VJP.  The paper gives no formula for its backward pass (Sec. 3.5
 *     only names an implicit-differentiation shortcut), so it is derived
 *     from Eq. boltzmann: with F = sum_t g_t c(s_t),  <g, w_soft> = E_p[F],
 *     and since d(-E/T)/dw_tau = -(w_tau - c(s_tau))/T,
 *        dW_tau = Cov_p(F, c(s_tau)) / T,
 *        dc_sig = sum_t p_t(sig) [ g_t + (w_t - c_sig)(E[F | s_t = sig] - E[F]) / T ].
 *     E[F | s_t = s] = A_t(s) + B_t(s) splits into the part of F up to t
 *     (forward conditional expectation A) and after t (backward, B); both
 *     follow recursions with the same weights as the alpha / beta sums;
 *   - Viterbi (Sec. 3.2): min-sum dynamic programming with backtrack.
 * The first state s_1 carries no prior weight: alpha_1(s) = exp(h_1(s)).
 *
 * Vector emission (Sec. 3.1, S = 2^{k+V}; Sec. 4.1, the V = 2 trellis): each
 * step emits V consecutive weights, the codeword c(s) is a V-vector stored at
 * c[s*V .. s*V+V-1], the step's energy is ||w_t - c(s)||^2 / 2 and F becomes
 * sum_t <g_t, c(s_t)>; every formula above holds per component.  A block of
 * L weights then has L/V steps.  V = 1 is the scalar case.
 */
#include "bcjr_oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

static int bad_args(int64_t B, int64_t L, const void *w, const void *c, int n,
                    int k, int V, double T) {
  if (B < 0 || L < 1 || !w || !c) return 1;
  if (V < 1 || V > 8 || L % V) return 1;
  if (k < 1 || n < k || n > 16) return 1;
  if (!(T > 0.0) || !isfinite(T)) return 1;
  return 0;
}

/* log(exp(a) + exp(b)), exact in the limits a or b = -inf */
static double log_add_exp(double a, double b) {
  if (a == -INFINITY) return b;
  if (b == -INFINITY) return a;
  double m = a > b ? a : b;
  return m + log1p(exp(-fabs(a - b)));
}

/* h_t(s) = -||w_t - c(s)||^2 / (2T) over the V components of step t */
static double field(const double *w, const double *c, int V, double T) {
  double e = 0.0;
  for (int a = 0; a < V; ++a) {
    double d = w[a] - c[a];
    e += d * d;
  }
  return -e / (2.0 * T);
}

/* <g_t, c(s)> */
static double dotv(const double *g, const double *c, int V) {
  double r = 0.0;
  for (int a = 0; a < V; ++a) r += g[a] * c[a];
  return r;
}

/* ------------------------------------------------------------------ */
/* one block: forward-backward, optional VJP                            */
/* ------------------------------------------------------------------ */

typedef struct {
  double *alpha; /* [L*S] */
  double *A;     /* [L*S] or NULL */
  double *acc;   /* [S] */
  double *num;   /* [S] */
  double *beta;  /* [S] current beta_t */
  double *betap; /* [S] beta_{t-1} being built */
  double *Bc;    /* [S] current B_t */
  double *Bp;    /* [S] B_{t-1} */
  double *p;     /* [S] */
} work_t;

static int work_alloc(work_t *wk, int64_t L, int64_t S, int want_vjp) {
  memset(wk, 0, sizeof(*wk));
  wk->alpha = (double *)malloc(sizeof(double) * (size_t)(L * S));
  wk->A = want_vjp ? (double *)malloc(sizeof(double) * (size_t)(L * S)) : NULL;
  wk->acc = (double *)malloc(sizeof(double) * (size_t)S);
  wk->num = (double *)malloc(sizeof(double) * (size_t)S);
  wk->beta = (double *)malloc(sizeof(double) * (size_t)S);
  wk->betap = (double *)malloc(sizeof(double) * (size_t)S);
  wk->Bc = (double *)malloc(sizeof(double) * (size_t)S);
  wk->Bp = (double *)malloc(sizeof(double) * (size_t)S);
  wk->p = (double *)malloc(sizeof(double) * (size_t)S);
  if (!wk->alpha || (want_vjp && !wk->A) || !wk->acc || !wk->num ||
      !wk->beta || !wk->betap || !wk->Bc || !wk->Bp || !wk->p)
    return -1;
  return 0;
}

static void work_free(work_t *wk) {
  free(wk->alpha);
  free(wk->A);
  free(wk->acc);
  free(wk->num);
  free(wk->beta);
  free(wk->betap);
  free(wk->Bc);
  free(wk->Bp);
  free(wk->p);
}

/* Forward sweep: log alpha_t(s) for all t (Eq. alpha and its recursion),
 * and, when g != NULL, A_t(s) = E[sum_{tau<=t} g_tau c(s_tau) | s_t = s,
 * w_1..w_t]: A_1(s) = g_1 c(s);
 * A_t(s) = g_t c(s) + sum_{s'->s} alpha_{t-1}(s') A_{t-1}(s') / sum_{s'->s} alpha_{t-1}(s'). */
static void forward_sweep(const double *w, int64_t L, const double *c, int n,
                          int k, int V, double T, const double *g, work_t *wk) {
  const int64_t S = (int64_t)1 << n, K = (int64_t)1 << k, mask = S - 1;
  double *alpha = wk->alpha, *A = wk->A, *acc = wk->acc, *num = wk->num;
  for (int64_t s = 0; s < S; ++s) {
    alpha[s] = field(w, c + s * V, V, T);
    if (g) A[s] = dotv(g, c + s * V, V);
  }
  for (int64_t t = 1; t < L; ++t) {
    const double *ap = alpha + (t - 1) * S;
    double *at = alpha + t * S;
    for (int64_t s = 0; s < S; ++s) acc[s] = -INFINITY;
    /* sum over s' with T_{s' -> s} = 1, in the log domain */
    for (int64_t sp = 0; sp < S; ++sp)
      for (int64_t b = 0; b < K; ++b) {
        int64_t d = ((sp << k) | b) & mask;
        acc[d] = log_add_exp(acc[d], ap[sp]);
      }
    for (int64_t s = 0; s < S; ++s) at[s] = field(w + t * V, c + s * V, V, T) + acc[s];
    if (g) {
      const double *Ap = A + (t - 1) * S;
      double *At = A + t * S;
      for (int64_t s = 0; s < S; ++s) num[s] = 0.0;
      for (int64_t sp = 0; sp < S; ++sp)
        for (int64_t b = 0; b < K; ++b) {
          int64_t d = ((sp << k) | b) & mask;
          num[d] += exp(ap[sp] - acc[d]) * Ap[sp];
        }
      for (int64_t s = 0; s < S; ++s) At[s] = dotv(g + t * V, c + s * V, V) + num[s];
    }
  }
}

static double lse_row(const double *x, int64_t S) {
  double m = -INFINITY;
  for (int64_t s = 0; s < S; ++s)
    if (x[s] > m) m = x[s];
  if (m == -INFINITY) return m;
  double sum = 0.0;
  for (int64_t s = 0; s < S; ++s) sum += exp(x[s] - m);
  return m + log(sum);
}

/* Backward step: from log beta_t (beta, 0-based index t) build log beta_{t-1}:
 * beta_{t-1}(s) = LSE_b [ h_t(next(s,b)) + beta_t(next(s,b)) ]  (recursion of
 * Eq. beta), and, when g != NULL, the backward conditional expectation
 * B_{t-1}(s) = E[sum_{tau>=t} g_tau c(s_tau) | s_{t-1} = s, w_t..w_L]. */
static void backward_step(const double *w, int64_t t, const double *c, int n,
                          int k, int V, double T, const double *g, work_t *wk) {
  const int64_t S = (int64_t)1 << n, K = (int64_t)1 << k, mask = S - 1;
  for (int64_t s = 0; s < S; ++s) {
    double acc = -INFINITY;
    for (int64_t b = 0; b < K; ++b) {
      int64_t d = ((s << k) | b) & mask;
      acc = log_add_exp(acc, field(w + t * V, c + d * V, V, T) + wk->beta[d]);
    }
    wk->betap[s] = acc;
    if (g) {
      double sum = 0.0;
      for (int64_t b = 0; b < K; ++b) {
        int64_t d = ((s << k) | b) & mask;
        double r = exp(field(w + t * V, c + d * V, V, T) + wk->beta[d] - acc);
        sum += r * (dotv(g + t * V, c + d * V, V) + wk->Bc[d]);
      }
      wk->Bp[s] = sum;
    }
  }
  double *tmp = wk->beta;
  wk->beta = wk->betap;
  wk->betap = tmp;
  tmp = wk->Bc;
  wk->Bc = wk->Bp;
  wk->Bp = tmp;
}

/* One block of L weights = N = L / V steps.  w_soft, dW: [L]; dc: [S*V]. */
static void block_run(const double *w, int64_t L, const double *c, int n,
                      int k, int V, double T, const double *g, double *w_soft,
                      double *logZ_out, double *dW, double *dc, work_t *wk) {
  const int64_t S = (int64_t)1 << n, N = L / V;
  forward_sweep(w, N, c, n, k, V, T, g, wk);
  const double *aL = wk->alpha + (N - 1) * S;
  const double logZ = lse_row(aL, S); /* Z = sum_s alpha_N(s), beta_N = 1 */
  if (logZ_out) *logZ_out = logZ;
  double EF = 0.0; /* E[F] = sum_s p_N(s) A_N(s) */
  if (g)
    for (int64_t s = 0; s < S; ++s) EF += exp(aL[s] - logZ) * wk->A[(N - 1) * S + s];
  for (int64_t s = 0; s < S; ++s) {
    wk->beta[s] = 0.0; /* log beta_N = 0 */
    wk->Bc[s] = 0.0;   /* B_N = 0 */
  }
  for (int64_t t = N - 1; t >= 0; --t) {
    const double *at = wk->alpha + t * S;
    for (int64_t s = 0; s < S; ++s) wk->p[s] = exp(at[s] + wk->beta[s] - logZ); /* Eq. marginal */
    for (int a = 0; a < V; ++a) {
      double ws = 0.0;
      for (int64_t s = 0; s < S; ++s) ws += c[s * V + a] * wk->p[s]; /* Eq. soft-codeword */
      if (w_soft) w_soft[t * V + a] = ws;
      if (g) {
        const double *At = wk->A + t * S;
        double cov = 0.0;
        for (int64_t s = 0; s < S; ++s) {
          double X = At[s] + wk->Bc[s] - EF; /* E[F | s_t = s] - E[F] */
          cov += wk->p[s] * (c[s * V + a] - ws) * X;
          if (dc)
            dc[s * V + a] += wk->p[s] * (g[t * V + a] + (w[t * V + a] - c[s * V + a]) * X / T);
        }
        if (dW) dW[t * V + a] = cov / T;
      }
    }
    if (t > 0) backward_step(w, t, c, n, k, V, T, g, wk);
  }
}

/* ------------------------------------------------------------------ */
/* threading over blocks                                                */
/* ------------------------------------------------------------------ */

typedef struct {
  const double *w, *c, *g;
  int64_t B, L;
  int n, k, V;
  double T;
  double *w_soft, *logZ, *dW;
  double *dc_part; /* [S] private to this thread, or NULL */
  int tid, nthreads;
  int status;
} job_t;

static void *job_main(void *arg) {
  job_t *j = (job_t *)arg;
  const int64_t S = (int64_t)1 << j->n;
  work_t wk;
  if (work_alloc(&wk, j->L / j->V, S, j->g != NULL) != 0) {
    work_free(&wk);
    j->status = -2;
    return NULL;
  }
  for (int64_t b = j->tid; b < j->B; b += j->nthreads) {
    block_run(j->w + b * j->L, j->L, j->c, j->n, j->k, j->V, j->T, j->g ? j->g + b * j->L : NULL,
              j->w_soft ? j->w_soft + b * j->L : NULL, j->logZ ? j->logZ + b : NULL,
              j->dW ? j->dW + b * j->L : NULL, j->dc_part, &wk);
  }
  work_free(&wk);
  j->status = 0;
  return NULL;
}

static int run_jobs(const double *w, int64_t B, int64_t L, const double *c,
                    int n, int k, int V, double T, const double *g, double *w_soft,
                    double *logZ, double *dW, double *dc, int nthreads) {
  const int64_t S = ((int64_t)1 << n) * V;  /* dCodebook entries */
  if (nthreads < 1) nthreads = 1;
  if ((int64_t)nthreads > B && B > 0) nthreads = (int)B;
  if (dc)
    for (int64_t s = 0; s < S; ++s) dc[s] = 0.0;
  if (B == 0) return 0;
  job_t *jobs = (job_t *)calloc((size_t)nthreads, sizeof(job_t));
  pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
  double *parts = dc ? (double *)calloc((size_t)(nthreads * S), sizeof(double)) : NULL;
  if (!jobs || !th || (dc && !parts)) {
    free(jobs);
    free(th);
    free(parts);
    return -2;
  }
  for (int i = 0; i < nthreads; ++i) {
    job_t *j = &jobs[i];
    j->w = w; j->c = c; j->g = g; j->B = B; j->L = L; j->n = n; j->k = k; j->V = V;
    j->T = T; j->w_soft = w_soft; j->logZ = logZ; j->dW = dW;
    j->dc_part = dc ? parts + (int64_t)i * S : NULL;
    j->tid = i; j->nthreads = nthreads; j->status = -3;
  }
  for (int i = 1; i < nthreads; ++i) pthread_create(&th[i], NULL, job_main, &jobs[i]);
  job_main(&jobs[0]);
  for (int i = 1; i < nthreads; ++i) pthread_join(th[i], NULL);
  int status = 0;
  for (int i = 0; i < nthreads; ++i)
    if (jobs[i].status != 0) status = jobs[i].status;
  if (dc)
    for (int i = 0; i < nthreads; ++i)
      for (int64_t s = 0; s < S; ++s) dc[s] += parts[(int64_t)i * S + s];
  free(jobs);
  free(th);
  free(parts);
  return status;
}

int oracle_soft_codeword_v(const double *w, int64_t B, int64_t L, const double *c,
                           int n, int k, int V, double T, double *w_soft, double *logZ,
                           int nthreads) {
  if (bad_args(B, L, w, c, n, k, V, T)) return -1;
  return run_jobs(w, B, L, c, n, k, V, T, NULL, w_soft, logZ, NULL, NULL, nthreads);
}

int oracle_soft_codeword(const double *w, int64_t B, int64_t L, const double *c,
                         int n, int k, double T, double *w_soft, double *logZ,
                         int nthreads) {
  return oracle_soft_codeword_v(w, B, L, c, n, k, 1, T, w_soft, logZ, nthreads);
}

int oracle_soft_codeword_vjp_v(const double *w, int64_t B, int64_t L,
                               const double *c, int n, int k, int V, double T,
                               const double *g, double *w_soft, double *logZ,
                               double *dW, double *dc, int nthreads) {
  if (bad_args(B, L, w, c, n, k, V, T) || !g) return -1;
  return run_jobs(w, B, L, c, n, k, V, T, g, w_soft, logZ, dW, dc, nthreads);
}

int oracle_soft_codeword_vjp(const double *w, int64_t B, int64_t L,
                             const double *c, int n, int k, double T,
                             const double *g, double *w_soft, double *logZ,
                             double *dW, double *dc, int nthreads) {
  return oracle_soft_codeword_vjp_v(w, B, L, c, n, k, 1, T, g, w_soft, logZ, dW, dc, nthreads);
}

int oracle_block_tables_v(const double *w, int64_t L, const double *c, int n,
                          int k, int V, double T, const double *g, double *alpha,
                          double *beta, double *A, double *Bt) {
  if (bad_args(1, L, w, c, n, k, V, T) || !alpha || !beta) return -1;
  if (g && (!A || !Bt)) return -1;
  const int64_t S = (int64_t)1 << n, N = L / V;
  work_t wk;
  if (work_alloc(&wk, N, S, g != NULL) != 0) {
    work_free(&wk);
    return -2;
  }
  forward_sweep(w, N, c, n, k, V, T, g, &wk);
  memcpy(alpha, wk.alpha, sizeof(double) * (size_t)(N * S));
  if (g) memcpy(A, wk.A, sizeof(double) * (size_t)(N * S));
  for (int64_t s = 0; s < S; ++s) {
    wk.beta[s] = 0.0;
    wk.Bc[s] = 0.0;
  }
  for (int64_t t = N - 1; t >= 0; --t) {
    memcpy(beta + t * S, wk.beta, sizeof(double) * (size_t)S);
    if (g) memcpy(Bt + t * S, wk.Bc, sizeof(double) * (size_t)S);
    if (t > 0) backward_step(w, t, c, n, k, V, T, g, &wk);
  }
  work_free(&wk);
  return 0;
}

int oracle_block_tables(const double *w, int64_t L, const double *c, int n,
                        int k, double T, const double *g, double *alpha,
                        double *beta, double *A, double *Bt) {
  return oracle_block_tables_v(w, L, c, n, k, 1, T, g, alpha, beta, A, Bt);
}

/* ------------------------------------------------------------------ */
/* Viterbi                                                              */
/* ------------------------------------------------------------------ */

typedef struct {
  const double *w, *c;
  int64_t B, L;
  int n, k, V;
  int32_t *states;
  double *cost;
  int tid, nthreads, status;
} vjob_t;

/* squared distortion of one step, ||w_t - c(s)||^2: each square rounded,
 * then added in component order (no fused ops; the file is compiled with
 * -ffp-contract=off).  For V = 1 it is the plain (w - c)^2. */
static double sqdist(const double *w, const double *c, int V) {
  double d = w[0] - c[0];
  double e = d * d;
  for (int a = 1; a < V; ++a) {
    double da = w[a] - c[a];
    e = e + da * da;
  }
  return e;
}

/* One block of L weights, N = L / V steps; states[N]. */
static void viterbi_block(const double *w, int64_t L, const double *c, int n,
                          int k, int V, int32_t *states, double *cost, double *m,
                          double *mn, double *best, int32_t *from) {
  const int64_t S = (int64_t)1 << n, K = (int64_t)1 << k, mask = S - 1;
  L /= V;
  for (int64_t s = 0; s < S; ++s) m[s] = sqdist(w, c + s * V, V);
  for (int64_t t = 1; t < L; ++t) {
    int32_t *ft = from + t * S;
    for (int64_t s = 0; s < S; ++s) {
      best[s] = INFINITY;
      ft[s] = -1;
    }
    /* predecessors visited in increasing state order; strict '<' keeps the
     * smallest predecessor among equal minima */
    for (int64_t sp = 0; sp < S; ++sp)
      for (int64_t b = 0; b < K; ++b) {
        int64_t d = ((sp << k) | b) & mask;
        if (ft[d] < 0 || m[sp] < best[d]) {
          best[d] = m[sp];
          ft[d] = (int32_t)sp;
        }
      }
    for (int64_t s = 0; s < S; ++s) mn[s] = sqdist(w + t * V, c + s * V, V) + best[s];
    double *tmp = m;
    m = mn;
    mn = tmp;
  }
  int64_t sb = 0;
  for (int64_t s = 1; s < S; ++s)
    if (m[s] < m[sb]) sb = s;
  if (cost) *cost = m[sb];
  states[L - 1] = (int32_t)sb;
  for (int64_t t = L - 1; t >= 1; --t) states[t - 1] = from[t * S + states[t]];
}

static void *vjob_main(void *arg) {
  vjob_t *j = (vjob_t *)arg;
  const int64_t S = (int64_t)1 << j->n;
  double *m = (double *)malloc(sizeof(double) * (size_t)S);
  double *mn = (double *)malloc(sizeof(double) * (size_t)S);
  double *best = (double *)malloc(sizeof(double) * (size_t)S);
  int32_t *from = (int32_t *)malloc(sizeof(int32_t) * (size_t)(j->L / j->V * S));
  if (!m || !mn || !best || !from) {
    j->status = -2;
  } else {
    for (int64_t b = j->tid; b < j->B; b += j->nthreads)
      viterbi_block(j->w + b * j->L, j->L, j->c, j->n, j->k, j->V, j->states + b * (j->L / j->V),
                    j->cost ? j->cost + b : NULL, m, mn, best, from);
    j->status = 0;
  }
  free(m);
  free(mn);
  free(best);
  free(from);
  return NULL;
}

int oracle_viterbi_v(const double *w, int64_t B, int64_t L, const double *c,
                     int n, int k, int V, int32_t *states, double *cost, int nthreads) {
  if (bad_args(B, L, w, c, n, k, V, 1.0) || !states) return -1;
  if (B == 0) return 0;
  if (nthreads < 1) nthreads = 1;
  if ((int64_t)nthreads > B) nthreads = (int)B;
  vjob_t *jobs = (vjob_t *)calloc((size_t)nthreads, sizeof(vjob_t));
  pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
  if (!jobs || !th) {
    free(jobs);
    free(th);
    return -2;
  }
  for (int i = 0; i < nthreads; ++i) {
    vjob_t *j = &jobs[i];
    j->w = w; j->c = c; j->B = B; j->L = L; j->n = n; j->k = k; j->V = V;
    j->states = states; j->cost = cost; j->tid = i; j->nthreads = nthreads;
    j->status = -3;
  }
  for (int i = 1; i < nthreads; ++i) pthread_create(&th[i], NULL, vjob_main, &jobs[i]);
  vjob_main(&jobs[0]);
  for (int i = 1; i < nthreads; ++i) pthread_join(th[i], NULL);
  int status = 0;
  for (int i = 0; i < nthreads; ++i)
    if (jobs[i].status != 0) status = jobs[i].status;
  free(jobs);
  free(th);
  return status;
}

int oracle_viterbi(const double *w, int64_t B, int64_t L, const double *c,
                   int n, int k, int32_t *states, double *cost, int nthreads) {
  return oracle_viterbi_v(w, B, L, c, n, k, 1, states, cost, nthreads);
}

/* ------------------------------------------------------------------ */
/* Min-sum max-marginals and the margin of the decoded codeword         */
/* ------------------------------------------------------------------ */

typedef struct {
  const double *w, *c;
  int64_t B, L;
  int n, k, V;
  const int32_t *states;
  double *gap;
  int tid, nthreads, status;
} gjob_t;

static int same_codeword(const double *a, const double *b, int V) {
  for (int q = 0; q < V; ++q)
    if (a[q] != b[q]) return 0;
  return 1;
}

/* One block, N = L / V steps.  mf[N*S]: the forward min-sum metric (the
 * smallest distortion of a path prefix ending in s at t, its own step
 * included); mb[S] / mbn[S]: the backward metric (the smallest distortion of
 * the steps after t for a path leaving s at t).  Their sum is the
 * max-marginal M_t(s). */
static void gap_block(const double *w, int64_t L, const double *c, int n, int k, int V,
                      const int32_t *st, double *gap, double *mf, double *mb, double *mbn) {
  const int64_t S = (int64_t)1 << n, K = (int64_t)1 << k, mask = S - 1;
  const int64_t N = L / V;
  for (int64_t s = 0; s < S; ++s) mf[s] = sqdist(w, c + s * V, V);
  for (int64_t t = 1; t < N; ++t) {
    double *cur = mf + t * S;
    const double *prev = mf + (t - 1) * S;
    for (int64_t s = 0; s < S; ++s) cur[s] = INFINITY;
    for (int64_t sp = 0; sp < S; ++sp)
      for (int64_t b = 0; b < K; ++b) {
        int64_t d = ((sp << k) | b) & mask;
        if (prev[sp] < cur[d]) cur[d] = prev[sp];
      }
    for (int64_t s = 0; s < S; ++s) cur[s] = sqdist(w + t * V, c + s * V, V) + cur[s];
  }
  for (int64_t s = 0; s < S; ++s) mb[s] = 0.0;
  for (int64_t t = N - 1; t >= 0; --t) {
    const double *f = mf + t * S;
    const int64_t sb = st[t];
    const double best = f[sb] + mb[sb];
    double alt = INFINITY;
    for (int64_t s = 0; s < S; ++s) {
      if (same_codeword(c + s * V, c + sb * V, V)) continue;
      double m = f[s] + mb[s];
      if (m < alt) alt = m;
    }
    gap[t] = 0.5 * (alt - best);
    if (t == 0) break;
    /* mb_{t-1}(s) = min_b [ d_t(next(s, b)) + mb_t(next(s, b)) ] */
    for (int64_t s = 0; s < S; ++s) {
      double m = INFINITY;
      for (int64_t b = 0; b < K; ++b) {
        int64_t d = ((s << k) | b) & mask;
        double v = sqdist(w + t * V, c + d * V, V) + mb[d];
        if (v < m) m = v;
      }
      mbn[s] = m;
    }
    double *tmp = mb;
    mb = mbn;
    mbn = tmp;
  }
}

static void *gjob_main(void *arg) {
  gjob_t *j = (gjob_t *)arg;
  const int64_t S = (int64_t)1 << j->n, N = j->L / j->V;
  double *mf = (double *)malloc(sizeof(double) * (size_t)(N * S));
  double *mb = (double *)malloc(sizeof(double) * (size_t)S);
  double *mbn = (double *)malloc(sizeof(double) * (size_t)S);
  if (!mf || !mb || !mbn) {
    j->status = -2;
  } else {
    for (int64_t b = j->tid; b < j->B; b += j->nthreads)
      gap_block(j->w + b * j->L, j->L, j->c, j->n, j->k, j->V, j->states + b * N, j->gap + b * N,
                mf, mb, mbn);
    j->status = 0;
  }
  free(mf);
  free(mb);
  free(mbn);
  return NULL;
}

int oracle_maxmarginal_gap_v(const double *w, int64_t B, int64_t L, const double *c, int n,
                             int k, int V, const int32_t *states, double *gap, int nthreads) {
  if (bad_args(B, L, w, c, n, k, V, 1.0) || !states || !gap) return -1;
  if (B == 0) return 0;
  const int64_t S = (int64_t)1 << n, N = L / V;
  for (int64_t i = 0; i < B * N; ++i)
    if (states[i] < 0 || states[i] >= S) return -1;
  if (nthreads < 1) nthreads = 1;
  if ((int64_t)nthreads > B) nthreads = (int)B;
  gjob_t *jobs = (gjob_t *)calloc((size_t)nthreads, sizeof(gjob_t));
  pthread_t *th = (pthread_t *)calloc((size_t)nthreads, sizeof(pthread_t));
  if (!jobs || !th) {
    free(jobs);
    free(th);
    return -2;
  }
  for (int i = 0; i < nthreads; ++i) {
    gjob_t *j = &jobs[i];
    j->w = w; j->c = c; j->B = B; j->L = L; j->n = n; j->k = k; j->V = V;
    j->states = states; j->gap = gap; j->tid = i; j->nthreads = nthreads;
    j->status = -3;
  }
  for (int i = 1; i < nthreads; ++i) pthread_create(&th[i], NULL, gjob_main, &jobs[i]);
  gjob_main(&jobs[0]);
  for (int i = 1; i < nthreads; ++i) pthread_join(th[i], NULL);
  int status = 0;
  for (int i = 0; i < nthreads; ++i)
    if (jobs[i].status != 0) status = jobs[i].status;
  free(jobs);
  free(th);
  return status;
}
