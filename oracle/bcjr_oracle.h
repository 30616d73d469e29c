/*
 * bcjr_oracle.h -- plain fp64 CPU oracle for the temperature-T BCJR soft
 * codeword over a bitshift trellis, its vector-Jacobian product, and the
 * Viterbi (T -> 0) decode.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
 * calls this library: only the tests, the package smoke check and the CPU
 * baseline leg of the benchmark do.  It shares no code, header, table or
 * helper with the HIP implementation.
 *
 * Model (paper, Sec. 3.1 "Trellis setup", Eq. boltzmann):
 *   states s in {0..S-1}, S = 2^n, K = 2^k inputs per step,
 *   transition  next(s, b) = ((s << k) | b) & (S - 1),
 *   a block is w[0..L-1]; a path is s_1..s_L (every state may start),
 *   energy E(path) = sum_t (w_t - c(s_t))^2 / 2,
 *   p_T(path) = exp(-E/T) / Z_T.
 * Indices here are 0-based: w[t], t = 0..L-1, corresponds to w_{t+1}.
 *
 * All inputs are double.  Callers holding fp32 data convert it exactly, so
 * the oracle and the GPU see the same numbers.  T > 0.
 * Every function returns 0 on success and a negative value on bad arguments.
 */
#ifndef BCJR_ORACLE_H
#define BCJR_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Soft codeword (Eq. soft-codeword via Eqs. alpha, beta, marginal,
 * softcode-final) and log Z_T (natural log) for B independent blocks.
 * w[B*L], c[S]; outputs w_soft[B*L], logZ[B].  nthreads <= 0 means one. */
int oracle_soft_codeword(const double *w, int64_t B, int64_t L,
                         const double *c, int n, int k, double T,
                         double *w_soft, double *logZ, int nthreads);

/* Forward outputs plus the VJP of  <g, w_soft>  with respect to w and c.
 * g[B*L] is the upstream gradient.  dW[B*L] (may be NULL); dc[S] (may be
 * NULL) is summed over the B blocks.  w_soft/logZ may be NULL. */
int oracle_soft_codeword_vjp(const double *w, int64_t B, int64_t L,
                             const double *c, int n, int k, double T,
                             const double *g, double *w_soft, double *logZ,
                             double *dW, double *dc, int nthreads);

/* Minimum-distortion path (paper Sec. 3.2): argmin over legal paths of
 * sum_t (w_t - c(s_t))^2.  Ties: the predecessor with the smallest state
 * index, then the smallest final state.  states[B*L] (s_1..s_L per block),
 * cost[B] (may be NULL). */
int oracle_viterbi(const double *w, int64_t B, int64_t L, const double *c,
                   int n, int k, int32_t *states, double *cost, int nthreads);

/* Full log-domain tables of ONE block for invariant checks:
 * alpha[L*S] = log alpha_t(s), beta[L*S] = log beta_t(s) (Eqs. alpha, beta);
 * optional A[L*S], Bt[L*S] = forward / backward conditional expectations of
 * the partial sums of g_t c(s_t) (used by the VJP), only if g != NULL. */
int oracle_block_tables(const double *w, int64_t L, const double *c, int n,
                        int k, double T, const double *g, double *alpha,
                        double *beta, double *A, double *Bt);

/* Vector emission (Sec. 3.1, S = 2^{k+V}; the V = 2 trellis of Sec. 4.1):
 * the same four functions with V weights per step.  L counts weights and
 * must be a multiple of V (L / V steps); the codebook is c[S*V] with the
 * V-vector of state s at c[s*V ..]; dc is [S*V]; states is [B*(L/V)];
 * alpha, beta, A, Bt are [(L/V)*S].  Energy ||w_t - c(s)||^2 / 2 per step;
 * the Viterbi step distortion adds the V rounded squares in component
 * order.  The functions above are these with V = 1. */
int oracle_soft_codeword_v(const double *w, int64_t B, int64_t L, const double *c,
                           int n, int k, int V, double T, double *w_soft,
                           double *logZ, int nthreads);
int oracle_soft_codeword_vjp_v(const double *w, int64_t B, int64_t L,
                               const double *c, int n, int k, int V, double T,
                               const double *g, double *w_soft, double *logZ,
                               double *dW, double *dc, int nthreads);
int oracle_viterbi_v(const double *w, int64_t B, int64_t L, const double *c,
                     int n, int k, int V, int32_t *states, double *cost,
                     int nthreads);
int oracle_block_tables_v(const double *w, int64_t L, const double *c, int n,
                          int k, int V, double T, const double *g, double *alpha,
                          double *beta, double *A, double *Bt);

/* Min-sum max-marginals (Sec. 3.2; the T -> 0 limit of Sec. 3.3).  For a
 * step t and state s, M_t(s) = min over legal paths with s_t = s of
 * sum_tau ||w_tau - c(s_tau)||^2 (each step's distortion as in
 * oracle_viterbi).  Given a decoded path states[B*(L/V)] (oracle_viterbi's
 * output), gap[B*(L/V)] receives per step
 *     ( min_{s : c(s) != c(states_t)} M_t(s)  -  M_t(states_t) ) / 2,
 * the energy (Eq. boltzmann, E = distortion / 2) by which the best path
 * emitting another codeword at step t loses; +inf when every state emits
 * the same codeword.  Returns -1 for a state index outside [0, S). */
int oracle_maxmarginal_gap_v(const double *w, int64_t B, int64_t L, const double *c,
                             int n, int k, int V, const int32_t *states, double *gap,
                             int nthreads);

#ifdef __cplusplus
}
#endif

#endif
