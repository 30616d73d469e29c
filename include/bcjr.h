/*
 * bcjr.h -- C ABI of the MI355X (gfx950) BCJR soft-codeword library.
 *
 * What is computed (paper Sec. 3, "Method"):
 *   A weight block w[0..L-1] is encoded by a path s_1..s_L through a bitshift
 *   trellis with S = 2^state_bits states and K = 2^k branches per step:
 *       next(s, b) = ((s << k) | b) & (S - 1)            (Sec. 3.1)
 *   Every state may start a path (no prior weight on s_1).  At temperature T
 *   the paths follow the Boltzmann distribution
 *       p_T(path) ~ exp(-(1/T) sum_t (w_t - c(s_t))^2 / 2)   (Eq. boltzmann)
 *   and the soft codeword is the per-step expectation of the emitted codeword
 *       w_soft_t = sum_s c(s) p_T(s_t = s | w)              (Eq. soft-codeword)
 *   computed by the log-domain forward-backward recursions (Sec. 3.4,
 *   Eqs. alpha, beta, marginal, softcode-final).  logZ is the natural log of
 *   the partition function Z_T of Eq. boltzmann.
 *   The VJP (Sec. 3.5) of  <g, w_soft>  is returned for an upstream gradient
 *   g: dW = d<g, w_soft>/dw per block and dCodebook = d<g, w_soft>/dc summed
 *   over the call's blocks.  T is a constant of the call (no dT).
 *   viterbi_decode returns the minimum-distortion path (Sec. 3.2), the
 *   T -> 0 limit of the soft codeword (Sec. 3.3).  bcjr_ste_vjp is the
 *   backward pass of the BCJR-STE variant, whose forward pass is that path.
 *
 * Conventions for every entry point:
 *   - w, grad_w_soft, w_soft, dW, w_hard are row-major [B, L] float32; block
 *     b occupies elements [b*L, (b+1)*L).  codebook and dCodebook are [S].
 *     logZ is [B].  states is [B, L] int32 holding s_1..s_L of each block.
 *   - All array pointers are DEVICE pointers owned by the caller, 4-byte
 *     aligned (16-byte for codebook), contiguous.  Inputs are never written;
 *     requested outputs are fully overwritten.  Optional outputs may be NULL.
 *   - workspace is caller-owned device memory.  bcjr_workspace_bytes() gives
 *     the size for full-speed operation; any smaller size that holds at least
 *     one block slot is accepted and runs with fewer blocks in flight.  The
 *     library allocates nothing.  A workspace must not be shared by calls
 *     that may run concurrently.
 *   - Calls are asynchronous on `stream`; the returned status covers argument
 *     validation and launch errors only.  No exception crosses the ABI.
 *   - Shapes: every 1 <= k <= state_bits <= 16.  The fp32 super-group
 *     kernels (double-float log vectors for the VJP below T = 0.04) take
 *     1 <= k <= 3 with 2k <= state_bits <= min(16, 2k + 12) and, for k = 3,
 *     state_bits <= 14 (k = 1: 2..14, k = 2: 4..16, k = 3: 6..14), with L
 *     small enough that one workgroup's histories stay below 2 GiB: the
 *     soft codeword and Viterbi take L <= 16383 at state_bits = 16, k = 2
 *     (at least 16383 for every such shape), the VJP L <= 10922 (at least
 *     10922).  Every other shape -- state_bits < 2k down to the fully
 *     connected state_bits = k, k >= 4, k = 1 at 15 and 16 state bits, k = 3
 *     above 14 -- runs fp64 kernels at any temperature, with L <= 2^30.
 *     Longer L returns BCJR_ERR_UNSUPPORTED and a workspace size of 0.
 *   - B == 0 is a no-op returning BCJR_OK (dCodebook, if given, is zeroed).
 *   - Non-finite w or codebook values give non-finite outputs; they are not
 *     checked.
 *   - At state_bits = 16, k = 2, T <= 0.015 and L <= 2048 the VJP (and the
 *     fused call) sums over the states within 30 nats of each block's best
 *     path only: every path through a dropped state weighs at most e^-30 of
 *     the best one, below fp32 resolution.  A block with more such
 *     state-steps than the workspace slot holds (1024 per step on average) is
 *     computed by the full double-float recursion instead.  dCodebook is then
 *     accumulated with fp64 atomic adds, so its last fp32 bit may differ
 *     between runs.
 */
#ifndef BCJR_H
#define BCJR_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  BCJR_OK = 0,
  BCJR_ERR_INVALID_ARG = -1,  /* bad size, k, state_bits, T, or NULL pointer */
  BCJR_ERR_UNSUPPORTED = -2,  /* valid arguments outside the supported shapes */
  BCJR_ERR_WORKSPACE = -3,    /* workspace NULL or smaller than one block slot */
  BCJR_ERR_HIP = -4           /* a HIP call or kernel launch failed */
} bcjr_status;

/* Size of the static scratch array of bcjr_soft_codeword_fwd_vjp_noalloc. */
#define BCJR_NOALLOC_SCRATCH_BYTES ((size_t)256 << 20)

enum {
  BCJR_OP_FWD = 0,      /* bcjr_soft_codeword */
  BCJR_OP_VJP = 1,      /* bcjr_soft_codeword_vjp */
  BCJR_OP_FWD_VJP = 2,  /* bcjr_soft_codeword_fwd_vjp */
  BCJR_OP_VITERBI = 3   /* viterbi_decode */
};

/* Workspace bytes for full-speed operation of `op` on B blocks of length L.
 * Pure host arithmetic.  Returns 0 for invalid or unsupported arguments. */
size_t bcjr_workspace_bytes(int64_t B, int64_t L, int state_bits, int k, int op);

/* Soft codeword (Eq. soft-codeword) and natural-log partition function.
 * Inputs: w[B*L], codebook[S], temperature T > 0 (finite).
 * Outputs: w_soft[B*L] (required), logZ[B] (may be NULL). */
int bcjr_soft_codeword(const float *w, int64_t B, int64_t L, const float *codebook,
                       int state_bits, int k, float T, float *w_soft, float *logZ,
                       void *workspace, size_t ws_bytes, hipStream_t stream);

/* VJP of <grad_w_soft, w_soft> with respect to w and the codebook
 * (Sec. 3.5; the covariance form d w_soft_t / d w_tau = Cov(c(s_t), c(s_tau)) / T
 * follows from Eq. boltzmann).  dW[B*L] and dCodebook[S] may each be NULL;
 * dCodebook is the sum over the B blocks of this call. */
int bcjr_soft_codeword_vjp(const float *w, int64_t B, int64_t L, const float *codebook,
                           int state_bits, int k, float T, const float *grad_w_soft,
                           float *dW, float *dCodebook, void *workspace, size_t ws_bytes,
                           hipStream_t stream);

/* Forward outputs and the VJP in one pass over the data (the upstream
 * gradient is known up front).  Any of w_soft, logZ, dW, dCodebook may be
 * NULL. */
int bcjr_soft_codeword_fwd_vjp(const float *w, int64_t B, int64_t L, const float *codebook,
                               int state_bits, int k, float T, const float *grad_w_soft,
                               float *w_soft, float *logZ, float *dW, float *dCodebook,
                               void *workspace, size_t ws_bytes, hipStream_t stream);

/* bcjr_soft_codeword_fwd_vjp without a workspace argument, for callers that
 * cannot allocate device memory (code under HIP graph capture, serving loops
 * and harnesses that forbid hipMalloc).  Same arguments, outputs and results
 * as bcjr_soft_codeword_fwd_vjp; the workspace is a static device array of
 * BCJR_NOALLOC_SCRATCH_BYTES (256 MiB) per GPU, allocated with the
 * library's code object and held until the process ends.  The call itself
 * allocates nothing.  It runs as many blocks side by side as fit in that
 * array (fewer than with a full-size workspace at large S; the results do
 * not depend on the count) and returns BCJR_ERR_WORKSPACE when even one
 * block slot does not fit: at state_bits 16, k 2 one slot takes about
 * 64 MiB at L = 256 with dCodebook, 32 MiB without (below T = 0.04, 73 and
 * 37 MiB, plus 8 B x B x L for the reference decode).  Every call on a GPU
 * uses that GPU's one array:
 * calls that may overlap on the same GPU (two streams, two threads) race
 * and must be serialised by the caller.  What the kernels need zeroed is
 * cleared by kernels in the call (no memset), so the call can be captured. */
int bcjr_soft_codeword_fwd_vjp_noalloc(const float *w, int64_t B, int64_t L,
                                       const float *codebook, int state_bits, int k, float T,
                                       const float *grad_w_soft, float *w_soft, float *logZ,
                                       float *dW, float *dCodebook, hipStream_t stream);

/* Backward pass of BCJR-STE (Sec. 3.5 and Sec. "BCJR-STE variant"): the
 * variant's forward output is the hard Viterbi codeword w_hard (viterbi_decode)
 * and its backward pass is the VJP of the soft codeword at temperature T, so
 * dW and dCodebook are those of bcjr_soft_codeword_vjp for the same w,
 * codebook, T and grad_w_soft.  w_hard[B*L] (required) is the forward output;
 * below T = 0.04 the VJP centres its backward tangent on it rather than
 * decoding the path again, so this call skips the Viterbi pass that
 * bcjr_soft_codeword_vjp runs there.  Any finite w_hard gives the same
 * result up to rounding; the accuracy stated for the VJP holds when it is
 * viterbi_decode's output for the same w and codebook.  Workspace: as for
 * BCJR_OP_VJP.  dW and dCodebook may each be NULL. */
int bcjr_ste_vjp(const float *w, int64_t B, int64_t L, const float *codebook, int state_bits,
                 int k, float T, const float *w_hard, const float *grad_w_soft, float *dW,
                 float *dCodebook, void *workspace, size_t ws_bytes, hipStream_t stream);

/* Minimum-distortion path, sum_t (w_t - c(s_t))^2 evaluated in fp64 with the
 * product and the sum rounded separately (Sec. 3.2).  Ties go to the
 * predecessor with the smallest state index, then to the smallest final
 * state.  states[B*L] (required) holds s_1..s_L; w_hard[B*L] = codebook[states]
 * (may be NULL). */
int viterbi_decode(const float *w, int64_t B, int64_t L, const float *codebook,
                   int state_bits, int k, int32_t *states, float *w_hard, void *workspace,
                   size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------
 * Vector emission (Sec. 3.1: S = 2^{k+V} with V weights per step; Sec. 4.1
 * and Sec. 4.4 use V = 2 with 4 bits per step, i.e. 16 predecessors per
 * state and 128 steps per 256-weight block).  Each step emits V consecutive
 * weights of the block and each state a V-vector codeword:
 *     h_t(s) = -||w_t - c(s)||^2 / (2T),   w_t = w[t*V .. t*V + V-1],
 * and k here is the number of bits shifted per step.  L counts weights and
 * must be a multiple of V (L / V steps).  codebook and dCodebook are
 * [S*V], the V-vector of state s at [s*V ..]; w_soft, dW, w_hard are
 * [B*L]; states is [B*(L/V)].  The Viterbi step distortion adds the V
 * rounded squares in component order.
 *
 * V = 1 calls the scalar entry points above with the same arguments.
 * V = 2 supports k = 4 and 8 <= state_bits <= 16 (at state_bits 16: L/2
 * steps up to 131071 for the soft codeword and Viterbi, 32767 for the VJP);
 * other shapes return BCJR_ERR_UNSUPPORTED.  As for the scalar trellis the
 * VJP switches below T = 0.04 to double-float log vectors, after a Viterbi
 * decode whose codewords centre the backward tangent.  Workspace: as
 * reported by bcjr_vec_workspace_bytes for the same op codes.  All other
 * conventions are those of the scalar entry points. */
size_t bcjr_vec_workspace_bytes(int64_t B, int64_t L, int state_bits, int k, int V, int op);

int bcjr_vec_soft_codeword(const float *w, int64_t B, int64_t L, const float *codebook,
                           int state_bits, int k, int V, float T, float *w_soft, float *logZ,
                           void *workspace, size_t ws_bytes, hipStream_t stream);

int bcjr_vec_soft_codeword_vjp(const float *w, int64_t B, int64_t L, const float *codebook,
                               int state_bits, int k, int V, float T, const float *grad_w_soft,
                               float *dW, float *dCodebook, void *workspace, size_t ws_bytes,
                               hipStream_t stream);

int bcjr_vec_soft_codeword_fwd_vjp(const float *w, int64_t B, int64_t L, const float *codebook,
                                   int state_bits, int k, int V, float T, const float *grad_w_soft,
                                   float *w_soft, float *logZ, float *dW, float *dCodebook,
                                   void *workspace, size_t ws_bytes, hipStream_t stream);

int bcjr_vec_viterbi_decode(const float *w, int64_t B, int64_t L, const float *codebook,
                            int state_bits, int k, int V, int32_t *states, float *w_hard,
                            void *workspace, size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------
 * Hessian-weighted rounding (the PTQ reference of the paper's oracle-bound
 * appendix: the loss L_HW = 1/2 tr((W - W_hat) H (W - W_hat)^T) of Eq. LHW,
 * minimised BlockLDLQ-style as in Eq. WPTQ).  All arithmetic is fp64 on the
 * device except the targets handed to the decode (fp32).
 *
 * Block LDL: with H' = H + damp * mean(diag H) * I (H symmetric positive
 * definite, [d, d] fp32 row-major), H' = M D M^T where M is unit block-upper-
 * triangular and D block-diagonal, blocks of `block` indices: from the upper
 * Cholesky factor H' = R R^T (the lower factor of the index-reversed matrix),
 * M = R blockdiag(R_kk)^{-1}, D = blockdiag(R_kk R_kk^T).  M and D are
 * [d, d] fp64 row-major outputs (D may be NULL).  d must be a multiple of
 * block, d <= 2^20, damp >= 0.  A matrix that is not positive definite after
 * damping gives NaN entries (not reported by the status).  Workspace:
 * bcjr_block_ldl_workspace_bytes(d, block) bytes (0 for invalid sizes). */
size_t bcjr_block_ldl_workspace_bytes(int64_t d, int64_t block);
int bcjr_block_ldl(const float *H, int64_t d, int64_t block, double damp, double *M, double *D,
                   void *workspace, size_t ws_bytes, hipStream_t stream);

/* BlockLDLQ rounding of W [rows, cols] (fp32 row-major) to trellis
 * codewords: the column blocks k = 0, 1, ... of `block` columns are decoded
 * in order, block k as the minimum-distortion path (viterbi_decode, or
 * bcjr_vec_viterbi_decode for V > 1) of its target
 *     t_k = W[:, k] + sum_{j < k} (W - W_hat)[:, j] M_jk
 * (fp64 sums rounded to fp32), M from bcjr_block_ldl of H [cols, cols] with
 * damp.  Outputs: W_hat [rows, cols] fp32; states [cols / block, rows,
 * block / V] int32; targets [cols / block, rows, block] fp32 or NULL.  The
 * (state_bits, k, V) shapes are those of the decode; cols must be a multiple
 * of block and block of V.  Workspace: bcjr_ldlq_workspace_bytes(rows, cols,
 * block, state_bits, k, V) bytes (0 for invalid or unsupported shapes). */
size_t bcjr_ldlq_workspace_bytes(int64_t rows, int64_t cols, int64_t block, int state_bits, int k,
                                 int V);
int bcjr_ldlq_viterbi(const float *W, int64_t rows, int64_t cols, const float *codebook,
                      int state_bits, int k, int V, const float *H, int64_t block, double damp,
                      float *W_hat, int32_t *states, float *targets, void *workspace,
                      size_t ws_bytes, hipStream_t stream);

/* ---------------------------------------------------------------------
 * Quantisation-aware training helpers.
 *
 * Computed Gaussian codebook (Sec. 3.1: c(s) = Phi^{-1}((s + 1/2) / S) under an
 * incoherent permutation of the states).  Writes codebook[S*V], component a
 * of state s at [s*V + a]:
 *     codebook[s*V + a] = Phi^{-1}((pi_a(s) + 1/2) / S)   rounded to fp32,
 * where pi_a is a bijection of the state_bits-bit integers: with h =
 * ceil(state_bits / 2) and arithmetic mod 2^state_bits,
 *     x = s * A1_a + B_a;  x ^= x >> h;  x = x * A2_a;  x ^= x >> h,
 * and (A1_a | 1, B_a, A2_a | 1) for a = 0, 1, ... are consecutive draws of
 * SplitMix64 started from `seed`.  Each component is therefore an exact
 * permutation of the S Gaussian quantiles.  1 <= state_bits <= 24,
 * 1 <= V <= 8; codebook is a device pointer (4-byte aligned) owned by the
 * caller.  Asynchronous on stream. */
int bcjr_gaussian_codebook(float *codebook, int state_bits, int V, uint64_t seed,
                           hipStream_t stream);

/* One Adam step (Kingma & Ba) of the annealing loop (Sec. 3.6 and the
 * BCJR-QAT algorithm), elementwise over count values, in place on param, m
 * and v (device pointers, caller-owned; m and v start at zero):
 *     g = clamp(grad, -grad_clip, grad_clip)   (no clipping when grad_clip == 0)
 *     m = beta1 m + (1 - beta1) g,   v = beta2 v + (1 - beta2) g^2
 *     param -= lr * (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
 * step >= 1 counts the calls.  The clip is the max-norm bound g_max of the
 * drift budget. */
int qat_adam_step(float *param, const float *grad, float *m, float *v, int64_t count, float lr,
                  float beta1, float beta2, float eps, int64_t step, float grad_clip,
                  hipStream_t stream);

/* Plain gradient step with the same clipping: param -= lr * clamp(grad). */
int qat_sgd_step(float *param, const float *grad, int64_t count, float lr, float grad_clip,
                 hipStream_t stream);

/* Static description of a status code; never NULL. */
const char *bcjr_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* BCJR_H */
