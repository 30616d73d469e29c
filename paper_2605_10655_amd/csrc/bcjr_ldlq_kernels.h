// bcjr_ldlq_kernels.h -- Hessian-weighted trellis rounding (the PTQ
// reference of the paper's oracle-bound appendix: the loss of Eq. LHW,
// minimised BlockLDLQ-style as in Eq. WPTQ).
//
// Block LDL of the damped Hessian H' = H + damp * mean(diag H) * I:
//   H' = R R^T with R upper triangular, obtained as the lower Cholesky factor
//   C of the index-reversed matrix (R(i, j) = C(d-1-i, d-1-j)); then with
//   blocks of b columns, M = R blockdiag(R_kk)^{-1} (unit block-upper-
//   triangular) and D = blockdiag(R_kk R_kk^T), so that H' = M D M^T.
// Rounding, column block k in order: target
//   t_k = w_k + sum_{j < k} (w_j - w_hat_j) M_jk,
// then the exact minimum-distortion trellis path of t_k (the library's
// Viterbi kernels) gives w_hat_k.
//
// Everything is fp64 except the targets handed to the decode (fp32, the
// decode's input type).  The Cholesky is right-looking over panels of 32
// columns: the diagonal block is factored by one workgroup in LDS, the rows
// below by a triangular solve (one thread per row, the factored block in
// LDS), the trailing lower triangle by a tiled rank-32 update.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bcjr {
namespace ldl {

constexpr int kPanel = 32;

// out[0] = mean of diag(H)
__global__ void __launch_bounds__(256) diag_mean_kernel(const float* H, int64_t d, double* out) {
  __shared__ double red[4];
  double s = 0.0;
  for (int64_t i = threadIdx.x; i < d; i += 256) s += (double)H[i * d + i];
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) out[0] = (((red[0] + red[1]) + red[2]) + red[3]) / (double)d;
}

// A = the lower triangle of the index-reversed damped Hessian, zero above
__global__ void flip_damp_kernel(const float* H, int64_t d, double damp, const double* mean,
                                 double* A) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d * d) return;
  const int64_t i = e / d, j = e % d;
  double v = 0.0;
  if (j <= i) {
    v = (double)H[(d - 1 - i) * d + (d - 1 - j)];
    if (i == j) v += damp * mean[0];
  }
  A[e] = v;
}

// Factor the w x w diagonal block at (p, p) in place (lower Cholesky).  A
// non-positive pivot gives NaN, which then spreads to everything after it.
__global__ void __launch_bounds__(256) chol_diag_kernel(double* A, int64_t d, int64_t p, int w) {
  __shared__ double T[kPanel][kPanel + 1];
  const int tid = threadIdx.x;
  for (int e = tid; e < w * w; e += 256) T[e / w][e % w] = A[(p + e / w) * d + p + e % w];
  __syncthreads();
  for (int j = 0; j < w; ++j) {
    if (tid == 0) T[j][j] = sqrt(T[j][j]);
    __syncthreads();
    for (int r = j + 1 + tid; r < w; r += 256) T[r][j] /= T[j][j];
    __syncthreads();
    for (int e = tid; e < w * w; e += 256) {
      const int r = e / w, c = e % w;
      if (c > j && c <= r) T[r][c] -= T[r][j] * T[c][j];
    }
    __syncthreads();
  }
  for (int e = tid; e < w * w; e += 256) {
    const int r = e / w, c = e % w;
    if (c <= r) A[(p + r) * d + p + c] = T[r][c];
  }
}

// Rows i >= p + w: A[i, p:p+w] <- A[i, p:p+w] L_pp^{-T} (forward substitution)
__global__ void __launch_bounds__(256) chol_trsm_kernel(double* A, int64_t d, int64_t p, int w) {
  __shared__ double T[kPanel][kPanel + 1];
  for (int e = threadIdx.x; e < w * w; e += 256) T[e / w][e % w] = A[(p + e / w) * d + p + e % w];
  __syncthreads();
  const int64_t i = p + w + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= d) return;
  double x[kPanel];
#pragma unroll
  for (int j = 0; j < kPanel; ++j) {
    if (j < w) {
      double a = A[i * d + p + j];
#pragma unroll
      for (int q = 0; q < kPanel; ++q)
        if (q < j) a -= x[q] * T[j][q];
      x[j] = a / T[j][j];
    }
  }
#pragma unroll
  for (int j = 0; j < kPanel; ++j)
    if (j < w) A[i * d + p + j] = x[j];
}

// Trailing update A[i][j] -= sum_{q < w} A[i][p+q] A[j][p+q] for
// p + w <= j <= i < d, over 32 x 32 tiles of the lower triangle (the
// workgroup index enumerates the tile pairs ti >= tj).
__global__ void __launch_bounds__(256) chol_update_kernel(double* A, int64_t d, int64_t p, int w) {
  __shared__ double Pi[kPanel][kPanel + 1], Pj[kPanel][kPanel + 1];
  const int64_t idx = blockIdx.x;
  int64_t ti = (int64_t)((sqrt(8.0 * (double)idx + 1.0) - 1.0) * 0.5);
  while (ti * (ti + 1) / 2 > idx) --ti;
  while ((ti + 1) * (ti + 2) / 2 <= idx) ++ti;
  const int64_t tj = idx - ti * (ti + 1) / 2;
  const int64_t r0 = p + w + ti * kPanel, c0 = p + w + tj * kPanel;
  for (int e = threadIdx.x; e < kPanel * kPanel; e += 256) {
    const int r = e / kPanel, q = e % kPanel;
    Pi[r][q] = (r0 + r < d && q < w) ? A[(r0 + r) * d + p + q] : 0.0;
    Pj[r][q] = (c0 + r < d && q < w) ? A[(c0 + r) * d + p + q] : 0.0;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < kPanel * kPanel; e += 256) {
    const int r = e / kPanel, c = e % kPanel;
    const int64_t i = r0 + r, j = c0 + c;
    if (i < d && j <= i) {
      double s = 0.0;
#pragma unroll
      for (int q = 0; q < kPanel; ++q) s = fma(Pi[r][q], Pj[c][q], s);
      A[i * d + j] -= s;
    }
  }
}

// R(i, j) = C(d-1-i, d-1-j), C the lower factor held in A
__device__ __forceinline__ double rget(const double* C, int64_t d, int64_t i, int64_t j) {
  return C[(d - 1 - i) * d + (d - 1 - j)];
}

// Rinv[k] = (R_kk)^{-1}, upper triangular, b x b per diagonal block; one
// workgroup per block, one thread per column (back substitution)
__global__ void __launch_bounds__(256) rinv_kernel(const double* C, int64_t d, int64_t b, double* Rinv) {
  const int64_t k = blockIdx.x, kb = k * b;
  double* X = Rinv + k * b * b;
  for (int64_t c = threadIdx.x; c < b; c += 256) {
    for (int64_t i = b - 1; i > c; --i) X[i * b + c] = 0.0;
    for (int64_t i = c; i >= 0; --i) {
      double s = i == c ? 1.0 : 0.0;
      for (int64_t q = i + 1; q <= c; ++q) s -= rget(C, d, kb + i, kb + q) * X[q * b + c];
      X[i * b + c] = s / rget(C, d, kb + i, kb + i);
    }
  }
}

// M[i][kb + c] = sum_q R(i, kb + q) Rinv[k][q][c]; zero below block row k
// (R is upper triangular, so only q >= i - kb contribute)
__global__ void m_kernel(const double* C, int64_t d, int64_t b, const double* Rinv, double* M) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d * d) return;
  const int64_t i = e / d, j = e % d;
  const int64_t k = j / b, kb = k * b, c = j - kb;
  double s = 0.0;
  if (i < kb + b) {
    const double* X = Rinv + k * b * b;
    for (int64_t q = (i > kb ? i - kb : 0); q < b; ++q) s = fma(rget(C, d, i, kb + q), X[q * b + c], s);
  }
  M[e] = s;
}

// D = blockdiag(R_kk R_kk^T)
__global__ void dblk_kernel(const double* C, int64_t d, int64_t b, double* D) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= d * d) return;
  const int64_t i = e / d, j = e % d;
  double s = 0.0;
  if (i / b == j / b) {
    const int64_t kb = (i / b) * b;
    for (int64_t q = (i > j ? i : j); q < kb + b; ++q) s = fma(rget(C, d, i, q), rget(C, d, j, q), s);
  }
  D[e] = s;
}

// target[r][c] = W[r][kb + c] + sum_{q < kb} (W[r][q] - W_hat[r][q]) M[q][kb + c]
// for r < rows, c < b: 32 x 32 output tiles, fp64 accumulation over
// 32-wide chunks of q staged in LDS; the sum is rounded to fp32 once.
__global__ void __launch_bounds__(256) feedback_kernel(const float* W, const float* What, const double* M,
                                                       int64_t rows, int64_t cols, int64_t b, int64_t kb,
                                                       float* target) {
  __shared__ double E[kPanel][kPanel + 1], Mt[kPanel][kPanel + 1];
  const int64_t r0 = (int64_t)blockIdx.x * kPanel, c0 = (int64_t)blockIdx.y * kPanel;
  const int tx = threadIdx.x % kPanel, ty = threadIdx.x / kPanel;  // ty < 8
  double acc[4] = {0.0, 0.0, 0.0, 0.0};
  for (int64_t q0 = 0; q0 < kb; q0 += kPanel) {
    for (int e = threadIdx.x; e < kPanel * kPanel; e += 256) {
      const int r = e / kPanel, q = e % kPanel;
      const int64_t gr = r0 + r, gq = q0 + q;
      E[r][q] = (gr < rows && gq < kb) ? (double)W[gr * cols + gq] - (double)What[gr * cols + gq] : 0.0;
      const int64_t gc = c0 + q;  // here q indexes the column of the M tile
      Mt[r][q] = (q0 + r < kb && gc < b) ? M[(q0 + r) * cols + kb + gc] : 0.0;
    }
    __syncthreads();
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const int r = ty + 8 * m;
#pragma unroll
      for (int q = 0; q < kPanel; ++q) acc[m] = fma(E[r][q], Mt[q][tx], acc[m]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    const int64_t gr = r0 + ty + 8 * m, gc = c0 + tx;
    if (gr < rows && gc < b) target[gr * b + gc] = (float)((double)W[gr * cols + kb + gc] + acc[m]);
  }
}

// W_hat[r][kb + c] = wh[r][c]
__global__ void scatter_kernel(const float* wh, int64_t rows, int64_t cols, int64_t b, int64_t kb, float* What) {
  const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= rows * b) return;
  What[(e / b) * cols + kb + e % b] = wh[e];
}

}  // namespace ldl
}  // namespace bcjr
