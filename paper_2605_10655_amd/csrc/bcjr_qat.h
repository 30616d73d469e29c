// bcjr_qat.h -- kernels around the soft codeword for quantisation-aware
// training: the computed Gaussian codebook (paper Sec. 3.1) and the
// optimiser updates of the annealing loop (Sec. 3.6, Algorithm "BCJR-QAT").
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bcjr {
namespace {

// The permutation of one codeword component: a bijection of the n-bit
// integers built from steps that are each bijective on n bits (an affine map
// with an odd multiplier, an xor with the value shifted right by h >= 1, a
// multiplication by an odd constant, the xor shift again).
struct PermConst {
  uint64_t a1, b, a2;
};

__host__ __device__ __forceinline__ uint32_t perm_n(uint32_t s, int n, PermConst p) {
  const uint64_t mask = (n >= 64) ? ~0ull : ((1ull << n) - 1);
  const int h = (n + 1) / 2;
  uint64_t x = ((uint64_t)s * p.a1 + p.b) & mask;
  x ^= x >> h;
  x = (x * p.a2) & mask;
  x ^= x >> h;
  return (uint32_t)x;
}

// Inverse of the standard normal CDF in fp64: the rational starting value of
// Abramowitz & Stegun 26.2.23 (absolute error below 4.5e-4), then three
// Halley steps on Phi(x) - p with Phi(x) = erfc(-x / sqrt 2) / 2 (cubic
// convergence: the error after the last step is at the rounding level of
// erfc).  Symmetric: the lower half is computed and the sign flipped.
__device__ __forceinline__ double norm_inv(double p) {
  const bool upper = p > 0.5;
  const double q = upper ? 1.0 - p : p;
  const double t = sqrt(-2.0 * log(q));
  double x = -(t - (2.515517 + t * (0.802853 + t * 0.010328)) /
                   (1.0 + t * (1.432788 + t * (0.189269 + t * 0.001308))));
  const double rt2 = 1.4142135623730950488, rt2pi = 2.5066282746310005024;
#pragma unroll 1
  for (int it = 0; it < 3; ++it) {
    const double e = 0.5 * erfc(-x / rt2) - q;
    const double u = e * rt2pi * exp(0.5 * x * x);
    x = x - u / (1.0 + 0.5 * x * u);
  }
  return upper ? -x : x;
}

constexpr int kMaxV = 8;
struct PermSet {
  PermConst p[kMaxV];
};

// SplitMix64 (Steele, Lea and Flood, 2014): the stream that draws the
// permutation constants from the seed, three per component (a1 and a2 made
// odd).
__host__ __forceinline__ uint64_t splitmix64(uint64_t& state) {
  state += 0x9E3779B97F4A7C15ull;
  uint64_t z = state;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

__host__ __forceinline__ PermSet perm_set(uint64_t seed, int V) {
  PermSet ps = {};
  uint64_t st = seed;
  for (int a = 0; a < V && a < kMaxV; ++a) {
    ps.p[a].a1 = splitmix64(st) | 1ull;
    ps.p[a].b = splitmix64(st);
    ps.p[a].a2 = splitmix64(st) | 1ull;
  }
  return ps;
}

// c[s * V + a] = Phi^{-1}((perm_a(s) + 1/2) / S), rounded to fp32.
__global__ void gauss_codebook_kernel(float* c, int n, int V, PermSet perms) {
  const int64_t S = (int64_t)1 << n;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= S * V) return;
  const int64_t s = i / V;
  const int a = (int)(i - s * V);
  const uint32_t r = perm_n((uint32_t)s, n, perms.p[a]);
  c[i] = (float)norm_inv(((double)r + 0.5) / (double)S);
}

// Adam (Kingma and Ba, 2015) with bias correction; the gradient is first
// clipped elementwise to [-clip, clip] when clip > 0 (the max-norm bound of
// the drift budget).  step counts from 1.
__global__ void adam_kernel(float* __restrict__ p, const float* __restrict__ g, float* __restrict__ m,
                            float* __restrict__ v, int64_t count, float lr, float b1, float b2, float eps,
                            float c1, float c2, float clip) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= count) return;
  float gi = g[i];
  if (clip > 0.f) gi = fminf(fmaxf(gi, -clip), clip);
  const float mi = fmaf(b1, m[i], (1.f - b1) * gi);
  const float vi = fmaf(b2, v[i], (1.f - b2) * gi * gi);
  m[i] = mi;
  v[i] = vi;
  // c1 = 1 / (1 - b1^step), c2 = 1 / (1 - b2^step)
  p[i] -= lr * (mi * c1) / (sqrtf(vi * c2) + eps);
}

// Plain gradient descent with the same elementwise clipping.
__global__ void sgd_kernel(float* __restrict__ p, const float* __restrict__ g, int64_t count, float lr,
                           float clip) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= count) return;
  float gi = g[i];
  if (clip > 0.f) gi = fminf(fmaxf(gi, -clip), clip);
  p[i] -= lr * gi;
}

}  // namespace
}  // namespace bcjr
