// bcjr_generic_kernels.h -- fp64 kernels for every trellis shape outside the
// super-group families of bcjr_kernels.h: fewer state bits than two shift
// digits (n < 2k, down to the fully connected n = k), shifts of k >= 4 bits,
// and the state counts whose group vectors do not fit in LDS (k = 1 at 15
// and 16 state bits, k = 3 above 14).
//
// Same recursions as the fast kernels (paper Sec. 3.4, Eqs. alpha, beta,
// marginal, soft-codeword; the VJP of Sec. 3.5 in its covariance form), in
// the group form that holds for any 1 <= k <= n:
//   log alpha_t(s) = h_t(s) + G_t(s >> k),   G_{t+1}(v) = LSE_j log alpha_t(j S/K + v)
//   log beta_t(s)  = H_t(s mod S/K),         H_{t-1}(v) = LSE_b [h_t(vK + b) + H_t((vK + b) mod S/K)]
// for v < S/K, so one step costs O(S) whatever K is.  Log values, tangents
// and every sum are fp64 (natural logs), with no renormalisation and no
// centring: at the temperatures the library takes, fp64 keeps the VJP's
// 1/T-amplified cancellations far below the tolerances.
//
// One block per workgroup of 256 threads, persistent over the blocks.  The
// group vectors and the per-step histories live in the workgroup's
// workspace slot (global memory, L2-resident for small S).  A K-way
// log-sum-exp is spread over TPO = min(K, 64, 256 / (S/K)) lanes (an aligned
// lane segment), each folding K / TPO inputs online, then merged with lane
// exchanges; merges are commutative, so every lane of a segment holds the
// same bits and the result does not depend on the schedule.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bcjr {

constexpr int kGenThreads = 256;

struct GenArgs {
  const float* w;      // [B, L]
  const float* g;      // [B, L] upstream gradient (VJP)
  const float* c;      // [S]
  int64_t B, L;
  int n, k;
  double inv2T;        // 1 / (2T)
  double invT;         // 1 / T
  float* w_soft;       // [B, L] or null
  float* logZ;         // [B] or null
  float* dW;           // [B, L] or null
  float* dc;           // [S] final dCodebook (written by gen_dc_reduce_kernel)
  double* ws;          // workspace: slots of slot_doubles
  int64_t slot_doubles;
  // Viterbi
  int32_t* states;     // [B, L]
  float* w_hard;       // [B, L] or null
  uint16_t* bp;        // [slots][L][S/K] winning predecessor digit j
};

namespace gen {

__device__ __forceinline__ double field(float w, float c, double inv2T) {
  const double d = (double)w - (double)c;
  return -(d * d) * inv2T;
}

// online (max, scaled sum, scaled weighted sum) accumulation of exp(x) and y exp(x)
__device__ __forceinline__ void acc3(double& m, double& s, double& y, double x, double yv) {
  if (x > m) {
    const double f = exp(m - x);  // m = -inf gives 0
    s = s * f + 1.0;
    y = y * f + yv;
    m = x;
  } else {
    const double e = exp(x - m);
    s += e;
    y += e * yv;
  }
}

__device__ __forceinline__ void merge3(double& m, double& s, double& y, double mo, double so, double yo) {
  const double M = fmax(m, mo);
  if (M == -INFINITY) return;
  const double f = exp(m - M), fo = exp(mo - M);
  s = s * f + so * fo;
  y = y * f + yo * fo;
  m = M;
}

// merge over an aligned segment of `width` lanes (a power of two <= 64)
__device__ __forceinline__ void seg_merge3(double& m, double& s, double& y, int width) {
  for (int o = 1; o < width; o <<= 1) {
    const double mo = __shfl_xor(m, o), so = __shfl_xor(s, o), yo = __shfl_xor(y, o);
    merge3(m, s, y, mo, so, yo);
  }
}

// (value, index) minimum over a segment: smaller value, then smaller index
__device__ __forceinline__ void seg_argmin(double& v, int& j, int width) {
  for (int o = 1; o < width; o <<= 1) {
    const double vo = __shfl_xor(v, o);
    const int jo = __shfl_xor(j, o);
    if (vo < v || (vo == v && jo < j)) {
      v = vo;
      j = jo;
    }
  }
}

// block-wide sums of NQ doubles (every thread gets the same bits); red holds
// [waves][NQ] doubles; the caller's barriers separate consecutive uses
template <int NQ>
__device__ __forceinline__ void block_sum(double (&v)[NQ], double* red) {
#pragma unroll
  for (int q = 0; q < NQ; ++q)
    for (int o = 32; o >= 1; o >>= 1) v[q] += __shfl_xor(v[q], o);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) red[wave * NQ + q] = v[q];
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    double t = red[q];
    for (int i = 1; i < kGenThreads / 64; ++i) t += red[i * NQ + q];
    v[q] = t;
  }
  __syncthreads();
}

// block-wide log-sum-exp of (m, s) pairs
__device__ __forceinline__ void block_lse(double& m, double& s, double* red) {
  double y = 0.0;
  seg_merge3(m, s, y, 64);
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[2 * wave] = m;
    red[2 * wave + 1] = s;
  }
  __syncthreads();
  m = red[0];
  s = red[1];
  for (int i = 1; i < kGenThreads / 64; ++i) merge3(m, s, y, red[2 * i], red[2 * i + 1], 0.0);
  __syncthreads();
}

struct Layout {
  int64_t GS;   // S / K
  int tpo;      // lanes per K-way reduction
  double *H, *Bt, *G0, *G1, *A0, *A1, *dcp;
};

__device__ __forceinline__ Layout layout(const GenArgs& a, bool vjp, bool dc) {
  Layout l;
  const int64_t S = (int64_t)1 << a.n;
  l.GS = S >> a.k;
  const int64_t K = (int64_t)1 << a.k;
  int64_t tpo = kGenThreads / l.GS;
  if (tpo < 1) tpo = 1;
  if (tpo > K) tpo = K;
  if (tpo > 64) tpo = 64;
  l.tpo = (int)tpo;
  double* p = a.ws + (int64_t)blockIdx.x * a.slot_doubles;
  l.H = p;           p += a.L * l.GS;
  l.Bt = vjp ? p : nullptr;  if (vjp) p += a.L * l.GS;
  l.G0 = p;          p += l.GS;
  l.G1 = p;          p += l.GS;
  l.A0 = p;          p += l.GS;
  l.A1 = p;          p += l.GS;
  l.dcp = dc ? p : nullptr;
  return l;
}

}  // namespace gen

// Soft codeword, logZ and (VJP) dW and the per-slot dCodebook partial.
template <bool VJP, bool DC>
__global__ void __launch_bounds__(kGenThreads) gen_fb_kernel(GenArgs a) {
  using namespace gen;
  __shared__ double red[(kGenThreads / 64) * 4];
  const int tid = threadIdx.x;
  const int64_t S = (int64_t)1 << a.n, K = (int64_t)1 << a.k;
  const Layout l = layout(a, VJP, DC);
  const int64_t GS = l.GS, mask = GS - 1;
  const int tpo = l.tpo, part = tid % tpo;
  const int64_t per_pass = kGenThreads / tpo, first_v = tid / tpo;
  const int kb = a.k;
  if (DC)
    for (int64_t s = tid; s < S; s += kGenThreads) l.dcp[s] = 0.0;
  for (int64_t blk = blockIdx.x; blk < a.B; blk += gridDim.x) {
    const float* wb = a.w + blk * a.L;
    const float* gb = VJP ? a.g + blk * a.L : nullptr;
    const int64_t L = a.L;
    // ---------------------------------------------------------- backward
    for (int64_t v = tid; v < GS; v += kGenThreads) {
      l.H[(L - 1) * GS + v] = 0.0;
      if (VJP) l.Bt[(L - 1) * GS + v] = 0.0;
    }
    __syncthreads();
    for (int64_t t = L - 1; t >= 1; --t) {
      const float wt = wb[t];
      const double gt = VJP ? (double)gb[t] : 0.0;
      const double* Hn = l.H + t * GS;
      const double* Bn = VJP ? l.Bt + t * GS : nullptr;
      for (int64_t v0 = first_v; v0 - first_v < GS; v0 += per_pass) {
        const int64_t v = v0 < GS ? v0 : GS - 1;  // idle lanes repeat the last output
        double m = -INFINITY, s = 0.0, y = 0.0;
        for (int64_t b = part; b < K; b += tpo) {
          const int64_t sp = v * K + b;
          const double yv = VJP ? gt * (double)a.c[sp] + Bn[sp & mask] : 0.0;
          acc3(m, s, y, field(wt, a.c[sp], a.inv2T) + Hn[sp & mask], yv);
        }
        seg_merge3(m, s, y, tpo);
        if (part == 0 && v0 < GS) {
          l.H[(t - 1) * GS + v] = m + log(s);
          if (VJP) l.Bt[(t - 1) * GS + v] = y / s;
        }
      }
      __syncthreads();
    }
    // logZ = LSE_s [h_0(s) + H_0(s mod S/K)]; with the VJP also E[X_0]
    double lz;
    {
      const float w0 = wb[0];
      double m = -INFINITY, s = 0.0, y = 0.0;
      for (int64_t st = tid; st < S; st += kGenThreads) acc3(m, s, y, field(w0, a.c[st], a.inv2T) + l.H[st & mask], 0.0);
      block_lse(m, s, red);
      lz = m + log(s);
      if (tid == 0 && a.logZ) a.logZ[blk] = (float)lz;
    }
    // ---------------------------------------------------------- forward
    for (int64_t v = tid; v < GS; v += kGenThreads) {
      l.G0[v] = 0.0;
      if (VJP) l.A0[v] = 0.0;
    }
    __syncthreads();
    double *Gc = l.G0, *Gn = l.G1, *Ac = l.A0, *An = l.A1;
    for (int64_t t = 0; t < L; ++t) {
      const float wt = wb[t];
      const double gt = VJP ? (double)gb[t] : 0.0;
      const double* Ht = l.H + t * GS;
      const double* Bt = VJP ? l.Bt + t * GS : nullptr;
      // marginal moments: sum p, sum p c, sum p X, sum p c X
      double mom[4] = {0.0, 0.0, 0.0, 0.0};
      for (int64_t st = tid; st < S; st += kGenThreads) {
        const double cs = (double)a.c[st];
        const double p = exp(field(wt, a.c[st], a.inv2T) + Gc[st >> kb] + Ht[st & mask] - lz);
        mom[0] += p;
        mom[1] += p * cs;
        if (VJP) {
          const double X = gt * cs + Ac[st >> kb] + Bt[st & mask];
          mom[2] += p * X;
          mom[3] += p * cs * X;
        }
      }
      // the next group vector (reads only step t's vectors)
      if (t + 1 < L) {
        for (int64_t v0 = first_v; v0 - first_v < GS; v0 += per_pass) {
          const int64_t v = v0 < GS ? v0 : GS - 1;
          double m = -INFINITY, s = 0.0, y = 0.0;
          for (int64_t j = part; j < K; j += tpo) {
            const int64_t sp = j * GS + v;
            const double yv = VJP ? gt * (double)a.c[sp] + Ac[sp >> kb] : 0.0;
            acc3(m, s, y, field(wt, a.c[sp], a.inv2T) + Gc[sp >> kb], yv);
          }
          seg_merge3(m, s, y, tpo);
          if (part == 0 && v0 < GS) {
            Gn[v] = m + log(s);
            if (VJP) An[v] = y / s;
          }
        }
      }
      block_sum<4>(mom, red);  // (its barriers also publish Gn, An)
      const double ws_t = mom[1] / mom[0];
      if (tid == 0) {
        if (a.w_soft) a.w_soft[blk * L + t] = (float)ws_t;
        if (VJP && a.dW) a.dW[blk * L + t] = (float)((mom[3] - ws_t * mom[2]) / mom[0] * a.invT);
      }
      if (DC) {
        // dc(s) += p_t(s) [g_t + (w_t - c(s)) (X_t(s) - E_p[X_t]) / T]
        const double xbar = mom[2] / mom[0];
        for (int64_t st = tid; st < S; st += kGenThreads) {
          const double cs = (double)a.c[st];
          const double p = exp(field(wt, a.c[st], a.inv2T) + Gc[st >> kb] + Ht[st & mask] - lz) / mom[0];
          const double X = gt * cs + Ac[st >> kb] + Bt[st & mask];
          l.dcp[st] += p * (gt + ((double)wt - cs) * (X - xbar) * a.invT);
        }
      }
      double* tg = Gc; Gc = Gn; Gn = tg;
      double* ta = Ac; Ac = An; An = ta;
      __syncthreads();
    }
  }
}

// dCodebook = sum over the slots of the fp64 partials, in slot order
__global__ void gen_dc_reduce_kernel(GenArgs a, int64_t nslots) {
  const int64_t S = (int64_t)1 << a.n;
  const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  const int64_t GS = S >> a.k;
  // the partial sits after H, B (2 L GS) and the four group vectors
  const int64_t off = 2 * a.L * GS + 4 * GS;
  double acc = 0.0;
  for (int64_t q = 0; q < nslots; ++q) acc += a.ws[q * a.slot_doubles + off + s];
  a.dc[s] = (float)acc;
}

// Min-sum decode (Sec. 3.2): m_t(s) = d_t(s) + Mn_t(s >> k),
// Mn_{t+1}(v) = min_j m_t(j S/K + v) (ties to the smallest j), the winning j
// kept per (t + 1, v); fp64 with the product and the sum rounded separately;
// the final state is the smallest one of minimal metric.
__global__ void __launch_bounds__(kGenThreads) gen_viterbi_kernel(GenArgs a) {
  __shared__ double redv[kGenThreads / 64];
  __shared__ int redi[kGenThreads / 64];
  const int tid = threadIdx.x;
  const int64_t S = (int64_t)1 << a.n, K = (int64_t)1 << a.k, GS = S >> a.k;
  int64_t tpo64 = kGenThreads / GS;
  if (tpo64 < 1) tpo64 = 1;
  if (tpo64 > K) tpo64 = K;
  if (tpo64 > 64) tpo64 = 64;
  const int tpo = (int)tpo64, part = tid % tpo;
  const int64_t per_pass = kGenThreads / tpo, first_v = tid / tpo;
  double* M0 = a.ws + (int64_t)blockIdx.x * a.slot_doubles;
  double* M1 = M0 + GS;
  uint16_t* bp = a.bp + (int64_t)blockIdx.x * a.L * GS;
  const int kb = a.k;
  for (int64_t blk = blockIdx.x; blk < a.B; blk += gridDim.x) {
    const float* wb = a.w + blk * a.L;
    const int64_t L = a.L;
    for (int64_t v = tid; v < GS; v += kGenThreads) M0[v] = 0.0;
    __syncthreads();
    double *Mc = M0, *Mn = M1;
    for (int64_t t = 0; t + 1 < L; ++t) {
      const double wt = (double)wb[t];
      for (int64_t v0 = first_v; v0 - first_v < GS; v0 += per_pass) {
        const int64_t v = v0 < GS ? v0 : GS - 1;
        double best = INFINITY;
        int bj = 0x7fffffff;
        for (int64_t j = part; j < K; j += tpo) {
          const int64_t s = j * GS + v;
          const double d = wt - (double)a.c[s];
          const double m = __dadd_rn(__dmul_rn(d, d), Mc[s >> kb]);
          if (m < best) {  // j ascending within the lane: strict keeps the smallest
            best = m;
            bj = (int)j;
          }
        }
        gen::seg_argmin(best, bj, tpo);
        if (part == 0 && v0 < GS) {
          Mn[v] = best;
          bp[(t + 1) * GS + v] = (uint16_t)(bj < K ? bj : 0);  // (no winner: non-finite input)
        }
      }
      double* tm = Mc; Mc = Mn; Mn = tm;
      __syncthreads();
    }
    // final metric and argmin over all states
    const double wl = (double)wb[L - 1];
    double best = INFINITY;
    int bs = 0x7fffffff;
    for (int64_t s = tid; s < S; s += kGenThreads) {
      const double d = wl - (double)a.c[s];
      const double m = __dadd_rn(__dmul_rn(d, d), Mc[s >> kb]);
      if (m < best) {
        best = m;
        bs = (int)s;
      }
    }
    gen::seg_argmin(best, bs, 64);
    if ((tid & 63) == 0) {
      redv[tid >> 6] = best;
      redi[tid >> 6] = bs;
    }
    __syncthreads();  // also publishes the digits
    if (tid == 0) {
      for (int i = 1; i < kGenThreads / 64; ++i)
        if (redv[i] < best || (redv[i] == best && redi[i] < bs)) {
          best = redv[i];
          bs = redi[i];
        }
      int32_t* st = a.states + blk * L;
      float* wh = a.w_hard ? a.w_hard + blk * L : nullptr;
      int64_t s = (bs >= 0 && bs < S) ? bs : 0;  // (non-finite inputs: no state below +inf)
      for (int64_t t = L - 1;; --t) {
        st[t] = (int32_t)s;
        if (wh) wh[t] = a.c[s];
        if (t == 0) break;
        const int64_t v = s >> kb;
        s = (int64_t)bp[t * GS + v] * GS + v;
      }
    }
    __syncthreads();
  }
}

}  // namespace bcjr
