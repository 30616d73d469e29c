// bcjr_rot_kernels.h -- fused forward-backward + VJP at S = 65536, k = 2 with
// the group vectors exchanged in place through a rotating LDS layout.
//
// fb_kernel's exchange reads a super-group's K entries in one form (rows in
// the backward sweep, columns in the forward) and writes its K outputs in
// the other, so every step needs all reads done before any write: two
// barriers per step and the outputs held in registers across the first.
// Here each super-group writes its K outputs into the K slots it has just
// read.  With the group index g (14 bits, 7 base-4 digits) and
//   column entry (j, x) = j * NSG + x,   row entry (x, u) = x * K + u,
// the row entry (x, u) of step t + 1 (forward) must then sit where the
// column entry (u, x) of step t sat; row (x, u) is the column index rotated
// left by one digit, so logical entry g of a vector is stored at
//   slot(g, r) = Phi(rotr(g, 2r)),   r = the step's rotation (period 7),
// and one barrier per step separates a step's writes from the next step's
// reads.  Both sweeps address column entries at a rotation r: the forward at
// r = t mod 7, the backward reads the row entries of step t, which are the
// column entries of rotation (t - 1) mod 7, and writes its outputs (the
// column entries of step t - 1) at that same rotation.
//
// Phi is a GF(2)-linear bijection of the 14 bits, circulant over the base-4
// digits (so it commutes with the rotation), chosen so that for every
// rotation the 64 lanes of a wave -- consecutive super-groups, which differ
// in the low 6 bits of x -- reach 64 distinct 4-byte banks and each half
// wave 32 distinct 8-byte slots: the (value, tangent) pairs are read and
// written with 8-byte accesses and no bank conflicts.  Because Phi commutes
// with the rotation, the slot of (j, x = tb + i * TPB) is
//   rotr(Phi(tb), 2r) ^ rotr(Phi(i << 9), 2r) ^ rotr(Phi(j << 12), 2r):
// a per-thread term (one bit-field extract per step) and two scalars.
//
// Values are written unshifted: the integer shift of the step (the floor of
// its maximum, known after the barrier) and, in the forward sweep, the
// centring of the A tangent on g_t w_soft_t are applied when the entries are
// read at the next step; the (H, B) history keeps the unshifted values and
// the forward sweep folds the recorded shift into its lambda estimate.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bcjr_device.h"
#include "bcjr_internal.h"

namespace bcjr {
namespace rot {

// Phi(e_p) for the 14 input bits (bit p of the group index)
constexpr uint32_t kPhiCol[14] = {0x2149, 0x328e, 0x0526, 0x0a3b, 0x1498, 0x28ec, 0x1261,
                                  0x23b2, 0x0985, 0x0eca, 0x2614, 0x3b28, 0x1852, 0x2ca3};

__host__ __device__ constexpr uint32_t phi(uint32_t x) {
  uint32_t v = 0;
  for (int p = 0; p < 14; ++p)
    if ((x >> p) & 1u) v ^= kPhiCol[p];
  return v;
}

// v in 14 bits, stored twice side by side: rotr(v, s) = (rep >> s) & 0x3FFF
__host__ __device__ constexpr uint32_t rep(uint32_t v) { return v | (v << 14); }

// byte offset of an (value, tangent) pair slot from its replicated Phi term
__device__ __forceinline__ uint32_t slot8(uint32_t repv, uint32_t r2) {
  return ((repv >> r2) & 0x3FFFu) << 3;
}

// the same for a compile-time Phi term: a scalar (SGPR) value
__device__ __forceinline__ uint32_t slot8s(uint32_t repv, uint32_t r2) {
  return __builtin_amdgcn_readfirstlane(((repv >> r2) & 0x3FFFu) << 3);
}

__device__ __forceinline__ float2 ld_pair(const float* lds, uint32_t off) {
  return *reinterpret_cast<const float2*>(reinterpret_cast<const char*>(lds) + off);
}

__device__ __forceinline__ void st_pair(float* lds, uint32_t off, float a, float b) {
  *reinterpret_cast<float2*>(reinterpret_cast<char*>(lds) + off) = make_float2(a, b);
}

}  // namespace rot

// S = 65536 (n = 16), k = 2: 4096 super-groups, 512 threads of 8 each, the
// codebook rows of a thread's super-groups resident in registers (as in
// fb_kernel's 512-thread family); fwd + w_soft + logZ + dW, no dCodebook.
// With no outputs held across a barrier the kernel needs ~190 of its 256
// VGPRs under the default scheduler; its translation unit is built with the
// ILP-oriented one and no scheduling fences between output groups, which
// lets consecutive output groups and super-groups overlap (the sweeps are
// bound by the latency of their dependence chains at two waves per SIMD).
__global__ void __launch_bounds__(512) fb_kernel_rot(FbArgs a) {
  constexpr int KB = 2, K = 4, n = 16;
  constexpr int GS = 1 << (n - KB);        // 16384 groups
  constexpr int NSG = 1 << (n - 2 * KB);   // 4096 super-groups
  constexpr int SGT = 8, TPB = 512, NT = 512;
  extern __shared__ float lds[];           // [GS] (value, tangent) pairs, then the reduction area
  const int64_t L = a.L;
  const float kap = a.kap;

  RedCtx rc;
  rc.width = 64;
  rc.rw = TPB / 64;
  rc.wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  float* const red0 = lds + 2 * GS;

  const rsrc_t cbk = make_rsrc(a.cs, (uint32_t)4 << n);
  const uint32_t tb0 = threadIdx.x;
  const uint32_t voK = tb0 << (KB + 2);
  constexpr uint32_t hstep = (uint32_t)GS * 2;   // floats per history step: H then B, [S/K] each
  const uint32_t wave_s = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // the thread's Phi term, replicated for the rotation
  uint32_t phtb = 0;
#pragma unroll
  for (int p = 0; p < 9; ++p) phtb ^= ((tb0 >> p) & 1u) ? rot::kPhiCol[p] : 0u;
  phtb = rot::rep(phtb);
  // repair pass after the linear-domain kernel: only the blocks it marked
  if (a.repair) {
    int any = 0;
    for (int64_t base = blockIdx.x; base < a.B; base += gridDim.x) any |= ld_uniform_i(a.flags, base);
    if (!any) return;
  }
  float cbr[SGT][K][K];
#pragma unroll
  for (int i = 0; i < SGT; ++i) {
#pragma unroll
    for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((i * TPB) << KB)) * 4, cbr[i][j]);
  }

  for (int64_t base = blockIdx.x; base < a.B; base += gridDim.x) {
    if (a.repair && !ld_uniform_i(a.flags, base)) continue;
    const int64_t bb = base;            // the block (one per workgroup)
    const int64_t slot = blockIdx.x;
    // its rows are wave-uniform: w_t and g_t come through scalar loads
    const int64_t bbu = (int64_t)__builtin_amdgcn_readfirstlane((int)bb);
    const float* wbu = a.w + bbu * L;
    const float* gbu = a.g + bbu * L;
    const rsrc_t hist = make_rsrc(a.histHB + slot * L * hstep, (uint32_t)L * hstep * 4u);
    float* sm_mB = a.small + slot * 3 * L;  // shift of H_t (applied on read)

    // ------------------------------------------------------------------ S0
    // Backward: H and B in the pair slots, in place; one barrier per step.
    for (int i = threadIdx.x; i < 2 * GS; i += NT) lds[i] = 0.f;
    __syncthreads();
    int shiftB = 0;
    float lam0 = 0.f, xbar = 0.f;
    float offc = 0.f;  // shift of the H values being read
    float wnx = ld_uniform(wbu, L - 1);
    float gnx = ld_uniform(gbu, L - 1);
    uint32_t r2 = (uint32_t)(2 * (((L - 1) + 6) % 7));  // rotation of step L - 1's reads
    for (int64_t t = L - 1;; --t) {
      const uint32_t tid_s = lane_tid(wave_s);
      const uint32_t vcH = tid_s * 4u;
      rc.red = red0 + ((L - 1 - t) & 1) * (NT / 64) * kRed;
      const float wt = wnx * kap, gt = gnx;
      {
        const int64_t tn = t > 0 ? t - 1 : 0;
        wnx = ld_uniform(wbu, tn);
        gnx = ld_uniform(gbu, tn);
      }
      const uint32_t rs = __builtin_amdgcn_readfirstlane(r2);
      const uint32_t tslot = rot::slot8(phtb, rs);
      const uint32_t soH = (uint32_t)t * hstep * 4u;
      if (t == 0) {
        float lm = -INFINITY, ls = 0.f, ly = 0.f;
#pragma unroll
        for (int i = 0; i < SGT; ++i) {
          uint32_t ts = tslot;
          float wtl = wt;
          pin_u(ts);
          pin(wtl);
          const uint32_t si = ts ^ rot::slot8s(rot::rep(rot::phi((uint32_t)i << 9)), rs);
          float Hin[K], Bin[K];
#pragma unroll
          for (int b = 0; b < K; ++b) {
            const float2 v = rot::ld_pair(lds, si ^ rot::slot8s(rot::rep(rot::phi((uint32_t)b << 12)), rs));
            Hin[b] = v.x - offc;
            Bin[b] = v.y;
          }
#pragma unroll
          for (int j = 0; j < K; ++j) {
            float x[K];
#pragma unroll
            for (int b = 0; b < K; ++b) {
              const float d = wtl - cbr[i][j][b];
              x[b] = fmaf(-d, d, Hin[b]);
            }
            const float m = max_of<K>(x);
            float E[K];
#pragma unroll
            for (int b = 0; b < K; ++b) E[b] = ex2(x[b] - m);
            float s = E[0];
#pragma unroll
            for (int b = 1; b < K; ++b) s += E[b];
            float sy = E[0] * fmaf(gt, cbr[i][j][0], Bin[0]);
#pragma unroll
            for (int b = 1; b < K; ++b) sy = fmaf(E[b], fmaf(gt, cbr[i][j][b], Bin[b]), sy);
            lse3_pair(lm, ls, ly, m, s, sy);
          }
          asm volatile("" ::: "memory");  // the super-groups' LDS accesses stay in order
        }
        lse3_pre(lm, ls, ly, rc);
        if (threadIdx.x == 0) sm_mB[L - 1] = 0.f;
        __syncthreads();
        lse3_post(lm, ls, ly, rc);
        xbar = ly / ls;
        lam0 = lm + lg2(ls);
        if (threadIdx.x == 0 && a.logZ)
          a.logZ[bb] = (float)(((double)shiftB + (double)lam0) * 0.69314718055994530942);
        __syncthreads();
        break;
      }
      float vmax[1] = {-INFINITY};
#pragma unroll
      for (int i = 0; i < SGT; ++i) {
        uint32_t ts = tslot;
        float wtl = wt;
        pin_u(ts);
        pin(wtl);
        const uint32_t si = ts ^ rot::slot8s(rot::rep(rot::phi((uint32_t)i << 9)), rs);
        uint32_t sl[K];
#pragma unroll
        for (int b = 0; b < K; ++b) sl[b] = si ^ rot::slot8s(rot::rep(rot::phi((uint32_t)b << 12)), rs);
        float Hin[K], Bin[K];
#pragma unroll
        for (int b = 0; b < K; ++b) {
          const float2 v = rot::ld_pair(lds, sl[b]);
          Hin[b] = v.x - offc;
          Bin[b] = v.y;
        }
#pragma unroll
        for (int j = 0; j < K; ++j) {
          float x[K], d[K];
#pragma unroll
          for (int b = 0; b < K; ++b) {
            d[b] = wtl - cbr[i][j][b];
            x[b] = fmaf(-d[b], d[b], Hin[b]);
          }
          const float m = max_of<K>(x);
          float E[K];
#pragma unroll
          for (int b = 0; b < K; ++b) E[b] = ex2(x[b] - m);
          float s = E[0];
#pragma unroll
          for (int b = 1; b < K; ++b) s += E[b];
          const float h = m + lg2(s);
          vmax[0] = fmaxf(vmax[0], h);
          // B_{t-1} = E-weighted mean of g_t (c - w_t) + B_t over the K successors
          float num = E[0] * fmaf(-gt, d[0], Bin[0]);
#pragma unroll
          for (int b = 1; b < K; ++b) num = fmaf(E[b], fmaf(-gt, d[b], Bin[b]), num);
          const float hv[1] = {h}, bv[1] = {num * rcp(s)};
          rot::st_pair(lds, sl[j], hv[0], bv[0]);
          // history entries of step t - 1: group j NSG + i TPB + tb (unshifted)
          const uint32_t so = soH - hstep * 4u + (uint32_t)(j * NSG + i * TPB) * 4u;
          buf_st<1, kStream>(hist, vcH, so, hv);
          buf_st<1, kStream>(hist, vcH, so + (uint32_t)GS * 4u, bv);
        }
        asm volatile("" ::: "memory");  // the super-groups' LDS accesses stay in order
      }
      red_pre<1, 1u>(vmax, rc);
      __syncthreads();
      red_post<1, 1u>(vmax, rc);
      const float off = floorf(vmax[0]);
      shiftB += __builtin_amdgcn_readfirstlane((int)off);
      if (threadIdx.x == 0) sm_mB[t - 1] = off;
      offc = off;
      r2 = r2 == 0 ? 12u : r2 - 2u;
    }

    // ------------------------------------------------------------------ S1
    // Forward: G and the A tangent in the pair slots, in place; one barrier
    // per step.  A_t(s) = E[sum_{tau < t} g_tau (c(s_tau) - w_soft_tau) | s_t = s]
    // is centred on the soft codeword when it is read; X_t = g_t c + A_t + B_t
    // - xbar_t as in fb_kernel.
    for (int i = threadIdx.x; i < 2 * GS; i += NT) lds[i] = 0.f;
    __syncthreads();
    const float dws = a.dws;
    float lam_est = lam0;
    float goff = 0.f, cprev = 0.f;  // shift of G and centring of A, applied on read
    float pH[K], pB[K];
    wnx = ld_uniform(wbu, 0);
    gnx = ld_uniform(gbu, 0);
    {
      const uint32_t voH0 = lane_tid(wave_s) * K * 4u;
      hist_row<K, true>(hist, voH0, 0, 0, (uint32_t)GS * 4u, pH, pB);
    }
    r2 = 0;
    for (int64_t t = 0; t < L; ++t) {
      const uint32_t tid_s = lane_tid(wave_s);
      const uint32_t voH_s = tid_s * K * 4u;
      rc.red = red0 + (t & 1) * (NT / 64) * kRed;
      const float wt = wnx * kap, gt = gnx;
      {
        const int64_t tn = t + 1 < L ? t + 1 : t;
        wnx = ld_uniform(wbu, tn);
        gnx = ld_uniform(gbu, tn);
      }
      if (t > 0) xbar = fmaf(gt, wt, xbar);  // B_t no longer holds step t
      const float mBt = sm_mB[t];
      const float lam_adj = lam_est + mBt;  // the history holds H_t + mBt
      const uint32_t rs = __builtin_amdgcn_readfirstlane(r2);
      const uint32_t tslot = rot::slot8(phtb, rs);
      // max G_{t+1}, sum p, sum p c, sum p X, sum p c X
      float rv[5] = {-INFINITY, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < SGT; ++i) {
        uint32_t ts = tslot;
        float wtl = wt;
        pin_u(ts);
        pin(wtl);
        const uint32_t si = ts ^ rot::slot8s(rot::rep(rot::phi((uint32_t)i << 9)), rs);
        uint32_t sl[K];
#pragma unroll
        for (int j = 0; j < K; ++j) sl[j] = si ^ rot::slot8s(rot::rep(rot::phi((uint32_t)j << 12)), rs);
        float Gin[K], Ain[K];
#pragma unroll
        for (int j = 0; j < K; ++j) {
          const float2 v = rot::ld_pair(lds, sl[j]);
          Gin[j] = v.x - goff;
          Ain[j] = v.y - cprev;
        }
        float Hc[K], Bc[K];
#pragma unroll
        for (int u = 0; u < K; ++u) {
          Hc[u] = pH[u];
          Bc[u] = pB[u];
        }
        {  // the next super-group's history row (the first of the next step after the last)
          const bool last = i + 1 >= SGT;
          const int64_t tn = last && t + 1 < L ? t + 1 : t;
          hist_row<K, true>(hist, voH_s, (uint32_t)tn * hstep * 4u,
                            last ? 0u : (uint32_t)(i + 1) * TPB * K * 4u, (uint32_t)GS * 4u, pH, pB);
        }
#pragma unroll
        for (int u = 0; u < K; ++u) {
          float al[K];
#pragma unroll
          for (int j = 0; j < K; ++j) {
            const float d = wtl - cbr[i][j][u];
            al[j] = fmaf(-d, d, Gin[j]);
          }
          const float m = max_of<K>(al);
          float E[K];
#pragma unroll
          for (int j = 0; j < K; ++j) E[j] = ex2(al[j] - m);
          float s = E[0], ec = E[0] * cbr[i][0][u], sc = ec;
          float y = fmaf(gt, cbr[i][0][u], Ain[0]);
          float sy = E[0] * y, scy = ec * y;
#pragma unroll
          for (int j = 1; j < K; ++j) {
            s += E[j];
            ec = E[j] * cbr[i][j][u];
            sc += ec;
            y = fmaf(gt, cbr[i][j][u], Ain[j]);
            sy = fmaf(E[j], y, sy);
            scy = fmaf(ec, y, scy);
          }
          const float go = m + lg2(s);
          rv[0] = fmaxf(rv[0], go);
          const float fac = ex2(m + Hc[u] - lam_adj);
          rv[1] = fmaf(fac, s, rv[1]);
          rv[2] = fmaf(fac, sc, rv[2]);
          const float bx = Bc[u] - xbar;
          rv[3] = fmaf(fac, fmaf(s, bx, sy), rv[3]);
          rv[4] = fmaf(fac, fmaf(sc, bx, scy), rv[4]);
          rot::st_pair(lds, sl[u], go, sy * rcp(s));
        }
        asm volatile("" ::: "memory");  // the super-groups' LDS accesses stay in order
      }
      red_pre<5, 1u>(rv, rc);
      __syncthreads();
      red_post<5, 1u>(rv, rc);
      const float off = floorf(rv[0]);
      const float r1 = 1.f / rv[1];
      const float wst = rv[2] * r1;
      const float lamt = lam_est + lg2(rv[1]);
      if (threadIdx.x == 0) {
        if (a.w_soft) a.w_soft[bb * L + t] = wst * a.inv_kap;
        if (a.dW) a.dW[bb * L + t] = (rv[4] - wst * rv[3]) * r1 * dws;
      }
      lam_est = lamt - off + mBt;
      goff = off;
      cprev = gt * wst;
      // E_p[X_t] = xbar + sum p X / sum p; X_{t+1} drops g_t w_soft_t (A is
      // centred on read); it gains g_{t+1} w_{t+1} at the top of the next step
      xbar = fmaf(rv[3], r1, xbar) - cprev;
      r2 = r2 == 12u ? 0u : r2 + 2u;
    }
    __syncthreads();
  }
}

namespace rot {
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) f32x2 lds_f2;

// (value, tangent) pair at an absolute LDS byte address
__device__ __forceinline__ float2 ld_pair_at(uint32_t addr) {
  const f32x2 v = *reinterpret_cast<const lds_f2*>(addr);
  const float x = v.x, y = v.y;
  return make_float2(x, y);
}
__device__ __forceinline__ void st_pair_at(uint32_t addr, float a, float b) {
  const f32x2 v = {a, b};
  *reinterpret_cast<lds_f2*>(addr) = v;
}

constexpr int kTopExp = 40;                  // a rescale puts the largest entry at 2^40
constexpr float kTop = 1099511627776.0f;     // 2^40

// e with x = m 2^e, 1 <= m < 2, for a positive normal x (-127 for zero or a
// denormal, 128 for inf or NaN)
__device__ __forceinline__ int exp_of(float x) { return (int)((__float_as_uint(x) >> 23) & 0xFFu) - 127; }
}  // namespace rot

// The same call (S = 65536, k = 2, fwd + w_soft + logZ + dW, no dCodebook) on
// the same rotating layout, workspace and history, with the group vectors
// kept in the linear domain instead of the log domain:
//   G_{t+1}(v) = sum_j e_t(j, v) G_t(j, v >> 2),  H_{t-1}(v) = sum_b e_t(v, b) H_t(...),
// e_t(s) = 2^(h_t(s)) = 2^(-(w'_t - c'_s)^2) (the Boltzmann weight of the
// local field, Eq. boltzmann), and the tangents carried unnormalised
// (G A and H B), so that a step needs one exponential per state and no
// logarithm, maximum or reciprocal per group.  After each step the vector
// is rescaled by an exact power of two that puts its largest entry at 2^40
// (the exponent is folded into the next step's exponentials); fp32 then
// holds every state within ~166 log2 units of the step's maximum at full
// precision, where the states that carry the posterior lie within ~60-90
// at T >= 0.04 on unit-variance data.  The marginals and the four dW moments
// are products of the two sweeps' values, scale-invariant per step.
//
// A block whose vectors leave that range -- a step whose largest entry
// falls below 2^-30 (a single-step decay of 70 log2 units, which the
// posterior states would not survive) or the forward's per-step mass
// sum_s alpha_t beta_t departing from Z by more than 2e-4 log2 units -- is
// marked in a.flags and recomputed by a second launch of the log-domain
// (or, at field scales above 18, the double-float) kernel in repair mode.
template <int NT, bool VJP>
__global__ void __launch_bounds__(NT) fb_kernel_lin(FbArgs a) {
  constexpr int KB = 2, K = 4, n = 16;
  constexpr int GS = 1 << (n - KB);        // 16384 groups
  constexpr int NSG = 1 << (n - 2 * KB);   // 4096 super-groups
  constexpr int TPB = NT, SGT = NSG / NT;
  constexpr int TB_BITS = NT == 1024 ? 10 : 9;
  static_assert(NT == 512 || NT == 1024, "512 or 1024 threads");
  extern __shared__ float lds[];           // [GS] (value, tangent) pairs, then the reduction area
  const int64_t L = a.L;
  const float kap = a.kap;

  RedCtx rc;
  rc.width = 64;
  rc.rw = TPB / 64;
  rc.wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  float* const red0 = lds + 2 * GS;

  // LDS byte address of the pair vector: it starts on a 128 KiB boundary
  // (at 0: the kernel has no static LDS), so it is XORed into the scalar
  // slot terms and no address needs an add.  Were it not aligned, every
  // block is marked for the repair pass (whose kernels address LDS plainly).
  const uint32_t lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  const bool lds_aligned = (lds0 & 0x1FFFFu) == 0u;
  const rsrc_t cbk = make_rsrc(a.cs, (uint32_t)4 << n);
  const uint32_t tb0 = threadIdx.x;
  const uint32_t voK = tb0 << (KB + 2);
  // floats per history step: H then (VJP) H B, [S/K] each
  constexpr uint32_t hstep = (uint32_t)GS * (VJP ? 2 : 1);
  const uint32_t wave_s = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  uint32_t phtb = 0;
#pragma unroll
  for (int p = 0; p < TB_BITS; ++p) phtb ^= ((tb0 >> p) & 1u) ? rot::kPhiCol[p] : 0u;
  phtb = rot::rep(phtb);
  float cbr[SGT][K][K];
#pragma unroll
  for (int i = 0; i < SGT; ++i) {
#pragma unroll
    for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((i * TPB) << KB)) * 4, cbr[i][j]);
  }

  for (int64_t base = blockIdx.x; base < a.B; base += gridDim.x) {
    const int64_t bb = base;
    const int64_t slot = blockIdx.x;
    const int64_t bbu = (int64_t)__builtin_amdgcn_readfirstlane((int)bb);
    const float* wbu = a.w + bbu * L;
    const float* gbu = VJP ? a.g + bbu * L : wbu;
    const rsrc_t hist = make_rsrc((VJP ? a.histHB : a.histH) + slot * L * hstep, (uint32_t)L * hstep * 4u);
    float* sm_eH = a.small + slot * 3 * L;  // exponent of the stored H_t: stored = true * 2^e
    bool bad = !lds_aligned;
    {  // the history's step L - 1 entries: H = 1, then H B = 0
      const float one[4] = {1.f, 1.f, 1.f, 1.f}, zero[4] = {0.f, 0.f, 0.f, 0.f};
      const uint32_t so = (uint32_t)(L - 1) * hstep * 4u;
      for (uint32_t q = threadIdx.x; q < (uint32_t)GS / 4; q += NT) {
        buf_st<4, kStream>(hist, q * 16u, so, one);
        if constexpr (VJP) buf_st<4, kStream>(hist, q * 16u, so + (uint32_t)GS * 4u, zero);
      }
    }

    // ------------------------------------------------------------------ S0
    // Backward: H and the unnormalised tangent H B in the pair slots, in
    // place; H_{L-1} = 1 is stored as 2^40.
    for (int i = threadIdx.x; i < 2 * GS; i += NT) lds[i] = (i & 1) ? 0.f : rot::kTop;
    __syncthreads();
    int ex = rot::kTopExp;  // exponent of the vector being read
    int off = 0;            // its rescale, folded into this step's exponentials
    float lz2 = 0.f, xbar = 0.f;
    float wnx = ld_uniform(wbu, L - 1);
    float gnx = VJP ? ld_uniform(gbu, L - 1) : 0.f;
    uint32_t r2 = (uint32_t)(2 * (((L - 1) + 6) % 7));
    for (int64_t t = L - 1;; --t) {
      const uint32_t tid_s = lane_tid(wave_s);
      const uint32_t vcH = tid_s * 4u;
      rc.red = red0 + ((L - 1 - t) & 1) * (NT / 64) * kRed;
      const float wt = wnx * kap, gt = gnx;
      {
        const int64_t tn = t > 0 ? t - 1 : 0;
        wnx = ld_uniform(wbu, tn);
        if constexpr (VJP) gnx = ld_uniform(gbu, tn);
      }
      const float noff = -(float)off;
      const uint32_t rs = __builtin_amdgcn_readfirstlane(r2);
      const uint32_t tslot = rot::slot8(phtb, rs);
      const uint32_t soH = (uint32_t)t * hstep * 4u;
      if (t == 0) {
        // Z = sum_s alpha_0(s) beta_0(s) and E_p[g_0 (c - w_0) + B_0]
        float ls = 0.f, ly = 0.f;
#pragma unroll
        for (int i = 0; i < SGT; ++i) {
          uint32_t ts = tslot;
          float wtl = wt;
          pin_u(ts);
          pin(wtl);
          const uint32_t si = ts ^ (rot::slot8s(rot::rep(rot::phi((uint32_t)i << TB_BITS)), rs) ^ lds0);
          float Hin[K], Bin[K];
#pragma unroll
          for (int b = 0; b < K; ++b) {
            const float2 v = rot::ld_pair_at(si ^ rot::slot8s(rot::rep(rot::phi((uint32_t)b << 12)), rs));
            Hin[b] = v.x;
            Bin[b] = v.y;
          }
#pragma unroll
          for (int j = 0; j < K; ++j) {
#pragma unroll
            for (int b = 0; b < K; ++b) {
              const float d = wtl - cbr[i][j][b];
              const float e = ex2(fmaf(-d, d, noff));
              ls = fmaf(e, Hin[b], ls);
              if constexpr (VJP) ly = fmaf(e, fmaf(-gt * d, Hin[b], Bin[b]), ly);
            }
          }
          asm volatile("" ::: "memory");
        }
        float sv[2] = {ls, ly};
        red_pre<2, 0u>(sv, rc);
        if (threadIdx.x == 0) sm_eH[L - 1] = 0.f;  // the history's H_{L-1} entries are 1
        __syncthreads();
        red_post<2, 0u>(sv, rc);
        if (!(sv[0] > 0.f && sv[0] < INFINITY)) bad = true;
        lz2 = lg2(sv[0]) - (float)(ex - off);
        xbar = sv[1] / sv[0];
        if (threadIdx.x == 0 && a.logZ) a.logZ[bb] = (float)((double)lz2 * 0.69314718055994530942);
        __syncthreads();
        break;
      }
      float vmax[1] = {0.f};
#pragma unroll
      for (int i = 0; i < SGT; ++i) {
        uint32_t ts = tslot;
        float wtl = wt;
        pin_u(ts);
        pin(wtl);
        const uint32_t si = ts ^ (rot::slot8s(rot::rep(rot::phi((uint32_t)i << TB_BITS)), rs) ^ lds0);
        uint32_t sl[K];
#pragma unroll
        for (int b = 0; b < K; ++b) sl[b] = si ^ rot::slot8s(rot::rep(rot::phi((uint32_t)b << 12)), rs);
        float Hin[K], Bin[K], gH[K];
#pragma unroll
        for (int b = 0; b < K; ++b) {
          const float2 v = rot::ld_pair_at(sl[b]);
          Hin[b] = v.x;
          Bin[b] = v.y;
          gH[b] = VJP ? gt * v.x : 0.f;  // shared by the K output groups
        }
#pragma unroll
        for (int j = 0; j < K; ++j) {
          float e[K], d[K];
#pragma unroll
          for (int b = 0; b < K; ++b) {
            d[b] = wtl - cbr[i][j][b];
            e[b] = ex2(fmaf(-d[b], d[b], noff));
          }
          float hv0 = e[0] * Hin[0];
#pragma unroll
          for (int b = 1; b < K; ++b) hv0 = fmaf(e[b], Hin[b], hv0);
          vmax[0] = fmaxf(vmax[0], hv0);
          const float hv[1] = {hv0};
          // history entries of step t - 1: group j NSG + i TPB + tb
          const uint32_t so = soH - hstep * 4u + (uint32_t)(j * NSG + i * TPB) * 4u;
          if constexpr (VJP) {
            // H B_{t-1} = sum_b e_b (H B_b + g_t H_b (c_b - w_t)), the
            // step's term -g_t H_b d_b folded in before the product with e_b
            float bv0 = e[0] * fmaf(-gH[0], d[0], Bin[0]);
#pragma unroll
            for (int b = 1; b < K; ++b) bv0 = fmaf(e[b], fmaf(-gH[b], d[b], Bin[b]), bv0);
            const float bv[1] = {bv0};
            rot::st_pair_at(sl[j], hv[0], bv[0]);
            buf_st<1, kStream>(hist, vcH, so, hv);
            buf_st<1, kStream>(hist, vcH, so + (uint32_t)GS * 4u, bv);
          } else {
            rot::st_pair_at(sl[j], hv[0], 0.f);
            buf_st<1, kStream>(hist, vcH, so, hv);
          }
        }
        asm volatile("" ::: "memory");
      }
      red_pre<1, 1u>(vmax, rc);
      __syncthreads();
      red_post<1, 1u>(vmax, rc);
      ex -= off;  // the exponent of what this step wrote
      if (threadIdx.x == 0) sm_eH[t - 1] = (float)ex;
      if (!(vmax[0] >= 0x1p-30f && vmax[0] <= 0x1p100f)) bad = true;
      off = bad ? 0 : rot::exp_of(vmax[0]) - rot::kTopExp;
      r2 = r2 == 0 ? 12u : r2 - 2u;
    }

    // ------------------------------------------------------------------ S1
    // Forward: G and the unnormalised tangent G A in the pair slots, in
    // place; G_0 = 1 stored as 2^40.  A is centred on g_{t-1} w_soft_{t-1}
    // when it is read (G A - c G).
    for (int i = threadIdx.x; i < 2 * GS; i += NT) lds[i] = (i & 1) ? 0.f : rot::kTop;
    __syncthreads();
    const float dws = a.dws;
    float cprev = 0.f;
    ex = rot::kTopExp;
    off = 0;
    float pH[K], pB[K];
    wnx = ld_uniform(wbu, 0);
    gnx = VJP ? ld_uniform(gbu, 0) : 0.f;
    {
      const uint32_t voH0 = lane_tid(wave_s) * K * 4u;
      hist_row<K, VJP>(hist, voH0, 0, 0, (uint32_t)GS * 4u, pH, pB);
    }
    r2 = 0;
    for (int64_t t = 0; t < L; ++t) {
      const uint32_t tid_s = lane_tid(wave_s);
      const uint32_t voH_s = tid_s * K * 4u;
      rc.red = red0 + (t & 1) * (NT / 64) * kRed;
      const float wt = wnx * kap, gt = gnx;
      {
        const int64_t tn = t + 1 < L ? t + 1 : t;
        wnx = ld_uniform(wbu, tn);
        if constexpr (VJP) gnx = ld_uniform(gbu, tn);
      }
      const float eHt = sm_eH[t];
      const float noff = -(float)off;
      const uint32_t rs = __builtin_amdgcn_readfirstlane(r2);
      const uint32_t tslot = rot::slot8(phtb, rs);
      // max G_{t+1}, sum P d, sum P, sum P (X - xbar), sum P (X - xbar) d with
      // P = alpha_t beta_t and d = w'_t - c' (moments about the weight: their
      // terms are of the size of the quantisation error, not of c')
      constexpr int NRV = VJP ? 5 : 3;
      float rv[NRV];
#pragma unroll
      for (int q = 0; q < NRV; ++q) rv[q] = 0.f;
#pragma unroll
      for (int i = 0; i < SGT; ++i) {
        uint32_t ts = tslot;
        float wtl = wt;
        pin_u(ts);
        pin(wtl);
        const uint32_t si = ts ^ (rot::slot8s(rot::rep(rot::phi((uint32_t)i << TB_BITS)), rs) ^ lds0);
        uint32_t sl[K];
#pragma unroll
        for (int j = 0; j < K; ++j) sl[j] = si ^ rot::slot8s(rot::rep(rot::phi((uint32_t)j << 12)), rs);
        float Gin[K], Ain[K], gG[K];
#pragma unroll
        for (int j = 0; j < K; ++j) {
          const float2 v = rot::ld_pair_at(sl[j]);
          Gin[j] = v.x;
          Ain[j] = VJP ? fmaf(-cprev, v.x, v.y) : 0.f;
          gG[j] = VJP ? gt * v.x : 0.f;  // shared by the K output groups
        }
        float Hc[K], Bc[K];
#pragma unroll
        for (int u = 0; u < K; ++u) {
          Hc[u] = pH[u];
          Bc[u] = VJP ? pB[u] : 0.f;
        }
        {
          const bool last = i + 1 >= SGT;
          const int64_t tn = last && t + 1 < L ? t + 1 : t;
          hist_row<K, VJP>(hist, voH_s, (uint32_t)tn * hstep * 4u,
                            last ? 0u : (uint32_t)(i + 1) * TPB * K * 4u, (uint32_t)GS * 4u, pH, pB);
        }
#pragma unroll
        for (int u = 0; u < K; ++u) {
          if constexpr (VJP) {
            // per input j: alpha = e G and q = e (G A - g_t G d), the state's
            // unnormalised tangent with the step's term g_t (c - w_t) = -g_t d
            float al[K], q[K], dd[K];
  #pragma unroll
            for (int j = 0; j < K; ++j) {
              dd[j] = wtl - cbr[i][j][u];
              const float e = ex2(fmaf(-dd[j], dd[j], noff));
              al[j] = e * Gin[j];
              q[j] = e * fmaf(-gG[j], dd[j], Ain[j]);
            }
            const float go = (al[0] + al[1]) + (al[2] + al[3]);   // sum alpha
            const float aout = (q[0] + q[1]) + (q[2] + q[3]);     // G A of the output group
            float sad = al[0] * dd[0], sqd = q[0] * dd[0];        // sum alpha d, sum q d
  #pragma unroll
            for (int j = 1; j < K; ++j) {
              sad = fmaf(al[j], dd[j], sad);
              sqd = fmaf(q[j], dd[j], sqd);
            }
            rv[0] = fmaxf(rv[0], go);
            const float Hu = Hc[u];
            const float bx = fmaf(-xbar, Hu, Bc[u]);              // H (B - xbar)
            rv[1] = fmaf(Hu, sad, rv[1]);
            rv[2] = fmaf(Hu, go, rv[2]);
            rv[3] = fmaf(go, bx, fmaf(Hu, aout, rv[3]));
            rv[4] = fmaf(sad, bx, fmaf(Hu, sqd, rv[4]));
            rot::st_pair_at(sl[u], go, aout);
          } else {
            // soft codeword alone: sum alpha, sum alpha d and the two moments
            float al[K], dd[K];
#pragma unroll
            for (int j = 0; j < K; ++j) {
              dd[j] = wtl - cbr[i][j][u];
              al[j] = ex2(fmaf(-dd[j], dd[j], noff)) * Gin[j];
            }
            const float go = (al[0] + al[1]) + (al[2] + al[3]);
            float sad = al[0] * dd[0];
#pragma unroll
            for (int j = 1; j < K; ++j) sad = fmaf(al[j], dd[j], sad);
            rv[0] = fmaxf(rv[0], go);
            rv[1] = fmaf(Hc[u], sad, rv[1]);
            rv[2] = fmaf(Hc[u], go, rv[2]);
            rot::st_pair_at(sl[u], go, 0.f);
          }
        }
        asm volatile("" ::: "memory");
      }
      red_pre<NRV, 1u>(rv, rc);
      __syncthreads();
      red_post<NRV, 1u>(rv, rc);
      const float r1 = 1.f / rv[2];
      const float md = rv[1] * r1;   // E_p[w' - c'] = w'_t - w_soft'_t
      if (threadIdx.x == 0) {
        if (a.w_soft) a.w_soft[bb * L + t] = (wt - md) * a.inv_kap;
        // dW = Cov_p(X, c') / (kappa^2 T), Cov_p(X, c') = -E[(X - xbar) d] + E[X - xbar] E[d]
        if (VJP && a.dW) a.dW[bb * L + t] = fmaf(rv[VJP ? 3 : 0] * r1, rv[1], -rv[VJP ? 4 : 0]) * r1 * dws;
      }
      // the step's mass sum_s alpha_t beta_t must equal Z
      const float lzt = lg2(rv[2]) - (float)(ex - off) - eHt;
      if (!(fabsf(lzt - lz2) <= 2e-4f)) bad = true;
      if (!(rv[0] >= 0x1p-30f && rv[0] <= 0x1p100f)) bad = true;
      ex -= off;
      off = bad ? 0 : rot::exp_of(rv[0]) - rot::kTopExp;
      // the step's term of A moves from g_t (c - w_t) to g_t (c - w_soft_t)
      // when it is read; E_p[X_{t+1}] = E_p[X_t] - g_t (w_soft_t - w_t)
      if constexpr (VJP) {
        cprev = -gt * md;
        xbar = fmaf(rv[3], r1, xbar) - cprev;
      }
      r2 = r2 == 12u ? 0u : r2 + 2u;
    }
    if (threadIdx.x == 0) a.flags[bb] = bad ? 1 : 0;
    __syncthreads();
  }
}

}  // namespace bcjr
