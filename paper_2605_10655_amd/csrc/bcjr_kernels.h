// bcjr_kernels.h -- gfx950 kernels for the temperature-T BCJR soft codeword
// over a bitshift trellis, its VJP, and the min-sum (Viterbi) decode.
//
// Index algebra (paper Sec. 3.1, next(s, b) = ((s << k) | b) & (S - 1)):
//   n = state bits, K = 2^k, S = 2^n.  Write a state as three digit fields
//       s = (j, sg, u)   j: top k bits, sg: middle n - 2k bits, u: low k bits.
//   The predecessors of s are (i, j, sg_hi...) -- all states whose low n - k
//   bits equal s >> k -- and the successors of s are (s & (S/K - 1)) * K + b.
//   Hence the log forward variable factors as
//       log alpha_t(s) = h_t(s) + G_t(s >> k)            (Eq. alpha, its recursion)
//       G_{t+1}(v)     = LSE_{j<K} log alpha_t(j * S/K + v),   v < S/K
//   and the log backward variable depends only on the low n - k bits:
//       log beta_t(s)  = H_t(s & (S/K - 1))              (Eq. beta, its recursion)
//       H_{t-1}(v)     = LSE_{b<K} [h_t(v*K + b) + H_t((v*K + b) & (S/K - 1))].
//   h_t(s) = -(w_t - c(s))^2 / (2T) is the local field of Eq. boltzmann.
//   The K^2 states (j, sg, u) for a fixed sg form one "super-group": they
//   read G_t(j, sg) (j < K) and produce G_{t+1}(sg, u) (u < K), and read
//   H_t(sg, u) and produce H_{t-1}(j, sg).  One thread owns a fixed set of
//   super-groups for the whole call, so every per-state quantity it
//   accumulates stays in its registers.
//
// All logs here are base 2 (v_exp_f32 / v_log_f32); natural-log results
// are converted at the end.  After every step the new G or H vector is
// shifted by floor(max) so that its largest entry is in [0, 1); the shifts
// are integers, so their sums are exact.
//
// Marginals (Eq. marginal) are formed inside the sweeps:
//   p_t(s) = 2^(log2 alpha + log2 beta - lambda_t),  lambda_t = log2 of the
//   normaliser in the shifted frame, carried from step to step and re-anchored
//   with the exact sum of the step.
//
// VJP (the paper's Sec. 3.5 gives no formula; it follows from Eq. boltzmann).
//   With F = sum_t g_t c(s_t):  dW_tau = Cov(F, c(s_tau)) / T and
//   dc_sig = sum_t p_t(sig)[g_t + (w_t - c_sig)(E[F|s_t=sig] - E[F]) / T].
//   E[F | s_t = s] = g_t c(s) + A_t(s) + B_t(s) with forward / backward
//   tangent recursions that reuse the alpha / beta softmax weights.  Each
//   tangent is kept small by subtracting a per-step constant from every
//   summand (covariances ignore such constants): the backward tangent
//   accumulates g_t (c(s_t) - w_t), the forward one g_t (c(s_t) - w_soft_t),
//   so fp32 keeps their differences accurate.  fb_kernel does two sweeps:
//     S0 backward: H and B (both stored per step);
//     S1 forward:  G, marginals -> w_soft_t, A, and the combine -> dW_t, dc.
//   The soft codeword alone is S0 (H only) + S1 (no tangents).
//   fb_kernel_hp (fp64 log vectors, low temperatures) centres both tangents
//   on w_soft and therefore needs a third sweep.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bcjr_device.h"
#include "bcjr_internal.h"

namespace bcjr {

// ---------------------------------------------------------------------------
// Forward-backward kernel.  One workgroup runs BPW blocks side by side (BPW =
// NT / TPB), each block's group vectors living in LDS (two vectors of S/K
// floats).  The grid is persistent: workgroup x handles blocks
// x*BPW + bw, x*BPW + bw + grid*BPW, ...  Per-step histories go to the
// workgroup's workspace slot.
// ---------------------------------------------------------------------------
// NB > 0 fixes the state bits at compile time (then SGT = SGMAX); NB == 0
// reads them from the arguments.
template <int KB, int NB, int SGMAX, int NT, bool VJP, bool DC>
__global__ void __launch_bounds__(NT) fb_kernel(FbArgs a) {
  constexpr int K = 1 << KB;
  extern __shared__ float lds[];
  const int n = NB ? NB : a.n;
  const int GS = 1 << (n - KB);          // size of a group vector (S / K)
  const int NSG = 1 << (n - 2 * KB);     // super-groups per block
  const int SGT = NB ? SGMAX : a.sgt;    // super-groups per thread (<= SGMAX)
  const int TPB = NSG / SGT;             // threads per block
  const int BPW = NT / TPB;              // blocks per workgroup
  const int tid = threadIdx.x;
  const int bw = BPW == 1 ? 0 : tid / TPB;
  const int tb = BPW == 1 ? tid : tid - bw * TPB;
  const int64_t L = a.L;
  // Emissions use the codebook scaled by kappa = sqrt(log2(e) / (2T)):
  // h_t(s) in log2 units is -(w'_t - c'(s))^2 with w' = kappa w, c' = kappa c.
  // Soft codeword and tangents are carried in scaled units as well.
  const float kap = a.kap;

  RedCtx rc;
  rc.width = TPB < 64 ? TPB : 64;
  rc.rw = TPB > 64 ? TPB / 64 : 1;
  rc.wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: a scalar
  // cross-wave partials, [2 parities][waves][kRed]: a sweep with one barrier
  // per step alternates them, so a fast wave's next partial never overwrites
  // one a slow wave is still reading
  float* const red0 = lds + (size_t)BPW * 2 * GS;
  rc.red = red0;

  // LDS: the block's two group vectors v0 = lds[vb ..), v1 = lds[vb + GS ..).
  // A super-group sg = tb + i*TPB reads / writes two patterns:
  //   column form  v[j*NSG + sg]  = lds[col + j*NSG + i*TPB]
  //   row form     v[sg*K + u]    = lds[row + i*TPB*K + u]
  // col / row (and their +GS twins) are re-pinned every step so the compiler
  // keeps one base register each and folds the rest into the instruction.
  const uint32_t vb = (uint32_t)bw * 2 * GS;
  const uint32_t col0 = vb + tb, row0 = vb + (uint32_t)tb * K;

  // Codebook row j of super-group i: byte offset (j*S/K + i*TPB*K)*4 + tb*K*4.
  const rsrc_t cbk = make_rsrc(a.cs, (uint32_t)4 << n);
  const uint32_t voK = (uint32_t)tb << (KB + 2);
  // Histories: one descriptor per workgroup over its BPW slots; the block's
  // slot and the thread's super-group row go into the per-thread offset.
  const uint32_t hstep = (uint32_t)GS * (VJP ? 2 : 1);   // floats per step
  const uint32_t voH = ((uint32_t)bw * (uint32_t)L * hstep + (uint32_t)tb * K) * 4u;
  const uint32_t voC = ((uint32_t)bw * (uint32_t)L * hstep + (uint32_t)tb) * 4u;
  // w and g of the step: when a block spans whole waves every lane needs the
  // same value, read 64 steps at a time and taken with a lane read
  const bool lane_rows = TPB >= 64;
  constexpr bool PF = true;  // forward-sweep prefetches
  // 512-thread families keep every codebook row of the thread's super-groups
  // in registers for the whole call (the super-groups a thread owns never
  // change): the sweeps then issue no codebook loads, and no wait for one
  // also waits for the history stores ahead of it.
  constexpr bool CBR = NT == 512 && NB != 0;
  const uint32_t wave_s = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave index (SGPR)
  float cbr[CBR ? SGMAX : 1][K][K];
  if constexpr (CBR) {
#pragma unroll
    for (int i = 0; i < SGMAX; ++i) {
#pragma unroll
      for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((i * TPB) << KB)) * 4, cbr[i][j]);
    }
  }

  // repair pass of the soft codeword after the linear-domain kernel (one
  // block per workgroup): only the blocks it marked
  const bool repair = !VJP && BPW == 1 && a.repair;
  if (repair) {
    int any = 0;
    for (int64_t base = blockIdx.x; base < a.B; base += gridDim.x) any |= ld_uniform_i(a.flags, base);
    if (!any) return;
  }

  for (int64_t base = (int64_t)blockIdx.x * BPW; base < a.B; base += (int64_t)gridDim.x * BPW) {
    if (repair && !ld_uniform_i(a.flags, base)) continue;
    const int64_t blk = base + bw;
    const bool valid = blk < a.B;
    const int64_t bb = valid ? blk : a.B - 1;
    const int64_t slot = (int64_t)blockIdx.x * BPW + bw;
    const float* wb = a.w + bb * L;
    const float* gb = VJP ? a.g + bb * L : nullptr;
    // when a block spans whole waves its row pointers are wave-uniform:
    // w_t and g_t are then read with scalar loads, one step ahead
    const int64_t bbu = lane_rows ? (int64_t)__builtin_amdgcn_readfirstlane((int)bb) : 0;
    const float* wbu = a.w + bbu * L;
    const float* gbu = VJP ? a.g + bbu * L : a.w;
    // history of each block: soft codeword alone [L][S/K] (H_t); with the VJP
    // [L][S/K/K][2K] (H_t, B_t of each super-group)
    const int64_t slot0 = (int64_t)blockIdx.x * BPW;
    const rsrc_t hist = make_rsrc(VJP ? a.histHB + slot0 * L * hstep : a.histH + slot0 * L * hstep,
                                  (uint32_t)BPW * (uint32_t)L * hstep * 4u);
    float* sm_mB = a.small + slot * 3 * L;  // shift applied to H_t
    float* sm_lam = sm_mB + L;              // dCodebook: lambda_t
    float* sm_xb = sm_lam + L;              // dCodebook: E_p[X_t]
    const rsrc_t hga = make_rsrc(DC ? a.histGA + slot0 * L * hstep : a.histHB,
                                 DC ? (uint32_t)BPW * (uint32_t)L * hstep * 4u : 0u);

    // ------------------------------------------------------------------ S0
    // Backward sweep.  Soft codeword alone: H only, v0 / v1 alternating as the
    // H_t being read and the H_{t-1} being written (one barrier per step; the
    // shift of H_{t-1}, known after the barrier, is subtracted when it is read
    // back).  With the VJP: H in v0 and the backward tangent B in v1, updated
    // in place (reads, barrier, writes, barrier).  B_t(s) = E[sum_{tau > t}
    // g_tau (c(s_tau) - w_tau) | s_t = s] is centred on the input weights, so
    // it stays O(quantisation error) in size.  Each thread stores the values
    // its super-groups read (H_t, and B_t for the VJP) as the step's history.
    for (int i = tb; i < GS; i += TPB) {
      lds[vb + i] = 0.f;
      if (VJP) lds[vb + GS + i] = 0.f;
    }
    __syncthreads();
    int shiftB = 0;  // sum of the integer shifts of H (exact)
    float lam0 = 0.f;
    float xbar = 0.f;     // VJP: E_p[X_0], see S1
    float offc = 0.f;     // soft codeword alone: shift of the H vector being read
    float wch = 0.f, gch = 0.f;
    int64_t cbase = 0;
    float wnx = lane_rows ? ld_uniform(wbu, L - 1) : 0.f;
    float gnx = lane_rows && VJP ? ld_uniform(gbu, L - 1) : 0.f;
    float q0[K][K];  // codebook rows of the next super-group, fetched one super-group ahead
    if constexpr (!CBR) {
#pragma unroll
      for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, (j << (n - KB)) * 4, q0[j]);
    }
    for (int64_t t = L - 1;; --t) {
      // with the register-resident codebook the per-lane offsets are
      // re-derived every step from a pinned thread index, not held live
      uint32_t tid_s = CBR ? lane_tid(wave_s) : (uint32_t)threadIdx.x;
      const uint32_t col0_s = CBR ? tid_s : col0, row0_s = CBR ? tid_s * K : row0;
      const uint32_t voH_s = CBR ? tid_s * K * 4u : voH;
      const uint32_t vcH = CBR ? tid_s * 4u : voC;
      rc.red = red0 + ((L - 1 - t) & 1) * (NT / 64) * kRed;
      float wt, gt = 0.f;
      if (lane_rows) {
        wt = wnx;
        gt = gnx;
        const int64_t tn = t > 0 ? t - 1 : 0;
        wnx = ld_uniform(wbu, tn);
        if (VJP) gnx = ld_uniform(gbu, tn);
      } else {
        wt = wb[t];
        if (VJP) gt = gb[t];
      }
      wt *= kap;
      // read side: the vector holding H_t (row form); write side: column form
      const bool odd = !VJP && ((L - 1 - t) & 1);
      uint32_t rrow = row0_s + (odd ? GS : 0), rrowB = row0_s + GS;
      uint32_t wcol = col0_s + (odd ? 0 : GS), wcolB = col0_s + GS;
      pin_u(rrow);
      pin_u(wcol);
      if (VJP) {
        pin_u(rrowB);
        wcol = col0_s;
        pin_u(wcol);
        pin_u(wcolB);
      }
      const uint32_t soH = (uint32_t)t * hstep * 4u;
      if (t == 0) {
        // lambda_0 = LSE_s [h_0(s) + H_0(s & (S/K-1))]  (log2 alpha_0 = h_0);
        // with the VJP also E_p[g_0 c(s_0) + B_0(s_0)], the mean of X_0
        float lm = -INFINITY, ls = 0.f, ly = 0.f;
#pragma unroll
        for (int i = 0; i < SGMAX; ++i) {
          if (i < SGT) {
            float Hin[K], Bin[K];  // row form: one 16-byte LDS read per K floats
            ld_vec<K>(lds + rrow + i * TPB * K, Hin);
            if constexpr (VJP) {
              ld_vec<K>(lds + rrowB + i * TPB * K, Bin);
            } else {
#pragma unroll
              for (int b = 0; b < K; ++b) Bin[b] = 0.f;
            }
#pragma unroll
            for (int b = 0; b < K; ++b) Hin[b] -= offc;
            if constexpr (!VJP) buf_st<K, kStream>(hist, voH_s, ((i * TPB) << (KB + 2)), Hin);
#pragma unroll
            for (int j = 0; j < K; ++j) {
              float cc[K];
              if constexpr (CBR) {
#pragma unroll
                for (int b = 0; b < K; ++b) cc[b] = cbr[CBR ? i : 0][j][b];
              } else {
                buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((i * TPB) << KB)) * 4, cc);
              }
              float x[K];
#pragma unroll
              for (int b = 0; b < K; ++b) {
                const float d = wt - cc[b];
                x[b] = fmaf(-d, d, Hin[b]);
              }
              const float m = max_of<K>(x);
              float E[K];
#pragma unroll
              for (int b = 0; b < K; ++b) E[b] = ex2(x[b] - m);
              float s = E[0];
#pragma unroll
              for (int b = 1; b < K; ++b) s += E[b];
              if constexpr (VJP) {
                float sy = E[0] * fmaf(gt, cc[0], Bin[0]);
#pragma unroll
                for (int b = 1; b < K; ++b) sy = fmaf(E[b], fmaf(gt, cc[b], Bin[b]), sy);
                lse3_pair(lm, ls, ly, m, s, sy);
              } else {
                lse_pair(lm, ls, m, s);
              }
            }
            sg_fence();
          }
        }
        if constexpr (VJP) {
          lse3_pre(lm, ls, ly, rc);
        } else {
          lse_pre(lm, ls, rc);
        }
        if (tb == 0) sm_mB[L - 1] = 0.f;
        __syncthreads();
        if constexpr (VJP) {
          lse3_post(lm, ls, ly, rc);
          xbar = ly / ls;
        } else {
          lse_post(lm, ls, rc);
        }
        lam0 = lm + lg2(ls);
        if (tb == 0 && valid && a.logZ)
          a.logZ[bb] = (float)(((double)shiftB + (double)lam0) * 0.69314718055994530942);
        __syncthreads();
        break;
      }
      float Hout[VJP ? SGMAX : 1][K], Bout[VJP ? SGMAX : 1][K];
      float vmax[1] = {-INFINITY};
#pragma unroll
      for (int i = 0; i < SGMAX; ++i) {
        if (i < SGT) {
          // this super-group's codebook rows were fetched one super-group
          // ahead; fetch the next one's (the first of the next step after the last)
          float cc[K][K];
#pragma unroll
          for (int j = 0; j < K; ++j) {
#pragma unroll
            for (int u = 0; u < K; ++u) cc[j][u] = CBR ? cbr[CBR ? i : 0][j][u] : q0[j][u];
          }
          if constexpr (!CBR) {
            const int inx = i + 1 < SGT ? i + 1 : 0;
#pragma unroll
            for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((inx * TPB) << KB)) * 4, q0[j]);
          }
          float Hin[K], Bin[K];  // row form: one 16-byte LDS read per K floats
          ld_vec<K>(lds + rrow + i * TPB * K, Hin);
          if constexpr (VJP) {
            ld_vec<K>(lds + rrowB + i * TPB * K, Bin);
          } else {
#pragma unroll
            for (int b = 0; b < K; ++b) Bin[b] = 0.f;
          }
#pragma unroll
          for (int b = 0; b < K; ++b) Hin[b] -= offc;
          if constexpr (!VJP) buf_st<K, kStream>(hist, voH_s, soH + ((i * TPB) << (KB + 2)), Hin);
#pragma unroll
          for (int j = 0; j < K; ++j) {
            float x[K], d[K];
#pragma unroll
            for (int b = 0; b < K; ++b) {
              d[b] = wt - cc[j][b];
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
            if constexpr (VJP) {
              // B_{t-1} = E-weighted mean of g_t (c - w_t) + B_t over the K successors
              float num = E[0] * fmaf(-gt, d[0], Bin[0]);
#pragma unroll
              for (int b = 1; b < K; ++b) num = fmaf(E[b], fmaf(-gt, d[b], Bin[b]), num);
              Hout[i][j] = h;
              pin(Hout[i][j]);
              Bout[i][j] = num * rcp(s);
              pin(Bout[i][j]);
            } else {
              lds[wcol + j * NSG + i * TPB] = h;
            }
          }
          sg_fence();
        }
      }
      red_pre<1, 1u>(vmax, rc);
      __syncthreads();
      red_post<1, 1u>(vmax, rc);
      const float off = floorf(vmax[0]);
      // (wave-uniform when a block spans whole waves; per lane otherwise)
      shiftB += lane_rows ? __builtin_amdgcn_readfirstlane((int)off) : (int)off;
      if (tb == 0) sm_mB[t - 1] = off;
      if constexpr (VJP) {
        // The exchange writes, and with them the history entries of step
        // t - 1 (the values the next step reads), one dword per lane at group
        // j NSG + i TPB + tb: stored here, where the VALU waits on the LDS
        // writes anyway, rather than as rows in the arithmetic phase.  (The
        // entries of step L - 1 are zero and are filled before the launch.)
#pragma unroll
        for (int i = 0; i < SGMAX; ++i) {
          if (i < SGT) {
#pragma unroll
            for (int j = 0; j < K; ++j) {
              const float hv[1] = {Hout[i][j] - off}, bv[1] = {Bout[i][j]};
              lds[wcol + j * NSG + i * TPB] = hv[0];
              lds[wcolB + j * NSG + i * TPB] = bv[0];
              const uint32_t so = soH - hstep * 4u + (uint32_t)(j * NSG + i * TPB) * 4u;
              buf_st<1, kStream>(hist, vcH, so, hv);
              buf_st<1, kStream>(hist, vcH, so + (uint32_t)GS * 4u, bv);
            }
          }
        }
        __syncthreads();
      } else {
        offc = off;
      }
    }

    // ------------------------------------------------------------------ S1
    // Forward sweep: G (and the forward tangent A) in v0 (v1), in place: all
    // reads, barrier, writes, barrier; outputs are held in registers across
    // the first barrier.  For each output group the K-way LSE gives G_{t+1};
    // its softmax weights E_j times one exponential 2^(m + H_t - lambda_t) are
    // the marginals p_t of the group's K states.  With the VJP:
    //   A_t(s) = E[sum_{tau < t} g_tau (c(s_tau) - w_soft_tau) | s_t = s]
    //   (centred on the soft codeword at write time),
    //   X_t(s) = g_t c(s) + A_t(s) + B_t(s) - xbar_t = E[F | s_t = s] - const,
    // where xbar_t predicts E_p[X_t] (exact at t = 0 from S0, then carried by
    // the known change of the centring constants and re-anchored each step),
    // so that dW_t = (sum p c X - w_soft_t sum p X) / (T sum p) and the
    // dCodebook summands p (g + (w - c) X / T) see a nearly centred X.  In
    // the scaled units used here c, w_soft and X carry a factor kappa, hence
    // the 1 / (kappa^2 T) of both formulas.
    for (int i = tb; i < GS; i += TPB) {
      lds[vb + i] = 0.f;
      if (VJP) lds[vb + GS + i] = 0.f;
    }
    __syncthreads();
    rc.red = red0;
    const float dws = a.dws;  // 1 / (kappa^2 T): scaled covariances -> dW, dCodebook
    float lam_est = lam0;
    // The history row of the next super-group is loaded one super-group
    // ahead (the last super-group of a step fetches the first of the next
    // step, so that HBM read is in flight across the barriers).
    float pH[K], pB[K];
    float p0[K][K];  // codebook rows of the next super-group, fetched one super-group ahead
    wnx = lane_rows ? ld_uniform(wbu, 0) : 0.f;
    gnx = lane_rows && VJP ? ld_uniform(gbu, 0) : 0.f;
    if constexpr (PF) {
      hist_row<K, VJP>(hist, voH, 0, 0, (uint32_t)GS * 4u, pH, pB);
      if constexpr (!CBR) {
#pragma unroll
        for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, (j << (n - KB)) * 4, p0[j]);
      }
    }
    for (int64_t t = 0; t < L; ++t) {
      // with the register-resident codebook the per-lane offsets are
      // re-derived every step from a pinned thread index, not held live
      uint32_t tid_s = CBR ? lane_tid(wave_s) : (uint32_t)threadIdx.x;
      const uint32_t col0_s = CBR ? tid_s : col0, row0_s = CBR ? tid_s * K : row0;
      const uint32_t voH_s = CBR ? tid_s * K * 4u : voH;
      float wt, gt = 0.f;
      if (lane_rows) {
        wt = wnx;
        gt = gnx;
        const int64_t tn = t + 1 < L ? t + 1 : t;
        wnx = ld_uniform(wbu, tn);
        if (VJP) gnx = ld_uniform(gbu, tn);
      } else {
        wt = wb[t];
        if (VJP) gt = gb[t];
      }
      wt *= kap;
      if (VJP && t > 0) xbar = fmaf(gt, wt, xbar);  // B_t no longer holds step t
      const float mBt = sm_mB[t];
      uint32_t rcol = col0_s, rcolA = col0_s + GS, wrow = row0_s, wrowA = row0_s + GS;
      pin_u(rcol);
      pin_u(wrow);
      if (VJP) {
        pin_u(rcolA);
        pin_u(wrowA);
      }
      float Gout[SGMAX][K];
      float Aout[VJP ? SGMAX : 1][K];
      // max G_{t+1}, sum p, sum p c, and with the VJP sum p X, sum p c X
      float rv[VJP ? 5 : 3];
      rv[0] = -INFINITY;
#pragma unroll
      for (int q = 1; q < (VJP ? 5 : 3); ++q) rv[q] = 0.f;
#pragma unroll
      for (int i = 0; i < SGMAX; ++i) {
        if (i < SGT) {
          float Gin[K], Ain[K];
#pragma unroll
          for (int j = 0; j < K; ++j) {
            Gin[j] = lds[rcol + j * NSG + i * TPB];
            Ain[j] = VJP ? lds[rcolA + j * NSG + i * TPB] : 0.f;
          }
          float Hc[K], Bc[K], cc[K][K];
          if constexpr (PF) {
#pragma unroll
            for (int u = 0; u < K; ++u) {
              Hc[u] = pH[u];
              Bc[u] = VJP ? pB[u] : 0.f;
            }
          } else {
            hist_row<K, VJP>(hist, voH_s, (uint32_t)t * hstep * 4u, (uint32_t)i * TPB * K * 4u,
                             (uint32_t)GS * 4u, Hc, Bc);
          }
          if constexpr (PF) {
#pragma unroll
            for (int j = 0; j < K; ++j) {
#pragma unroll
              for (int u = 0; u < K; ++u) cc[j][u] = CBR ? cbr[CBR ? i : 0][j][u] : p0[j][u];
            }
          } else {
#pragma unroll
            for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((i * TPB) << KB)) * 4, cc[j]);
          }
          if constexpr (PF) {
            if constexpr (!CBR) {  // the next super-group's codebook rows (the first of the next step after the last)
              const int inx = i + 1 < SGT ? i + 1 : 0;
#pragma unroll
              for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((inx * TPB) << KB)) * 4, p0[j]);
            }
            // (a select, not a branch: at t = L - 1 it re-reads row t, unused)
            const bool last = i + 1 >= SGT;
            const int64_t tn = last && t + 1 < L ? t + 1 : t;
            hist_row<K, VJP>(hist, voH_s, (uint32_t)tn * hstep * 4u,
                             last ? 0u : (uint32_t)(i + 1) * TPB * K * 4u, (uint32_t)GS * 4u,
                             pH, pB);
          }
#pragma unroll
          for (int u = 0; u < K; ++u) {
            float al[K];
#pragma unroll
            for (int j = 0; j < K; ++j) {
              const float d = wt - cc[j][u];
              al[j] = fmaf(-d, d, Gin[j]);
            }
            const float m = max_of<K>(al);
            float E[K];
#pragma unroll
            for (int j = 0; j < K; ++j) E[j] = ex2(al[j] - m);
            float s = E[0], ec = E[0] * cc[0][u], sc = ec;
            float y = 0.f, sy = 0.f, scy = 0.f;
            if constexpr (VJP) {
              y = fmaf(gt, cc[0][u], Ain[0]);
              sy = E[0] * y;
              scy = ec * y;
            }
#pragma unroll
            for (int j = 1; j < K; ++j) {
              s += E[j];
              ec = E[j] * cc[j][u];
              sc += ec;
              if constexpr (VJP) {
                y = fmaf(gt, cc[j][u], Ain[j]);
                sy = fmaf(E[j], y, sy);
                scy = fmaf(ec, y, scy);
              }
            }
            Gout[i][u] = m + lg2(s);
            pin(Gout[i][u]);
            rv[0] = fmaxf(rv[0], Gout[i][u]);
            const float fac = ex2(m + Hc[u] - lam_est);
            rv[1] = fmaf(fac, s, rv[1]);
            rv[2] = fmaf(fac, sc, rv[2]);
            if constexpr (VJP) {
              // X = y_j + bx over the group's states, bx = B_t - xbar
              const float bx = Bc[u] - xbar;
              rv[3] = fmaf(fac, fmaf(s, bx, sy), rv[3]);
              rv[4] = fmaf(fac, fmaf(sc, bx, scy), rv[4]);
              Aout[i][u] = sy * rcp(s);
              pin(Aout[i][u]);
            }
            __builtin_amdgcn_sched_barrier(0);  // one output group at a time
          }
          sg_fence();
        }
      }
      red_pre<VJP ? 5 : 3, 1u>(rv, rc);
      __syncthreads();
      red_post<VJP ? 5 : 3, 1u>(rv, rc);
      const float off = floorf(rv[0]);
      const float r1 = 1.f / rv[1];
      const float wst = rv[2] * r1;
      const float lamt = lam_est + lg2(rv[1]);
      if (t < L - 1) {
#pragma unroll
        for (int i = 0; i < SGMAX; ++i) {
          if (i < SGT) {
            float go[K];
#pragma unroll
            for (int u = 0; u < K; ++u) go[u] = Gout[i][u] - off;
            st_vec<K>(lds + wrow + i * TPB * K, go);
            if constexpr (VJP) {
              float ao[K];
#pragma unroll
              for (int u = 0; u < K; ++u) ao[u] = fmaf(-gt, wst, Aout[i][u]);
              st_vec<K>(lds + wrowA + i * TPB * K, ao);
              if constexpr (DC) {  // (G, A) entries of step t + 1 for the dCodebook sweep
                const uint32_t so = (uint32_t)(t + 1) * hstep * 4u + (uint32_t)i * TPB * K * 4u;
                buf_st<K, kStream>(hga, voH_s, so, go);
                buf_st<K, kStream>(hga, voH_s, so + (uint32_t)GS * 4u, ao);
              }
            }
          }
        }
      }
      if (DC && tb == 0) {
        sm_lam[t] = lamt;
        sm_xb[t] = fmaf(rv[VJP ? 3 : 0], r1, xbar);
      }
      if (tb == 0 && valid) {
        if (a.w_soft) a.w_soft[bb * L + t] = wst * a.inv_kap;
        if (VJP && a.dW) a.dW[bb * L + t] = (rv[VJP ? 4 : 0] - wst * rv[VJP ? 3 : 0]) * r1 * dws;
      }
      lam_est = lamt - off + mBt;
      // E_p[X_t] = xbar + sum p X / sum p; X_{t+1} drops g_t w_soft_t (A is
      // centred); it gains g_{t+1} w_{t+1} at the top of the next step
      if (VJP) xbar = fmaf(rv[VJP ? 3 : 0], r1, xbar) - gt * wst;
      __syncthreads();
    }

    // ------------------------------------------------------------------ S2
    // dCodebook: dc(s) = sum_t p_t(s) [g_t + (w_t - c(s)) (X_t(s) - E_p[X_t]) / T].
    // No recursion is left, so each thread runs super-group by super-group
    // over all steps with 16 accumulators: p_t(s) = 2^(G_t + h_t + H_t -
    // lambda_t) per state from the (G, A) and (H, B) histories, with the exact
    // lambda_t and E_p[X_t] recorded by S1.  The (G, A) entries of a
  // super-group are K dwords a column apart (S1 stored them as rows of the
  // next step's outputs), the (H, B) entries one 16-byte row.
    if constexpr (DC) {
      __syncthreads();  // S1's per-step scalars
      const bool first = base == (int64_t)blockIdx.x * BPW;
      double* part = a.dc_part + slot * ((int64_t)1 << n);
#pragma unroll 1
      for (int i = 0; i < SGT; ++i) {
        float cc[K][K], acc[K][K];
#pragma unroll
        for (int j = 0; j < K; ++j) {
          buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((i * TPB) << KB)) * 4, cc[j]);
#pragma unroll
          for (int u = 0; u < K; ++u) acc[j][u] = 0.f;
        }
        float lch = 0.f, xch = 0.f;
        // the four history rows of a step, loaded one step ahead
        float nH[K], nB[K], nG[K], nA[K];
        {
          const uint32_t sh = (uint32_t)i * TPB * K * 4u;
          buf_ld<K, kStream>(hist, voH, sh, nH);
          buf_ld<K, kStream>(hist, voH, sh + (uint32_t)GS * 4u, nB);
#pragma unroll
          for (int j = 0; j < K; ++j) {
            float g1[1], a1[1];
            buf_ld<1, kStream>(hga, voC, (uint32_t)(j * NSG + i * TPB) * 4u, g1);
            buf_ld<1, kStream>(hga, voC, (uint32_t)(j * NSG + i * TPB) * 4u + (uint32_t)GS * 4u, a1);
            nG[j] = g1[0];
            nA[j] = a1[0];
          }
        }
#pragma unroll 1
        for (int64_t t = 0; t < L; ++t) {
          float wt, gt, lt, xt;
          if (lane_rows) {
            if ((t & 63) == 0) {
              cbase = t;
              wch = row_chunk(wb, cbase, L);
              gch = row_chunk(gb, cbase, L);
              lch = row_chunk(sm_lam, cbase, L);
              xch = row_chunk(sm_xb, cbase, L);
            }
            const int ln = (int)(t - cbase);
            wt = read_lane(wch, ln);
            gt = read_lane(gch, ln);
            lt = read_lane(lch, ln);
            xt = read_lane(xch, ln);
          } else {
            wt = wb[t];
            gt = gb[t];
            lt = sm_lam[t];
            xt = sm_xb[t];
          }
          wt *= kap;
          float H[K], Bv[K], G[K], A[K];
#pragma unroll
          for (int q = 0; q < K; ++q) {
            H[q] = nH[q];
            Bv[q] = nB[q];
            G[q] = nG[q];
            A[q] = nA[q];
          }
          {  // (a select, not a branch: the last step re-reads its own rows)
            const int64_t tn = t + 1 < L ? t + 1 : t;
            const uint32_t sh = (uint32_t)tn * hstep * 4u + (uint32_t)i * TPB * K * 4u;
            buf_ld<K, kStream>(hist, voH, sh, nH);
            buf_ld<K, kStream>(hist, voH, sh + (uint32_t)GS * 4u, nB);
#pragma unroll
            for (int j = 0; j < K; ++j) {
              float g1[1], a1[1];
              const uint32_t sg = (uint32_t)tn * hstep * 4u + (uint32_t)(j * NSG + i * TPB) * 4u;
              buf_ld<1, kStream>(hga, voC, sg, g1);
              buf_ld<1, kStream>(hga, voC, sg + (uint32_t)GS * 4u, a1);
              nG[j] = g1[0];
              nA[j] = a1[0];
            }
          }
#pragma unroll
          for (int u = 0; u < K; ++u) {
            const float hb = H[u] - lt, bx = Bv[u] - xt;
#pragma unroll
            for (int j = 0; j < K; ++j) {
              const float d = wt - cc[j][u];
              const float p = ex2(fmaf(-d, d, G[j]) + hb);
              const float X = fmaf(gt, cc[j][u], A[j]) + bx;
              acc[j][u] = fmaf(p, fmaf(d * X, dws, gt), acc[j][u]);
            }
          }
        }
        if (valid) {
#pragma unroll
          for (int j = 0; j < K; ++j) {
            double* pj = part + ((int64_t)j << (n - KB)) + ((i * TPB) << KB) + ((uint32_t)tb << KB);
#pragma unroll
            for (int u = 0; u < K; ++u) pj[u] = first ? (double)acc[j][u] : pj[u] + (double)acc[j][u];
          }
        }
      }
    }

  }
}

// ---------------------------------------------------------------------------
// Low-temperature VJP kernel.  At small T the log-domain values of the states
// that carry the posterior lie hundreds of log2 units from the per-step
// maximum (|h_t| ~ (w - c)^2 / 2T), so fp32 log vectors round them at ~1e-5
// and the VJP loses its 1e-4 relative accuracy.  Here G and H are carried as
// pairs hi + lo (an fp32 word and an 8-bit correction: 32 significand bits)
// with fp64 LSE arithmetic; softmax weights and tangents stay fp32.
//   Exchange between threads: per block, the hi words and the fp32 tangent
//   fill two S/K vectors in LDS and the lo words a third of S/K bytes, each
//   lo an int8 multiple of ulp(hi) / 256 (a 32-bit significand in all); all
//   three are updated in place: reads, barrier, writes, barrier, with the
//   outputs held in registers across the first barrier.  The integer shift
//   of a step is the floor of the previous step's maximum (the stored maxima
//   stay within the per-step drift of 0), and the forward tangent is centred
//   on w_soft when it is read, one step later (the same arithmetic as
//   centring before the write).  The backward tangent is centred on a
//   reference path given per block (the minimum-distortion codewords), which
//   the posterior follows at low temperature.
//   S0 backward: H and B, history rows (H hi, B, H lo) as three planes of
//                [threads][K] per super-group (9 bytes per group-step),
//                written and read non-temporal;
//   S1 forward:  G and A, marginals, w_soft, dW; with dCodebook also the
//                (G hi, A, G lo) entries of the next step, stored from the
//                write phase, and the exact lambda_t, E_p[X_t];
//   S2 dCodebook as in fb_kernel, with p from the fp64 sums.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void lse_pair_d(double& m, float& s, double mo, float so) {
  const double M = fmax(m, mo);
  s = s * ex2((float)(m - M)) + so * ex2((float)(mo - M));
  m = M;
}

__device__ __forceinline__ void lse3_pair_d(double& m, float& s, float& y, double mo, float so,
                                            float yo) {
  const double M = fmax(m, mo);
  const float f = ex2((float)(m - M)), fo = ex2((float)(mo - M));
  s = s * f + so * fo;
  y = y * f + yo * fo;
  m = M;
}

// (max, sum, weighted sum) over the block with a double max; redd holds
// [waves] doubles, r.red the floats
__device__ __forceinline__ void lse3d_pre(double& m, float& s, float& y, const RedCtx& r, double* redd) {
  for (int off = 1; off < r.width; off <<= 1) {
    const double mo = __shfl_xor(m, off);
    const float so = __shfl_xor(s, off);
    const float yo = __shfl_xor(y, off);
    lse3_pair_d(m, s, y, mo, so, yo);
  }
  if (r.rw > 1 && lane_id() == 0) {
    redd[r.wave] = m;
    r.red[r.wave * kRed + 0] = s;
    r.red[r.wave * kRed + 1] = y;
  }
}

__device__ __forceinline__ void lse3d_post(double& m, float& s, float& y, const RedCtx& r,
                                           const double* redd) {
  if (r.rw > 1) {
    const int first = (r.wave / r.rw) * r.rw;
    m = redd[first];
    s = r.red[first * kRed + 0];
    y = r.red[first * kRed + 1];
    for (int i = 1; i < r.rw; ++i)
      lse3_pair_d(m, s, y, redd[first + i], r.red[(first + i) * kRed + 0], r.red[(first + i) * kRed + 1]);
  }
}

__device__ __forceinline__ void split_df(double v, float& hi, float& lo) {
  hi = (float)v;
  lo = (float)(v - (double)hi);
}

// The lo word of a double-float pair, kept as a signed 8-bit multiple of
// ulp(hi) / 256: hi + lo then carries a 32-bit significand, 2^8 times finer
// than hi alone (the VJP's tolerance needs about 2^5), in a quarter of the
// bytes.  hi = 0, denormal or non-finite keeps lo = 0.
__device__ __forceinline__ uint32_t lo8_enc(float hi, float lo) {
  const int e = (int)((as_u(hi) >> 23) & 0xFFu);
  const float q = fminf(fmaxf(rintf(ldexpf(lo, 158 - e)), -127.f), 127.f);
  return (e == 0 || e == 255) ? 0u : ((uint32_t)(int)q & 0xFFu);
}

__device__ __forceinline__ double df_join(float hi, uint32_t byte) {
  const int e = (int)((as_u(hi) >> 23) & 0xFFu);
  const int q = (int)(int8_t)(uint8_t)byte;  // 0 where the encoder keeps lo = 0
  return (double)hi + (double)ldexpf((float)q, e - 158);
}

// K lo bytes of one row, packed (byte u of the row in bits 8u..8u+7)
template <int K>
__device__ __forceinline__ uint64_t lo_row_lds(const uint8_t* p) {
  if constexpr (K == 2) return *reinterpret_cast<const uint16_t*>(p);
  else if constexpr (K == 4) return *reinterpret_cast<const uint32_t*>(p);
  else return *reinterpret_cast<const uint64_t*>(p);
}

template <int K>
__device__ __forceinline__ void lo_row_lds_st(uint8_t* p, uint64_t v) {
  if constexpr (K == 2) *reinterpret_cast<uint16_t*>(p) = (uint16_t)v;
  else if constexpr (K == 4) *reinterpret_cast<uint32_t*>(p) = (uint32_t)v;
  else *reinterpret_cast<uint64_t*>(p) = v;
}

template <int K, int CP = 0>
__device__ __forceinline__ uint64_t lo_row_ld(rsrc_t r, uint32_t voff, uint32_t soff) {
  if constexpr (K == 2) {
    return (uint64_t)(unsigned short)__builtin_amdgcn_raw_buffer_load_b16(r, (int)voff, (int)soff, CP);
  } else if constexpr (K == 4) {
    return (uint64_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, CP);
  } else {
    const u32x2 x = __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, (int)soff, CP);
    const unsigned x0 = x.x, x1 = x.y;
    return (uint64_t)x0 | ((uint64_t)x1 << 32);
  }
}

// (whole offset in the VGPR, as for buf_st)
template <int K, int CP = 0>
__device__ __forceinline__ void lo_row_st(rsrc_t r, uint32_t voff0, uint32_t soff0, uint64_t v) {
  const uint32_t voff = voff0 + soff0;
  if constexpr (K == 2) {
    __builtin_amdgcn_raw_buffer_store_b16((unsigned short)v, r, (int)voff, 0, CP);
  } else if constexpr (K == 4) {
    __builtin_amdgcn_raw_buffer_store_b32((uint32_t)v, r, (int)voff, 0, CP);
  } else {
    const u32x2 x = {(unsigned)v, (unsigned)(v >> 32)};
    __builtin_amdgcn_raw_buffer_store_b64(x, r, (int)voff, 0, CP);
  }
}

__device__ __forceinline__ uint32_t lo_byte_ld(rsrc_t r, uint32_t voff, uint32_t soff) {
  return (uint32_t)(unsigned char)__builtin_amdgcn_raw_buffer_load_b8(r, (int)voff, (int)soff, kStream);
}

template <int KB, int NB, int SGMAX, int NT, bool DC>
__global__ void __launch_bounds__(NT) fb_kernel_hp(FbArgs a) {
  constexpr int K = 1 << KB;
  extern __shared__ float lds[];
  const int n = NB ? NB : a.n;
  const int GS = 1 << (n - KB);
  const int NSG = 1 << (n - 2 * KB);
  const int SGT = NB ? SGMAX : a.sgt;
  const int TPB = NSG / SGT;
  const int BPW = NT / TPB;
  const int tid = threadIdx.x;
  const int bw = BPW == 1 ? 0 : tid / TPB;
  const int tb = BPW == 1 ? tid : tid - bw * TPB;
  const int64_t L = a.L;
  const double k2 = a.k2d;
  const float invT = a.invT;

  RedCtx rc;
  rc.width = TPB < 64 ? TPB : 64;
  rc.rw = TPB > 64 ? TPB / 64 : 1;
  rc.wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: a scalar
  // LDS: per block [hi: S/K][tangent: S/K] floats, then per block [lo: S/K]
  // bytes, then [2 parities][waves][kRed] floats and [waves] doubles
  uint8_t* const lo8 = reinterpret_cast<uint8_t*>(lds + (size_t)BPW * 2 * GS);
  float* red0 = reinterpret_cast<float*>(lo8 + (((size_t)BPW * GS + 15) & ~(size_t)15));
  double* redd = reinterpret_cast<double*>(red0 + 2 * (NT / 64) * kRed);

  const uint32_t vb = (uint32_t)bw * 2 * GS;
  const uint32_t col0 = vb + tb, row0 = vb + (uint32_t)tb * K;     // float planes
  const uint32_t lcol0 = (uint32_t)bw * GS + tb, lrow0 = (uint32_t)bw * GS + (uint32_t)tb * K;  // lo bytes
  const rsrc_t cbk = make_rsrc(a.c, (uint32_t)4 << n);
  const uint32_t voK = (uint32_t)tb << (KB + 2);
  // History step (bytes): H side, per super-group block of TPB*K entries, a
  // hi plane, a tangent plane ([threads][K] floats each) and a lo plane
  // ([threads][K] bytes); G side (dCodebook) three per-step vectors [S/K]
  // (hi floats, tangent floats, lo bytes).
  const uint32_t hstep = ((uint32_t)GS * 9u + 15u) & ~15u;
  const uint32_t sgb = (uint32_t)TPB * K * 9u;          // bytes of one super-group block
  const uint32_t pT = (uint32_t)TPB * K * 4u, pL = (uint32_t)TPB * K * 8u;  // plane offsets in a block
  const uint32_t vslot = (uint32_t)bw * (uint32_t)L * hstep;
  const uint32_t voH = vslot + (uint32_t)tb * K * 4u, voHL = vslot + (uint32_t)tb * K;
  const uint32_t voC = vslot + (uint32_t)tb * 4u, voCL = vslot + (uint32_t)tb;
  const uint32_t gT = (uint32_t)GS * 4u, gL = (uint32_t)GS * 8u;  // G-side vector offsets
  const bool lane_rows = TPB >= 64;
  // repair pass after the linear-domain kernel (one block per workgroup):
  // only the blocks it marked
  const bool repair = BPW == 1 && a.repair;
  if (repair) {
    int any = 0;
    for (int64_t base = blockIdx.x; base < a.B; base += gridDim.x) any |= ld_uniform_i(a.flags, base);
    if (!any) return;
  }

  for (int64_t base = (int64_t)blockIdx.x * BPW; base < a.B; base += (int64_t)gridDim.x * BPW) {
    if (repair && !ld_uniform_i(a.flags, base)) continue;
    const int64_t blk = base + bw;
    const bool valid = blk < a.B;
    const int64_t bb = valid ? blk : a.B - 1;
    const int64_t slot = (int64_t)blockIdx.x * BPW + bw;
    const int64_t slot0 = (int64_t)blockIdx.x * BPW;
    const float* wb = a.w + bb * L;
    const float* gb = a.g + bb * L;
    const float* rb = a.bref + bb * L;
    // when a block spans whole waves its rows are wave-uniform: w_t, g_t
    // and the reference are read with scalar loads, one step ahead
    const int64_t bbu = lane_rows ? (int64_t)__builtin_amdgcn_readfirstlane((int)bb) : 0;
    const float* wbu = a.w + bbu * L;
    const float* gbu = a.g + bbu * L;
    const float* rbu = a.bref + bbu * L;
    char* const hbase = reinterpret_cast<char*>(a.histHB) + slot0 * L * (int64_t)hstep;
    const rsrc_t hist = make_rsrc(hbase, (uint32_t)BPW * (uint32_t)L * hstep);
    const rsrc_t hga = make_rsrc(DC ? reinterpret_cast<char*>(a.histGA) + slot0 * L * (int64_t)hstep
                                    : reinterpret_cast<char*>(a.histHB),
                                 DC ? (uint32_t)BPW * (uint32_t)L * hstep : 0u);
    float* sm_mB = a.small + slot * 4 * L;   // shift applied to H_t (integer)
    float* sm_xb = sm_mB + L;                // dCodebook: E_p[X_t]
    double* sm_lam = reinterpret_cast<double*>(sm_xb + L);  // dCodebook: lambda_t (fp64)

    // ------------------------------------------------------------------ S0
    // H (hi in LDS plane 0, lo bytes) and the tangent B (plane 1), updated in
    // place: reads, barrier, writes, barrier
    for (int i = tb; i < GS; i += TPB) {
      lds[vb + i] = 0.f;
      lds[vb + GS + i] = 0.f;
      lo8[(uint32_t)bw * GS + i] = 0;
    }
    __syncthreads();
    double shiftB = 0.0;
    double lam0 = 0.0;
    float xbar = 0.f;
    float dlag = 0.f;   // shift applied to the values written this step
    float wch = 0.f, gch = 0.f;
    int64_t cbase = 0;
    float wnx = lane_rows ? ld_uniform(wbu, L - 1) : 0.f;
    float gnx = lane_rows ? ld_uniform(gbu, L - 1) : 0.f;
    float rnx = lane_rows ? ld_uniform(rbu, L - 1) : 0.f;
    // codebook rows of the next super-group, fetched one super-group ahead
    float pc[K][K];
#pragma unroll
    for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, (j << (n - KB)) * 4, pc[j]);
    for (int64_t t = L - 1;; --t) {
      const int par = (int)((L - 1 - t) & 1);
      rc.red = red0 + par * (NT / 64) * kRed;
      float wf, gt, rt;
      if (lane_rows) {
        wf = wnx;
        gt = gnx;
        rt = rnx;
        const int64_t tn = t > 0 ? t - 1 : 0;
        wnx = ld_uniform(wbu, tn);
        gnx = ld_uniform(gbu, tn);
        rnx = ld_uniform(rbu, tn);
      } else {
        wf = wb[t];
        gt = gb[t];
        rt = rb[t];
      }
      const double wt = (double)wf;
      // h_t(s) + H = k2 c (2 w - c) + H - k2 w^2: the state's part in two
      // FMAs, the step's k2 w^2 taken out once with the shift
      const double k2w2 = 2.0 * k2 * wt;
      const double hoff = k2 * wt * wt;
      uint32_t rrow = row0, rrowT = row0 + GS, wcol = col0, wcolT = col0 + GS;
      uint32_t lrow = lrow0, lcol = lcol0;
      pin_u(rrow);
      pin_u(rrowT);
      pin_u(wcol);
      pin_u(wcolT);
      const uint32_t soH = (uint32_t)t * hstep;
      if (t == 0) {
        // lambda_0 = LSE_s [h_0(s) + H_0] and E_p[g_0 c + B_0]
        double lm = -INFINITY;
        float ls = 0.f, ly = 0.f;
#pragma unroll 1
        for (int i = 0; i < SGT; ++i) {
          float Hh[K], Bin[K];
          ld_vec<K>(lds + rrow + i * TPB * K, Hh);
          ld_vec<K>(lds + rrowT + i * TPB * K, Bin);
          const uint64_t Hl = lo_row_lds<K>(lo8 + lrow + i * TPB * K);
          buf_st<K, kStream>(hist, voH, soH + (uint32_t)i * sgb, Hh);
          buf_st<K, kStream>(hist, voH, soH + (uint32_t)i * sgb + pT, Bin);
          lo_row_st<K, kStream>(hist, voHL, soH + (uint32_t)i * sgb + pL, Hl);
#pragma unroll
          for (int j = 0; j < K; ++j) {
            float cc[K];
            buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((i * TPB) << KB)) * 4, cc);
            double x[K];
#pragma unroll
            for (int b = 0; b < K; ++b) {
              const double d = wt - (double)cc[b];
              x[b] = fma(-d * k2, d, df_join(Hh[b], (uint32_t)(Hl >> (8 * b))));
            }
            const double m = max_of<K>(x);
            float s = 0.f, sy = 0.f;
#pragma unroll
            for (int b = 0; b < K; ++b) {
              const float E = ex2((float)(x[b] - m));
              s += E;
              sy = fmaf(E, fmaf(gt, cc[b], Bin[b]), sy);
            }
            lse3_pair_d(lm, ls, ly, m, s, sy);
          }
        }
        lse3d_pre(lm, ls, ly, rc, redd);
        if (tb == 0) sm_mB[L - 1] = 0.f;
        __syncthreads();
        lse3d_post(lm, ls, ly, rc, redd);
        xbar = ly / ls;
        lam0 = lm + (double)lg2(ls);
        if (tb == 0 && valid && a.logZ)
          a.logZ[bb] = (float)((shiftB + lam0) * 0.69314718055994530942);
        __syncthreads();
        break;
      }
      float vmax[1] = {-INFINITY};
      float oh[SGMAX][K], ot[SGMAX][K];  // outputs, held across the first barrier
      uint64_t ol[SGMAX];                // their lo bytes, packed
#pragma unroll
      for (int i = 0; i < SGMAX; ++i) {
        if (i < SGT) {
          float Hh[K], Bin[K], cc[K][K];
#pragma unroll
          for (int j = 0; j < K; ++j) {
#pragma unroll
            for (int u = 0; u < K; ++u) cc[j][u] = pc[j][u];
          }
          {  // the codebook wraps to the next step
            const int ic = i + 1 < SGT ? i + 1 : 0;
#pragma unroll
            for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((ic * TPB) << KB)) * 4, pc[j]);
          }
          ld_vec<K>(lds + rrow + i * TPB * K, Hh);
          ld_vec<K>(lds + rrowT + i * TPB * K, Bin);
          const uint64_t Hl = lo_row_lds<K>(lo8 + lrow + i * TPB * K);
          buf_st<K, kStream>(hist, voH, soH + (uint32_t)i * sgb, Hh);
          buf_st<K, kStream>(hist, voH, soH + (uint32_t)i * sgb + pT, Bin);
          lo_row_st<K, kStream>(hist, voHL, soH + (uint32_t)i * sgb + pL, Hl);
          double H[K];
#pragma unroll
          for (int b = 0; b < K; ++b) H[b] = df_join(Hh[b], (uint32_t)(Hl >> (8 * b)));
          ol[i] = 0;
#pragma unroll
          for (int j = 0; j < K; ++j) {
            double x[K];
#pragma unroll
            for (int b = 0; b < K; ++b) {
              const double cd = (double)cc[j][b];
              x[b] = fma(cd, fma(-k2, cd, k2w2), H[b]);
            }
            const double m = max_of<K>(x);
            float E[K];
#pragma unroll
            for (int b = 0; b < K; ++b) E[b] = ex2((float)(x[b] - m));
            float s = E[0];
#pragma unroll
            for (int b = 1; b < K; ++b) s += E[b];
            // B_{t-1}: E-weighted mean of g_t (c - r_t) + B_t over the K successors
            float num = E[0] * fmaf(gt, cc[j][0] - rt, Bin[0]);
#pragma unroll
            for (int b = 1; b < K; ++b) num = fmaf(E[b], fmaf(gt, cc[j][b] - rt, Bin[b]), num);
            const double hv = m + (double)lg2(s) - ((double)dlag + hoff);
            float lo;
            split_df(hv, oh[i][j], lo);
            ol[i] |= (uint64_t)lo8_enc(oh[i][j], lo) << (8 * j);
            vmax[0] = fmaxf(vmax[0], oh[i][j]);
            ot[i][j] = num * rcp(s);
            pin(oh[i][j]);
            pin(ot[i][j]);
          }
          sg_fence();
        }
      }
      shiftB += (double)dlag;
      if (tb == 0) sm_mB[t - 1] = dlag;
      red_pre<1, 1u>(vmax, rc);
      __syncthreads();
      red_post<1, 1u>(vmax, rc);
      dlag = floorf(vmax[0]);
#pragma unroll
      for (int i = 0; i < SGMAX; ++i) {
        if (i < SGT) {
#pragma unroll
          for (int j = 0; j < K; ++j) {
            lds[wcol + j * NSG + i * TPB] = oh[i][j];
            lds[wcolT + j * NSG + i * TPB] = ot[i][j];
            lo8[lcol + j * NSG + i * TPB] = (uint8_t)(ol[i] >> (8 * j));
          }
        }
      }
      __syncthreads();
    }

    // ------------------------------------------------------------------ S1
    // G (hi plane 0, lo bytes) and the tangent A (plane 1), updated in place
    for (int i = tb; i < GS; i += TPB) {
      lds[vb + i] = 0.f;
      lds[vb + GS + i] = 0.f;
      lo8[(uint32_t)bw * GS + i] = 0;
    }
    __syncthreads();
    double lam_est = lam0;
    float cprev = 0.f;  // g_{t-1} w_soft_{t-1}: the forward tangent's centring, applied on read
    dlag = 0.f;
    wnx = lane_rows ? ld_uniform(wbu, 0) : 0.f;
    gnx = lane_rows ? ld_uniform(gbu, 0) : 0.f;
    rnx = lane_rows ? ld_uniform(rbu, 0) : 0.f;
    // the history row and codebook rows of the next super-group (the first
    // of the next step after the last) are fetched one super-group ahead;
    // the shift of H_t one step ahead
    float pHh[K], pBc[K];
    buf_ld<K, kStream>(hist, voH, 0, pHh);
    buf_ld<K, kStream>(hist, voH, pT, pBc);
    uint64_t pHl = lo_row_ld<K, kStream>(hist, voHL, pL);
#pragma unroll
    for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, (j << (n - KB)) * 4, pc[j]);
    float mBnx = sm_mB[0];
    for (int64_t t = 0; t < L; ++t) {
      const int par = (int)(t & 1);
      rc.red = red0 + par * (NT / 64) * kRed;
      float wf, gt, rt;
      if (lane_rows) {
        wf = wnx;
        gt = gnx;
        rt = rnx;
        const int64_t tn = t + 1 < L ? t + 1 : t;
        wnx = ld_uniform(wbu, tn);
        gnx = ld_uniform(gbu, tn);
        rnx = ld_uniform(rbu, tn);
      } else {
        wf = wb[t];
        gt = gb[t];
        rt = rb[t];
      }
      if (t > 0) xbar = fmaf(gt, rt, xbar);  // B_t no longer holds step t
      const double wt = (double)wf;
      const double k2w2 = 2.0 * k2 * wt;  // as in S0: k2 w^2 out of the state terms
      const double hoff = k2 * wt * wt;
      const double lamh = lam_est + hoff;
      const double mBt = (double)mBnx;
      mBnx = sm_mB[t + 1 < L ? t + 1 : t];
      uint32_t rcol = col0, rcolT = col0 + GS, wrow = row0, wrowT = row0 + GS;
      uint32_t lcol = lcol0, lrow = lrow0;
      pin_u(rcol);
      pin_u(rcolT);
      pin_u(wrow);
      pin_u(wrowT);
      // max G_{t+1}, sum p, sum p c, sum p X, sum p c X
      float rv[5] = {-INFINITY, 0.f, 0.f, 0.f, 0.f};
      float oh[SGMAX][K], oa[SGMAX][K];  // outputs, held across the first barrier
      uint64_t ol[SGMAX];
#pragma unroll
      for (int i = 0; i < SGMAX; ++i) {
        if (i < SGT) {
          float Gh[K], Ar[K];
          float Hh[K], Bc[K], cc[K][K];
          const uint64_t Hl = pHl;
#pragma unroll
          for (int j = 0; j < K; ++j) {
            Hh[j] = pHh[j];
            Bc[j] = pBc[j];
#pragma unroll
            for (int u = 0; u < K; ++u) cc[j][u] = pc[j][u];
          }
          {  // (clamped indices, not branches)
            const bool last = i + 1 >= SGT;
            const int64_t tn = last && t + 1 < L ? t + 1 : t;
            const uint32_t so = (uint32_t)tn * hstep + (last ? 0u : (uint32_t)(i + 1) * sgb);
            buf_ld<K, kStream>(hist, voH, so, pHh);
            buf_ld<K, kStream>(hist, voH, so + pT, pBc);
            pHl = lo_row_ld<K, kStream>(hist, voHL, so + pL);
            const int ic = last ? 0 : i + 1;
#pragma unroll
            for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((ic * TPB) << KB)) * 4, pc[j]);
          }
          double G[K];
#pragma unroll
          for (int j = 0; j < K; ++j) {
            Gh[j] = lds[rcol + j * NSG + i * TPB];
            Ar[j] = lds[rcolT + j * NSG + i * TPB] - cprev;
            G[j] = df_join(Gh[j], lo8[lcol + j * NSG + i * TPB]);
          }
          ol[i] = 0;
#pragma unroll
          for (int u = 0; u < K; ++u) {
            double al[K];
#pragma unroll
            for (int j = 0; j < K; ++j) {
              const double cd = (double)cc[j][u];
              al[j] = fma(cd, fma(-k2, cd, k2w2), G[j]);
            }
            const double m = max_of<K>(al);
            float E[K];
#pragma unroll
            for (int j = 0; j < K; ++j) E[j] = ex2((float)(al[j] - m));
            // X is centred per state before the sums: at low T the moments of
            // an uncentred X cancel only to its rounding, amplified by 1/T
            const float bx = Bc[u] - xbar;
            float s = E[0], ec = E[0] * cc[0][u], sc = ec;
            float x = fmaf(gt, cc[0][u], Ar[0]) + bx;
            float sx = E[0] * x, scx = ec * x;
#pragma unroll
            for (int j = 1; j < K; ++j) {
              s += E[j];
              ec = E[j] * cc[j][u];
              sc += ec;
              x = fmaf(gt, cc[j][u], Ar[j]) + bx;
              sx = fmaf(E[j], x, sx);
              scx = fmaf(ec, x, scx);
            }
            const double gout = m + (double)lg2(s) - ((double)dlag + hoff);
            float lo;
            split_df(gout, oh[i][u], lo);
            ol[i] |= (uint64_t)lo8_enc(oh[i][u], lo) << (8 * u);
            rv[0] = fmaxf(rv[0], oh[i][u]);
            const float fac = ex2((float)(m + df_join(Hh[u], (uint32_t)(Hl >> (8 * u))) - lamh));
            rv[1] = fmaf(fac, s, rv[1]);
            rv[2] = fmaf(fac, sc, rv[2]);
            rv[3] = fmaf(fac, sx, rv[3]);
            rv[4] = fmaf(fac, scx, rv[4]);
            oa[i][u] = fmaf(sx, rcp(s), -bx);  // E-weighted mean of g c + A
            pin(oh[i][u]);
            pin(oa[i][u]);
          }
          sg_fence();
        }
      }
      red_pre<5, 1u>(rv, rc);
      __syncthreads();
      red_post<5, 1u>(rv, rc);
      const float r1 = 1.f / rv[1];
      const float wst = rv[2] * r1;
      const double lamt = lam_est + (double)lg2(rv[1]);
      const float xbe = fmaf(rv[3], r1, xbar);
      if (tb == 0) {
        if (DC) {
          sm_lam[t] = lamt;
          sm_xb[t] = xbe;
        }
        if (valid) {
          if (a.w_soft) a.w_soft[bb * L + t] = wst;
          if (a.dW) a.dW[bb * L + t] = (rv[4] - wst * rv[3]) * r1 * invT;
        }
      }
      lam_est = lamt - (double)dlag + mBt;
      dlag = floorf(rv[0]);
      cprev = gt * wst;
      xbar = xbe - cprev;
#pragma unroll
      for (int i = 0; i < SGMAX; ++i) {
        if (i < SGT) {
          st_vec<K>(lds + wrow + i * TPB * K, oh[i]);
          st_vec<K>(lds + wrowT + i * TPB * K, oa[i]);
          lo_row_lds_st<K>(lo8 + lrow + i * TPB * K, ol[i]);
          if constexpr (DC) {  // (G hi, A, G lo) entries of step t + 1, A centred as it is read
            if (t + 1 < L) {
              float ac[K];
#pragma unroll
              for (int u = 0; u < K; ++u) ac[u] = oa[i][u] - cprev;
              const uint32_t so = (uint32_t)(t + 1) * hstep + (uint32_t)i * TPB * K * 4u;
              buf_st<K, kStream>(hga, voH, so, oh[i]);
              buf_st<K, kStream>(hga, voH, so + gT, ac);
              lo_row_st<K, kStream>(hga, voHL, (uint32_t)(t + 1) * hstep + gL + (uint32_t)i * TPB * K, ol[i]);
            }
          }
        }
      }
      __syncthreads();
    }

    // ------------------------------------------------------------------ S2
    // dCodebook as in fb_kernel: per super-group over all steps, the (H, B,
    // H lo) row and the (G, A, G lo) column entries of a step loaded one
    // step ahead.
    if constexpr (DC) {
      __syncthreads();
      const bool first = base == (int64_t)blockIdx.x * BPW;
      double* part = a.dc_part + slot * ((int64_t)1 << n);
#pragma unroll 1
      for (int i = 0; i < SGT; ++i) {
        float cc[K][K], acc[K][K];
#pragma unroll
        for (int j = 0; j < K; ++j) {
          buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((i * TPB) << KB)) * 4, cc[j]);
#pragma unroll
          for (int u = 0; u < K; ++u) acc[j][u] = 0.f;
        }
        float xch = 0.f;
        float nH[K], nB[K], nG[K], nA[K];
        uint64_t nHl;
        uint32_t nGl[K];
        auto fetch = [&](int64_t ts) {
          const uint32_t so = (uint32_t)ts * hstep + (uint32_t)i * sgb;
          buf_ld<K, kStream>(hist, voH, so, nH);
          buf_ld<K, kStream>(hist, voH, so + pT, nB);
          nHl = lo_row_ld<K, kStream>(hist, voHL, so + pL);
#pragma unroll
          for (int j = 0; j < K; ++j) {  // (G, A, lo) entries a column apart
            float v1[1], v3[1];
            const uint32_t sg = (uint32_t)ts * hstep + (uint32_t)(j * NSG + i * TPB) * 4u;
            buf_ld<1, kStream>(hga, voC, sg, v1);
            buf_ld<1, kStream>(hga, voC, sg + gT, v3);
            nGl[j] = lo_byte_ld(hga, voCL, (uint32_t)ts * hstep + gL + (uint32_t)(j * NSG + i * TPB));
            nG[j] = v1[0];
            nA[j] = v3[0];
          }
        };
        fetch(0);
#pragma unroll 1
        for (int64_t t = 0; t < L; ++t) {
          float wf, gt, xt;
          if (lane_rows) {
            if ((t & 63) == 0) {
              cbase = t;
              wch = row_chunk(wb, cbase, L);
              gch = row_chunk(gb, cbase, L);
              xch = row_chunk(sm_xb, cbase, L);
            }
            const int ln = (int)(t - cbase);
            wf = read_lane(wch, ln);
            gt = read_lane(gch, ln);
            xt = read_lane(xch, ln);
          } else {
            wf = wb[t];
            gt = gb[t];
            xt = sm_xb[t];
          }
          const double wt = (double)wf;
          const double k2w2 = 2.0 * k2 * wt;
          const double lt = sm_lam[t] + k2 * wt * wt;
          float Hh[K], Bv[K], Gh[K], A[K];
          uint32_t Gl[K];
          const uint64_t Hl = nHl;
#pragma unroll
          for (int q = 0; q < K; ++q) {
            Hh[q] = nH[q];
            Bv[q] = nB[q];
            Gh[q] = nG[q];
            A[q] = nA[q];
            Gl[q] = nGl[q];
          }
          fetch(t + 1 < L ? t + 1 : t);  // (a select: the last step re-reads its own entries)
          double G[K];
#pragma unroll
          for (int j = 0; j < K; ++j) G[j] = df_join(Gh[j], Gl[j]);
#pragma unroll
          for (int u = 0; u < K; ++u) {
            const double hb = df_join(Hh[u], (uint32_t)(Hl >> (8 * u))) - lt;
            const float bx = Bv[u] - xt;
#pragma unroll
            for (int j = 0; j < K; ++j) {
              const double cd = (double)cc[j][u];
              const float p = ex2((float)(fma(cd, fma(-k2, cd, k2w2), G[j]) + hb));
              const float X = fmaf(gt, cc[j][u], A[j]) + bx;
              acc[j][u] = fmaf(p, fmaf((wf - cc[j][u]) * X, invT, gt), acc[j][u]);
            }
          }
        }
        if (valid) {
#pragma unroll
          for (int j = 0; j < K; ++j) {
            double* pj = part + ((int64_t)j << (n - KB)) + ((i * TPB) << KB) + ((uint32_t)tb << KB);
#pragma unroll
            for (int u = 0; u < K; ++u)  // (a repair pass adds into partials zeroed before it)
              pj[u] = first && !repair ? (double)acc[j][u] : pj[u] + (double)acc[j][u];
          }
        }
      }
    }
    __syncthreads();
  }
}

__global__ void dc_reduce_kernel(const double* part, int64_t nslots, int64_t S, float* out) {
  const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  double acc = 0.0;
  for (int64_t q = 0; q < nslots; ++q) acc += part[q * S + s];
  out[s] = (float)acc;
}

// c'(s) = kappa c(s): the codebook in the scaled units of fb_kernel.
__global__ void scale_kernel(const float* c, float kap, float* cs, int64_t S) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < S) cs[i] = c[i] * kap;
}

// rows[r * stride + c] = v for r < nrows, c < row_len
__global__ void fill_rows_kernel(float* rows, int64_t stride, int64_t nrows, int64_t row_len, float v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < nrows * row_len) rows[(i / row_len) * stride + i % row_len] = v;
}

__global__ void fill_kernel(float* out, int64_t count, float v) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) out[i] = v;
}

// ---------------------------------------------------------------------------
// Min-sum decode (paper Sec. 3.2), fp64 path metrics.  Same super-group
// layout as the forward sweep: Mn_{t+1}(v) = min_j [d_t(j*S/K + v) + Mn_t(j, v >> k)]
// with d_t(s) = (w_t - c(s))^2; the winning j is kept per (t, v).
// The metric vector lives in LDS as two 32-bit planes (low and high words
// of each double): the row-form writes are then 16-byte stores at a 16-byte
// lane stride and the column-form reads lane-contiguous 4-byte reads, both
// free of bank conflicts (8-byte rows at a 32-byte lane stride conflicted
// 4-way).  The K winning digits of a super-group row go out as one store.
// w_t comes through the scalar unit when a block spans whole waves.
// ---------------------------------------------------------------------------
__device__ __forceinline__ double join_d(float lo, float hi) {
  return __hiloint2double(__float_as_int(hi), __float_as_int(lo));
}

template <int K>
__device__ __forceinline__ void st_digits(uint8_t* p, const uint8_t (&arg)[K]) {
  if constexpr (K == 2) {
    *reinterpret_cast<uint16_t*>(p) = (uint16_t)(arg[0] | (arg[1] << 8));
  } else if constexpr (K == 4) {
    *reinterpret_cast<uint32_t*>(p) =
        (uint32_t)arg[0] | ((uint32_t)arg[1] << 8) | ((uint32_t)arg[2] << 16) | ((uint32_t)arg[3] << 24);
  } else {
#pragma unroll
    for (int q = 0; q < K / 4; ++q)
      reinterpret_cast<uint32_t*>(p)[q] = (uint32_t)arg[4 * q] | ((uint32_t)arg[4 * q + 1] << 8) |
                                          ((uint32_t)arg[4 * q + 2] << 16) | ((uint32_t)arg[4 * q + 3] << 24);
  }
}

template <int KB, int NB, int SGMAX, int NT>
__global__ void __launch_bounds__(NT) viterbi_kernel(VitArgs a) {
  constexpr int K = 1 << KB;
  extern __shared__ double ldsd[];
  const int n = NB ? NB : a.n;
  const int GS = 1 << (n - KB);
  const int NSG = 1 << (n - 2 * KB);
  const int SGT = NB ? SGMAX : a.sgt;
  const int TPB = NSG / SGT;
  const int BPW = NT / TPB;
  const int tid = threadIdx.x;
  const int bw = tid / TPB;
  const int tb = tid - bw * TPB;
  const uint32_t toK = (uint32_t)tb << KB;
  const int lane = tid & 63, wave = tid >> 6;
  const int width = TPB < 64 ? TPB : 64;
  const int rw = TPB > 64 ? TPB / 64 : 1;
  const int64_t L = a.L;
  float* const mlo = reinterpret_cast<float*>(ldsd) + (size_t)bw * 2 * GS;  // low words
  float* const mhi = mlo + GS;                                               // high words
  double* redv = ldsd + (size_t)BPW * GS;            // [waves]
  int* redi = reinterpret_cast<int*>(redv + NT / 64); // [waves]
  const bool lane_rows = TPB >= 64;
  // codebook rows through a buffer descriptor, one super-group ahead
  const rsrc_t cbk = make_rsrc(a.c, (uint32_t)4 << n);
  const uint32_t voK = (uint32_t)tb << (KB + 2);

  for (int64_t base = (int64_t)blockIdx.x * BPW; base < a.B; base += (int64_t)gridDim.x * BPW) {
    const int64_t blk = base + bw;
    const bool valid = blk < a.B;
    const int64_t bb = valid ? blk : a.B - 1;
    const int64_t slot = (int64_t)blockIdx.x * BPW + bw;
    const float* wb = a.w + bb * L;
    const int64_t bbu = lane_rows ? (int64_t)__builtin_amdgcn_readfirstlane((int)bb) : 0;
    const float* wbu = a.w + bbu * L;
    uint8_t* bp = a.bp + slot * L * GS;

    for (int i = tb; i < GS; i += TPB) {
      mlo[i] = 0.f;
      mhi[i] = 0.f;
    }
    __syncthreads();
    double bestv = INFINITY;
    int besti = 0x7fffffff;
    float wnx = lane_rows ? ld_uniform(wbu, 0) : 0.f;
    float pc[K][K];
#pragma unroll
    for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, (j << (n - KB)) * 4, pc[j]);
    for (int64_t t = 0; t < L; ++t) {
      float wf;
      if (lane_rows) {
        wf = wnx;
        wnx = ld_uniform(wbu, t + 1 < L ? t + 1 : t);
      } else {
        wf = wb[t];
      }
      const double wt = (double)wf;
      double Mout[SGMAX][K];
#pragma unroll
      for (int i = 0; i < SGMAX; ++i) {
        if (i < SGT) {
          const int sg = tb + i * TPB;
          double Min[K];
#pragma unroll
          for (int j = 0; j < K; ++j) Min[j] = join_d(mlo[j * NSG + sg], mhi[j * NSG + sg]);
          float cc[K][K];
#pragma unroll
          for (int j = 0; j < K; ++j) {
#pragma unroll
            for (int u = 0; u < K; ++u) cc[j][u] = pc[j][u];
          }
          {  // the next super-group's rows (the first of the next step after the last)
            const int ic = i + 1 < SGT ? i + 1 : 0;
#pragma unroll
            for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((ic * TPB) << KB)) * 4, pc[j]);
          }
          if (t < L - 1) {
            uint8_t arg[K];
#pragma unroll
            for (int u = 0; u < K; ++u) {
              double best = 0.0;
              int bj = 0;
#pragma unroll
              for (int j = 0; j < K; ++j) {
                const double d = wt - (double)cc[j][u];
                const double v = __dadd_rn(__dmul_rn(d, d), Min[j]);
                if (j == 0 || v < best) {
                  best = v;
                  bj = j;
                }
              }
              Mout[i][u] = best;
              arg[u] = (uint8_t)bj;
            }
            // bp[t+1][sg*K + u] = winning j of G-entry (sg, u)
            st_digits<K>(bp + (t + 1) * GS + sg * K, arg);
          } else {
#pragma unroll
            for (int j = 0; j < K; ++j)
#pragma unroll
              for (int u = 0; u < K; ++u) {
                const double d = wt - (double)cc[j][u];
                const double v = __dadd_rn(__dmul_rn(d, d), Min[j]);
                const int s = (j << (n - KB)) | (sg << KB) | u;
                if (v < bestv || (v == bestv && s < besti)) {
                  bestv = v;
                  besti = s;
                }
              }
          }
          sg_fence();
        }
      }
      if (t < L - 1) {
        __syncthreads();
#pragma unroll
        for (int i = 0; i < SGMAX; ++i) {
          if (i < SGT) {
            const int sg = tb + i * TPB;
            float lo[K], hi[K];
#pragma unroll
            for (int u = 0; u < K; ++u) {
              lo[u] = __int_as_float(__double2loint(Mout[i][u]));
              hi[u] = __int_as_float(__double2hiint(Mout[i][u]));
            }
            st_vec<K>(mlo + sg * K, lo);
            st_vec<K>(mhi + sg * K, hi);
          }
        }
        __syncthreads();
      }
    }
    // block argmin (value, then state index)
    for (int off = 1; off < width; off <<= 1) {
      const double ov = __shfl_xor(bestv, off);
      const int oi = __shfl_xor(besti, off);
      if (ov < bestv || (ov == bestv && oi < besti)) {
        bestv = ov;
        besti = oi;
      }
    }
    if (rw > 1 && lane == 0) {
      redv[wave] = bestv;
      redi[wave] = besti;
    }
    __syncthreads();  // also publishes every thread's bp stores to the block
    if (rw > 1) {
      const int first = (wave / rw) * rw;
      bestv = redv[first];
      besti = redi[first];
      for (int q = 1; q < rw; ++q) {
        const double ov = redv[first + q];
        const int oi = redi[first + q];
        if (ov < bestv || (ov == bestv && oi < besti)) {
          bestv = ov;
          besti = oi;
        }
      }
    }
    if (tb == 0 && valid) {
      int32_t* st = a.states + bb * L;
      float* wh = a.w_hard ? a.w_hard + bb * L : nullptr;
      // (non-finite inputs leave no state below +inf: start from state 0)
      int s = (unsigned)besti < (unsigned)(GS << KB) ? besti : 0;
      st[L - 1] = s;
      if (wh) wh[L - 1] = a.c[s];
      for (int64_t t = L - 1; t >= 1; --t) {
        const int v = s >> KB;
        const int j = bp[t * GS + v];
        s = (j << (n - KB)) | v;
        st[t - 1] = s;
        if (wh) wh[t - 1] = a.c[s];
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Approximate min-sum decode, used only for the centring reference of the
// low-temperature VJP (fb_kernel_hp): the same recursion, digits and
// traceback as viterbi_kernel with fp32 path metrics (exact ties and
// rounding-level near-ties may resolve differently; the VJP's mathematics
// holds for any reference, which only has to follow the posterior to keep
// the fp32 tangent well conditioned).  The metric vector is ping-ponged
// between two S/K planes in LDS (the footprint of viterbi_kernel's two
// 32-bit planes): one barrier per step and no metrics held across it.
// ---------------------------------------------------------------------------
template <int KB, int NB, int SGMAX, int NT>
__global__ void __launch_bounds__(NT) viterbi_ref_kernel(VitArgs a) {
  constexpr int K = 1 << KB;
  extern __shared__ float ldsv[];
  const int n = NB ? NB : a.n;
  const int GS = 1 << (n - KB);
  const int NSG = 1 << (n - 2 * KB);
  const int SGT = NB ? SGMAX : a.sgt;
  const int TPB = NSG / SGT;
  const int BPW = NT / TPB;
  const int tid = threadIdx.x;
  const int bw = tid / TPB;
  const int tb = tid - bw * TPB;
  const int lane = tid & 63, wave = tid >> 6;
  const int width = TPB < 64 ? TPB : 64;
  const int rw = TPB > 64 ? TPB / 64 : 1;
  const int64_t L = a.L;
  float* const m0 = ldsv + (size_t)bw * 2 * GS;   // plane read at even steps
  float* const m1 = m0 + GS;                      // plane read at odd steps
  float* redv = ldsv + (size_t)BPW * 2 * GS;      // [waves]
  int* redi = reinterpret_cast<int*>(redv + NT / 64);  // [waves]
  const bool lane_rows = TPB >= 64;
  const rsrc_t cbk = make_rsrc(a.c, (uint32_t)4 << n);
  const uint32_t voK = (uint32_t)tb << (KB + 2);
  const bool repair = BPW == 1 && a.flags;

  for (int64_t base = (int64_t)blockIdx.x * BPW; base < a.B; base += (int64_t)gridDim.x * BPW) {
    if (repair && !ld_uniform_i(a.flags, base)) continue;
    const int64_t blk = base + bw;
    const bool valid = blk < a.B;
    const int64_t bb = valid ? blk : a.B - 1;
    const int64_t slot = (int64_t)blockIdx.x * BPW + bw;
    const float* wb = a.w + bb * L;
    const int64_t bbu = lane_rows ? (int64_t)__builtin_amdgcn_readfirstlane((int)bb) : 0;
    const float* wbu = a.w + bbu * L;
    uint8_t* bp = a.bp + slot * L * GS;

    for (int i = tb; i < GS; i += TPB) m0[i] = 0.f;
    __syncthreads();
    float bestv = INFINITY;
    int besti = 0x7fffffff;
    float wnx = lane_rows ? ld_uniform(wbu, 0) : 0.f;
    float pc[K][K];
#pragma unroll
    for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, (j << (n - KB)) * 4, pc[j]);
    for (int64_t t = 0; t < L; ++t) {
      float wt;
      if (lane_rows) {
        wt = wnx;
        wnx = ld_uniform(wbu, t + 1 < L ? t + 1 : t);
      } else {
        wt = wb[t];
      }
      const float* min_ = (t & 1) ? m1 : m0;
      float* mout = (t & 1) ? m0 : m1;
#pragma unroll
      for (int i = 0; i < SGMAX; ++i) {
        if (i < SGT) {
          const int sg = tb + i * TPB;
          float Min[K];
#pragma unroll
          for (int j = 0; j < K; ++j) Min[j] = min_[j * NSG + sg];
          float cc[K][K];
#pragma unroll
          for (int j = 0; j < K; ++j) {
#pragma unroll
            for (int u = 0; u < K; ++u) cc[j][u] = pc[j][u];
          }
          {  // the next super-group's rows (the first of the next step after the last)
            const int ic = i + 1 < SGT ? i + 1 : 0;
#pragma unroll
            for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, ((j << (n - KB)) + ((ic * TPB) << KB)) * 4, pc[j]);
          }
          if (t < L - 1) {
            uint8_t arg[K];
            float mo[K];
#pragma unroll
            for (int u = 0; u < K; ++u) {
              float best = 0.f;
              int bj = 0;
#pragma unroll
              for (int j = 0; j < K; ++j) {
                const float d = wt - cc[j][u];
                const float v = fmaf(d, d, Min[j]);
                if (j == 0 || v < best) {
                  best = v;
                  bj = j;
                }
              }
              mo[u] = best;
              arg[u] = (uint8_t)bj;
            }
            st_vec<K>(mout + sg * K, mo);
            st_digits<K>(bp + (t + 1) * GS + sg * K, arg);
          } else {
#pragma unroll
            for (int j = 0; j < K; ++j)
#pragma unroll
              for (int u = 0; u < K; ++u) {
                const float d = wt - cc[j][u];
                const float v = fmaf(d, d, Min[j]);
                const int s = (j << (n - KB)) | (sg << KB) | u;
                if (v < bestv || (v == bestv && s < besti)) {
                  bestv = v;
                  besti = s;
                }
              }
          }
          sg_fence();
        }
      }
      if (t < L - 1) __syncthreads();
    }
    // block argmin (value, then state index)
    for (int off = 1; off < width; off <<= 1) {
      const float ov = __shfl_xor(bestv, off);
      const int oi = __shfl_xor(besti, off);
      if (ov < bestv || (ov == bestv && oi < besti)) {
        bestv = ov;
        besti = oi;
      }
    }
    if (rw > 1 && lane == 0) {
      redv[wave] = bestv;
      redi[wave] = besti;
    }
    __syncthreads();  // also publishes every thread's bp stores to the block
    if (rw > 1) {
      const int first = (wave / rw) * rw;
      bestv = redv[first];
      besti = redi[first];
      for (int q = 1; q < rw; ++q) {
        const float ov = redv[first + q];
        const int oi = redi[first + q];
        if (ov < bestv || (ov == bestv && oi < besti)) {
          bestv = ov;
          besti = oi;
        }
      }
    }
    if (tb == 0 && valid) {
      int32_t* st = a.states + bb * L;
      float* wh = a.w_hard ? a.w_hard + bb * L : nullptr;
      // (non-finite inputs leave no state below +inf: start from state 0)
      int s = (unsigned)besti < (unsigned)(GS << KB) ? besti : 0;
      st[L - 1] = s;
      if (wh) wh[L - 1] = a.c[s];
      for (int64_t t = L - 1; t >= 1; --t) {
        const int v = s >> KB;
        const int j = bp[t * GS + v];
        s = (j << (n - KB)) | v;
        st[t - 1] = s;
        if (wh) wh[t - 1] = a.c[s];
      }
    }
    __syncthreads();
  }
}

}  // namespace bcjr
