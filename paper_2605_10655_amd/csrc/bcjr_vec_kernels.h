// bcjr_vec_kernels.h -- gfx950 kernels for the vector-emission trellis:
// k = 4 bits per step (K = 16 predecessors and successors per state) and
// V = 2 weights per step, each state emitting a 2-vector codeword (paper
// Sec. 3.1 with V = 2, the trellis shape used in Sec. 4.1 and Sec. 4.4).
//
// Index algebra.  n state bits, S = 2^n, GS = S/16 groups, NSG = S/256.
// A state is s = (r, m, u): r the top 4 bits, m the middle n - 8 bits, u the
// low 4 bits.  With next(s, b) = ((s << 4) | b) & (S - 1):
//   log alpha_t(s) = h_t(s) + G_t(s >> 4),      s >> 4 = r * NSG + m
//   G_{t+1}(m * 16 + u) = LSE_r [h_t(r, m, u) + G_t(r * NSG + m)]
//   log beta_t(s)  = H_t(s & (GS - 1)) = H_t(m * 16 + u)
//   H_{t-1}(r * NSG + m) = LSE_u [h_t(r, m, u) + H_t(m * 16 + u)]
// so the 256 states of one m form a 16 x 16 tile whose forward step reduces
// the columns (over r) and whose backward step reduces the rows (over u).
// Sixteen lanes work one tile: lane l takes column l in the forward sweep and
// row l in the backward sweep, so every log-sum-exp is a 16-term loop in one
// lane and no lane exchange is needed.  h_t(s) = -||w_t - c(s)||^2 / (2T)
// (Eq. boltzmann with a 2-vector emission); in the scaled log2 units used
// here it is -(w'_0 - c'_0)^2 - (w'_1 - c'_1)^2 with w' = kappa w,
// c' = kappa c, kappa = sqrt(log2(e) / (2T)).
//
// Each step's group vectors live in LDS as (value, tangent) float2 pairs,
// alternating between two buffers, so a step needs a single barrier (plus
// its reductions).  The integer shift that keeps a vector near 0 is the
// floor of the maximum of the vector being read (known from the previous
// step's reduction), applied to the values written.  Entry v of a vector is
// stored at v + 4 (v >> lg NSG) (NSG >= 16): the backward step writes
// column-form entries r * NSG + m, whose 16 rows would otherwise fall in the
// same LDS banks; row-form runs m * 16 .. m * 16 + 15 stay contiguous.
//
// The marginal, soft codeword and VJP follow the scalar kernels: the
// backward tangent B accumulates <g_t, c(s_t) - w_t>, the forward tangent A
// accumulates <g_t, c(s_t)> and is centred on <g_t, w_soft_t> when it is
// read one step later, X_t = <g_t, c> + A_t + B_t - xbar_t, and
// dW_{t,a} = (sum p c_a X - w_soft_{t,a} sum p X) / (T sum p) per component.
#pragma once
#include "bcjr_kernels.h"

namespace bcjr {
namespace {

struct VecGeom {
  int n, GS, NSG, lgNSG, pad, VSZ;
  __device__ __forceinline__ int phys(int v) const { return v + pad * (v >> lgNSG); }
  // the same positions written per field: column-form entry r * NSG + m
  // (m < NSG) and the start of row-form run m * 16 + (0..15)
  __device__ __forceinline__ int col(int r, int m) const { return r * (NSG + pad) + m; }
  __device__ __forceinline__ int row(int m) const {
    return m * 16 + (pad ? pad * (m >> (lgNSG - 4)) : 0);
  }
};

__device__ __forceinline__ VecGeom vec_geom(int n) {
  VecGeom q;
  q.n = n;
  q.GS = 1 << (n - 4);
  q.NSG = 1 << (n - 8);
  q.lgNSG = n - 8;
  q.pad = q.NSG >= 16 ? 4 : 0;
  q.VSZ = q.GS + 16 * q.pad;
  return q;
}

// Step t's two weights (or gradients) of a block row: lane l of a wave holds
// row[base + l], 32 steps per chunk, taken with lane reads.
struct PairRows {
  float ch = 0.f;
  int64_t base = 0;
};

__device__ __forceinline__ void pair_at(const float* row, int64_t t, int64_t L, bool lane_rows,
                                        bool reload, PairRows& pr, float& x0, float& x1) {
  if (lane_rows) {
    if (reload) {
      pr.base = 2 * (t & ~(int64_t)31);
      pr.ch = row_chunk(row, pr.base, L);
    }
    const int o = (int)(2 * t - pr.base);
    x0 = read_lane(pr.ch, o);
    x1 = read_lane(pr.ch, o + 1);
  } else {
    x0 = row[2 * t];
    x1 = row[2 * t + 1];
  }
}

// The 16 codewords of one tile row (backward sweep) from the transposed
// scaled codebook: cc[2u], cc[2u + 1] = c'(r * GS + m * 16 + u).
__device__ __forceinline__ void row_codewords(rsrc_t cT, uint32_t voff, uint32_t soff, float (&cc)[32]) {
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    float v[2];
    buf_ld<2>(cT, voff, soff + (uint32_t)u * 128u, v);
    cc[2 * u] = v[0];
    cc[2 * u + 1] = v[1];
  }
}

// History entry of one lane: H, and B after it with the VJP (HW = 2).
template <int HW>
__device__ __forceinline__ void hist_entry(rsrc_t h, uint32_t voff, uint32_t soff, float (&e)[2]) {
  if constexpr (HW == 2) {
    buf_ld<2>(h, voff, soff, e);
  } else {
    float e1[1];
    buf_ld<1>(h, voff, soff, e1);
    e[0] = e1[0];
    e[1] = 0.f;
  }
}

// ---------------------------------------------------------------------------
// Soft codeword, logZ and the VJP (dW, and dCodebook with DC).  NB > 0 fixes
// the state bits at compile time (then SGT = SGMAX).
//   S0 backward: H (and B) per step, stored to the history;
//   S1 forward:  G (and A), marginals, w_soft, dW;
//   S2 (DC):     dCodebook per state from the (G, A) and (H, B) histories.
// ---------------------------------------------------------------------------
template <int NB, int SGMAX, int NT, bool VJP, bool DC>
__global__ void __launch_bounds__(NT) fbv_kernel(FbvArgs a) {
  extern __shared__ float lds[];
  const int n = NB ? NB : a.n;
  const VecGeom q = vec_geom(n);
  const int GS = q.GS, NSG = q.NSG;
  const int SGT = NB ? SGMAX : a.sgt;     // tiles per thread
  const int TPB = 16 * NSG / SGT;          // threads per block
  const int TQ = TPB / 16;                 // tiles per pass
  const int BPW = NT / TPB;                // blocks per workgroup
  const int tid = threadIdx.x;
  const int bw = BPW == 1 ? 0 : tid / TPB;
  const int tb = BPW == 1 ? tid : tid - bw * TPB;
  const int tq = tb >> 4, tl = tb & 15;
  const int64_t N = a.N, L = 2 * a.N;
  const float kap = a.kap;
  constexpr int HW = VJP ? 2 : 1;          // floats per history entry

  RedCtx rc;
  rc.width = TPB < 64 ? TPB : 64;
  rc.rw = TPB > 64 ? TPB / 64 : 1;
  rc.wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: a scalar
  float* const red0 = lds + (size_t)BPW * 4 * q.VSZ;  // [2 parities][waves][kRed]
  rc.red = red0;
  float* const vec0 = lds + (size_t)bw * 4 * q.VSZ;   // two float2 vectors
  float* const vec1 = vec0 + 2 * q.VSZ;

  const rsrc_t cbk = make_rsrc(a.cs, (uint32_t)8 << n);
  const rsrc_t cbkT = make_rsrc(a.csT, (uint32_t)8 << n);
  // forward sweep: column tl of tile m reads states r * GS + m * 16 + tl
  const uint32_t voC1 = ((uint32_t)tq * 16 + tl) * 8u;
  // backward sweep: row tl of tile m reads states tl * GS + m * 16 + u, u < 16,
  // from the transposed copy, entry (m * 16 + u) * 16 + tl: for each u the
  // 16 rows of a tile are one contiguous 128-byte line
  const uint32_t voC0 = ((uint32_t)tq * 256 + tl) * 8u;
  const uint32_t tileCT = (uint32_t)TQ * 2048u;        // transposed-copy bytes between tile slots
  const uint32_t tileC = (uint32_t)TQ * 128u;          // codebook bytes between tile slots
  const uint32_t hstep = (uint32_t)GS * HW * 4u;       // history bytes per step
  const uint32_t voH = (uint32_t)bw * (uint32_t)N * hstep + ((uint32_t)tq * 16 + tl) * HW * 4u;
  const uint32_t tileH = (uint32_t)TQ * 16u * HW * 4u;
  const bool lane_rows = TPB >= 64;

  for (int64_t base = (int64_t)blockIdx.x * BPW; base < a.B; base += (int64_t)gridDim.x * BPW) {
    const int64_t blk = base + bw;
    const bool valid = blk < a.B;
    const int64_t bb = valid ? blk : a.B - 1;
    const int64_t slot = (int64_t)blockIdx.x * BPW + bw;
    const int64_t slot0 = (int64_t)blockIdx.x * BPW;
    const float* wb = a.w + bb * L;
    const float* gb = VJP ? a.g + bb * L : nullptr;
    const rsrc_t hist = make_rsrc(a.hist + slot0 * N * GS * HW, (uint32_t)BPW * (uint32_t)N * hstep);
    const rsrc_t hga = make_rsrc(DC ? a.histGA + slot0 * N * GS * 2 : a.hist,
                                 DC ? (uint32_t)BPW * (uint32_t)N * (uint32_t)GS * 8u : 0u);
    float* sm_mB = a.small + slot * 4 * N;  // shift applied to H_t
    float* sm_lam = sm_mB + N;              // dCodebook: lambda_t
    float* sm_xb = sm_lam + N;              // dCodebook: E_p[X_t]
    float* sm_cp = sm_xb + N;               // dCodebook: centring constant of A_t

    // ---------------------------------------------------------------- S0
    for (int i = tb; i < 2 * q.VSZ; i += TPB) vec0[i] = 0.f;
    if (tb == 0) sm_mB[N - 1] = 0.f;
    __syncthreads();
    double shiftB = 0.0;   // sum of the shifts applied to H (exact)
    float dl = 0.f;        // shift for the values written this step
    float lam0 = 0.f, xbar = 0.f;
    PairRows rw_, rg_;
    // each tile's history entry is stored once the next tile's codebook
    // loads are issued: the vector-memory counter retires loads and stores in
    // order, so waiting for those loads would otherwise wait for the store
    float pend[2] = {0.f, 0.f};
    uint32_t pend_so = 0;
    bool pend_on = false;
    for (int64_t t = N - 1;; --t) {
      const int par = (int)((N - 1 - t) & 1);
      rc.red = red0 + par * (NT / 64) * kRed;
      float* cur = par ? vec1 : vec0;
      float* nxt = par ? vec0 : vec1;
      const bool reload = t == N - 1 || (t & 31) == 31;
      float w0, w1, g0 = 0.f, g1 = 0.f;
      pair_at(wb, t, L, lane_rows, reload, rw_, w0, w1);
      if (VJP) pair_at(gb, t, L, lane_rows, reload, rg_, g0, g1);
      w0 *= kap;
      w1 *= kap;
      const uint32_t soH = (uint32_t)t * hstep;
      if (t == 0) {
        if (pend_on) {
          if constexpr (VJP) {
            buf_st<2>(hist, voH, pend_so, pend);
          } else {
            float o1[1] = {pend[0]};
            buf_st<1>(hist, voH, pend_so, o1);
          }
        }
        // lambda_0 = LSE_s [h_0(s) + H_0(s & (GS - 1))] (log2 alpha_0 = h_0), and
        // with the VJP E_p[<g_0, c(s_0)> + B_0(s_0)], the mean of X_0
        float lm = -INFINITY, ls = 0.f, ly = 0.f;
#pragma unroll 1
        for (int i = 0; i < SGT; ++i) {
          {
            const int m = tq + i * TQ;
            float cc[32], hb[32];
            row_codewords(cbkT, voC0, (uint32_t)i * tileCT, cc);
#pragma unroll
            for (int u4 = 0; u4 < 8; ++u4) {
              float t4[4];
              ld_vec<4>(cur + 2 * q.row(m) + 4 * u4, t4);
#pragma unroll
              for (int e = 0; e < 4; ++e) hb[4 * u4 + e] = t4[e];
            }
            float own[2];
            ld_vec<2>(cur + 2 * (q.row(m) + tl), own);
            if constexpr (VJP) {
              buf_st<2>(hist, voH, soH + (uint32_t)i * tileH, own);
            } else {
              float o1[1] = {own[0]};
              buf_st<1>(hist, voH, soH + (uint32_t)i * tileH, o1);
            }
            float x[16];
#pragma unroll
            for (int u = 0; u < 16; ++u) {
              const float d0 = w0 - cc[2 * u], d1 = w1 - cc[2 * u + 1];
              x[u] = fmaf(-d1, d1, fmaf(-d0, d0, hb[2 * u]));
            }
            const float M = max_of<16>(x);
            float s = 0.f, sy = 0.f;
#pragma unroll
            for (int u = 0; u < 16; ++u) {
              const float E = ex2(x[u] - M);
              s += E;
              if constexpr (VJP) sy = fmaf(E, fmaf(g1, cc[2 * u + 1], fmaf(g0, cc[2 * u], hb[2 * u + 1])), sy);
            }
            if constexpr (VJP) {
              lse3_pair(lm, ls, ly, M, s, sy);
            } else {
              lse_pair(lm, ls, M, s);
            }
            sg_fence();
          }
        }
        if constexpr (VJP) {
          lse3_pre(lm, ls, ly, rc);
        } else {
          lse_pre(lm, ls, rc);
        }
        __syncthreads();
        if constexpr (VJP) {
          lse3_post(lm, ls, ly, rc);
          xbar = ly / ls;
        } else {
          lse_post(lm, ls, rc);
        }
        lam0 = lm + lg2(ls);
        if (tb == 0 && valid && a.logZ)
          a.logZ[bb] = (float)((shiftB + (double)lam0) * 0.69314718055994530942);
        __syncthreads();
        break;
      }
      float vmax[1] = {-INFINITY};
#pragma unroll 1
      for (int i = 0; i < SGT; ++i) {
        {
          const int m = tq + i * TQ;
          float cc[32], hb[32];
          row_codewords(cbkT, voC0, (uint32_t)i * tileCT, cc);
#pragma unroll
          for (int u4 = 0; u4 < 8; ++u4) {
            float t4[4];
            ld_vec<4>(cur + 2 * q.row(m) + 4 * u4, t4);
#pragma unroll
            for (int e = 0; e < 4; ++e) hb[4 * u4 + e] = t4[e];
          }
          if (pend_on) {
            if constexpr (VJP) {
              buf_st<2>(hist, voH, pend_so, pend);
            } else {
              float o1[1] = {pend[0]};
              buf_st<1>(hist, voH, pend_so, o1);
            }
          }
          ld_vec<2>(cur + 2 * (q.row(m) + tl), pend);
          pend_so = soH + (uint32_t)i * tileH;
          pend_on = true;
          // in place: hb[2u] <- log2 of the row's successor terms, hb[2u+1] <- the
          // summand of B_{t-1}, <g_t, c - w_t> + B_t (E-weighted mean below)
          float x[16];
#pragma unroll
          for (int u = 0; u < 16; ++u) {
            const float d0 = w0 - cc[2 * u], d1 = w1 - cc[2 * u + 1];
            x[u] = fmaf(-d1, d1, fmaf(-d0, d0, hb[2 * u]));
            if constexpr (VJP) hb[2 * u + 1] = fmaf(-g1, d1, fmaf(-g0, d0, hb[2 * u + 1]));
          }
          const float M = max_of<16>(x);
          float s = 0.f, sy = 0.f;
#pragma unroll
          for (int u = 0; u < 16; ++u) {
            const float E = ex2(x[u] - M);
            s += E;
            if constexpr (VJP) sy = fmaf(E, hb[2 * u + 1], sy);
          }
          const float Hn = M + lg2(s) - dl;
          vmax[0] = fmaxf(vmax[0], Hn);
          float o[2] = {Hn, VJP ? sy * rcp(s) : 0.f};
          st_vec<2>(nxt + 2 * q.col(tl, m), o);
          sg_fence();
        }
      }
      red_pre<1, 1u>(vmax, rc);
      __syncthreads();
      red_post<1, 1u>(vmax, rc);
      if (tb == 0) sm_mB[t - 1] = dl;
      shiftB += (double)dl;
      dl = floorf(vmax[0]);
    }

    // ---------------------------------------------------------------- S1
    for (int i = tb; i < 2 * q.VSZ; i += TPB) vec0[i] = 0.f;
    if constexpr (DC) {  // (G_0, A_0) = 0
      float z[2] = {0.f, 0.f};
#pragma unroll
      for (int i = 0; i < SGMAX; ++i)
        if (i < SGT) buf_st<2>(hga, voH, (uint32_t)i * tileH, z);
    }
    __syncthreads();
    const float dws = a.dws;
    float lam = lam0;
    float dlG = 0.f;   // shift for the G values written this step
    float cprev = 0.f; // <g_{t-1}, w_soft_{t-1}>: centring of the A being read
    // The history entry of the next tile is loaded one tile ahead (the last
    // tile of a step fetches the first of the next step), so its HBM latency
    // overlaps the current tile's arithmetic.
    float pH[2] = {0.f, 0.f};
    hist_entry<HW>(hist, voH, 0u, pH);
    for (int64_t t = 0; t < N; ++t) {
      const int par = (int)(t & 1);
      rc.red = red0 + par * (NT / 64) * kRed;
      float* cur = par ? vec1 : vec0;
      float* nxt = par ? vec0 : vec1;
      const bool reload = (t & 31) == 0;
      float w0, w1, g0 = 0.f, g1 = 0.f;
      pair_at(wb, t, L, lane_rows, reload, rw_, w0, w1);
      if (VJP) pair_at(gb, t, L, lane_rows, reload, rg_, g0, g1);
      w0 *= kap;
      w1 *= kap;
      if (VJP && t > 0) xbar = fmaf(g1, w1, fmaf(g0, w0, xbar));  // B_t no longer holds step t
      const float mBt = sm_mB[t];
      const uint32_t soH = (uint32_t)t * hstep;
      // max G_{t+1}, sum p, sum p c_0, sum p c_1, and with the VJP sum p X,
      // sum p c_0 X, sum p c_1 X
      constexpr int NR = VJP ? 7 : 4;
      float rv[NR];
      rv[0] = -INFINITY;
#pragma unroll
      for (int k = 1; k < NR; ++k) rv[k] = 0.f;
#pragma unroll 1
      for (int i = 0; i < SGT; ++i) {
        {
          const int m = tq + i * TQ;
          const float hu[2] = {pH[0], pH[1]};
          float c0[16], c1[16], G[16], A[16];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            float cv[2], ga[2];
            buf_ld<2>(cbk, voC1, (uint32_t)r * (uint32_t)GS * 8u + (uint32_t)i * tileC, cv);
            c0[r] = cv[0];
            c1[r] = cv[1];
            ld_vec<2>(cur + 2 * q.col(r, m), ga);
            G[r] = ga[0];
            A[r] = ga[1];
          }
          {
            // (a select, not a branch: at t = N - 1 it re-reads an entry of step t, unused)
            const bool last = i + 1 >= SGT;
            const int64_t tn = last && t + 1 < N ? t + 1 : t;
            hist_entry<HW>(hist, voH, (uint32_t)tn * hstep + (last ? 0u : (uint32_t)(i + 1) * tileH), pH);
          }
          // in place: G[r] <- log2 alpha_t of the column's states, A[r] <- y_r =
          // <g_t, c> + A_t (raw) of the same states
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float d0 = w0 - c0[r], d1 = w1 - c1[r];
            G[r] = fmaf(-d1, d1, fmaf(-d0, d0, G[r]));
            if constexpr (VJP) A[r] = fmaf(g1, c1[r], fmaf(g0, c0[r], A[r]));
          }
          const float M = max_of<16>(G);
          float s = 0.f, e0 = 0.f, e1 = 0.f, ey = 0.f, ey0 = 0.f, ey1 = 0.f;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float E = ex2(G[r] - M);
            s += E;
            e0 = fmaf(E, c0[r], e0);
            e1 = fmaf(E, c1[r], e1);
            if constexpr (VJP) {
              const float Ey = E * A[r];
              ey += Ey;
              ey0 = fmaf(Ey, c0[r], ey0);
              ey1 = fmaf(Ey, c1[r], ey1);
            }
          }
          const float Gn = M + lg2(s) - dlG;
          rv[0] = fmaxf(rv[0], Gn);
          const float f = ex2(M + hu[0] - lam);
          rv[1] = fmaf(f, s, rv[1]);
          rv[2] = fmaf(f, e0, rv[2]);
          rv[3] = fmaf(f, e1, rv[3]);
          float An = 0.f;
          if constexpr (VJP) {
            // X = <g_t, c> + A_raw - cprev + B_t - xbar over the column's states
            const float qv = hu[1] - xbar - cprev;
            rv[4] = fmaf(f, fmaf(qv, s, ey), rv[4]);
            rv[5] = fmaf(f, fmaf(qv, e0, ey0), rv[5]);
            rv[6] = fmaf(f, fmaf(qv, e1, ey1), rv[6]);
            An = fmaf(ey, rcp(s), -cprev);
          }
          if (t < N - 1) {
            float o[2] = {Gn, An};
            st_vec<2>(nxt + 2 * (q.row(m) + tl), o);
            // (G_{t+1}, A_{t+1}) as the next step reads them, for the dCodebook sweep
            if constexpr (DC) buf_st<2>(hga, voH, soH + hstep + (uint32_t)i * tileH, o);
          }
          sg_fence();
        }
      }
      red_pre<NR, 1u>(rv, rc);
      __syncthreads();
      red_post<NR, 1u>(rv, rc);
      const float r1 = 1.f / rv[1];
      const float ws0 = rv[2] * r1, ws1 = rv[3] * r1;
      const float lamt = lam + lg2(rv[1]);
      if (tb == 0 && valid) {
        if (a.w_soft) {
          a.w_soft[bb * L + 2 * t] = ws0 * a.inv_kap;
          a.w_soft[bb * L + 2 * t + 1] = ws1 * a.inv_kap;
        }
        if (VJP && a.dW) {
          a.dW[bb * L + 2 * t] = (rv[VJP ? 5 : 0] - ws0 * rv[VJP ? 4 : 0]) * r1 * dws;
          a.dW[bb * L + 2 * t + 1] = (rv[VJP ? 6 : 0] - ws1 * rv[VJP ? 4 : 0]) * r1 * dws;
        }
      }
      if (DC && tb == 0) {
        sm_lam[t] = lamt;
        sm_xb[t] = fmaf(rv[VJP ? 4 : 0], r1, xbar);
        sm_cp[t] = cprev;
      }
      lam = lamt - dlG + mBt;
      dlG = floorf(rv[0]);
      if (VJP) {
        // E_p[X_t] = xbar + sum p X / sum p; X_{t+1} drops <g_t, w_soft_t>
        // (A's centring); it gains <g_{t+1}, w_{t+1}> at the top of the next step
        const float gw = fmaf(g1, ws1, g0 * ws0);
        xbar = fmaf(rv[VJP ? 4 : 0], r1, xbar) - gw;
        cprev = gw;
      }
    }

    // ---------------------------------------------------------------- S2
    // dCodebook: dc_a(s) = sum_t p_t(s) [g_{t,a} + (w_{t,a} - c_a(s)) (X_t(s) - E_p[X_t]) / T].
    // No recursion is left: each lane takes one tile column (16 states) at a
    // time over all steps, with its 32 codebook values and 32 accumulators in
    // registers; p_t(s) = 2^(G_t + h_t + H_t - lambda_t) from the (G, A) and
    // (H, B) histories with the exact lambda_t and E_p[X_t] recorded by S1.
    if constexpr (DC) {
      __syncthreads();  // S1's histories and per-step scalars
      const bool first = base == (int64_t)blockIdx.x * BPW;
      double* part = a.dc_part + slot * ((int64_t)2 << n);
#pragma unroll 1
      for (int i = 0; i < SGT; ++i) {
        const int m = tq + i * TQ;
        float c0[16], c1[16], acc0[16], acc1[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float cv[2];
          buf_ld<2>(cbk, voC1, (uint32_t)r * (uint32_t)GS * 8u + (uint32_t)i * tileC, cv);
          c0[r] = cv[0];
          c1[r] = cv[1];
          acc0[r] = 0.f;
          acc1[r] = 0.f;
        }
        // (G_t, A_t) entries r * NSG + m of the step: same address for the 16
        // lanes of a tile
        const uint32_t voGA = (uint32_t)bw * (uint32_t)N * (uint32_t)GS * 8u + (uint32_t)m * 8u;
        PairRows cw, cg;
        for (int64_t t = 0; t < N; ++t) {
          const bool reload = (t & 31) == 0;
          float w0, w1, g0, g1;
          pair_at(wb, t, L, lane_rows, reload, cw, w0, w1);
          pair_at(gb, t, L, lane_rows, reload, cg, g0, g1);
          w0 *= kap;
          w1 *= kap;
          const uint32_t soH = (uint32_t)t * hstep;
          float hu[2];
          buf_ld<2>(hist, voH, soH + (uint32_t)i * tileH, hu);
          const float hl = hu[0] - sm_lam[t];
          const float bq = hu[1] - sm_xb[t] - sm_cp[t];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            float ga[2];
            buf_ld<2>(hga, voGA, soH + (uint32_t)r * (uint32_t)NSG * 8u, ga);
            const float d0 = w0 - c0[r], d1 = w1 - c1[r];
            const float p = ex2(fmaf(-d1, d1, fmaf(-d0, d0, ga[0] + hl)));
            const float X = fmaf(g1, c1[r], fmaf(g0, c0[r], ga[1] + bq));
            const float pX = p * X * dws;
            acc0[r] = fmaf(pX, d0, fmaf(p, g0, acc0[r]));
            acc1[r] = fmaf(pX, d1, fmaf(p, g1, acc1[r]));
          }
        }
        if (valid) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int64_t s = (int64_t)r * GS + m * 16 + tl;
            // d0 above is w' - c' in scaled units: (w - c) X / T = (w' - c') X' / (kappa^2 T)
            part[2 * s] = (first ? 0.0 : part[2 * s]) + (double)acc0[r];
            part[2 * s + 1] = (first ? 0.0 : part[2 * s + 1]) + (double)acc1[r];
          }
        }
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Low-temperature VJP of the vector-emission trellis (T < 0.04).  As in the
// scalar trellis's fb_kernel_hp, G and H are double-float pairs (an fp32 hi
// word and an fp32 lo word) with the emission and the log-sum-exp in fp64;
// softmax weights and tangents stay fp32.  The hi words and the tangent
// ping-pong in LDS as (hi, tangent) pairs, the lo words in a per-slot global
// buffer, one barrier per step.  The codebook is unscaled here (cs = c,
// csT its transposed copy).  The backward tangent is centred on the
// reference codewords bref (the minimum-distortion path, which the posterior
// follows at low temperature), X is centred per state before the moment
// sums, and the forward tangent is centred on <g_t, w_soft_t> when read.
//   S0 backward: H, B; history entries (H hi, H lo, B, 0);
//   S1 forward:  G, A, marginals, w_soft, dW; with DC the (G hi, G lo, A, 0)
//                entries and the exact lambda_t, E_p[X_t], A centring;
//   S2 (DC):     dCodebook per state over all steps.
// ---------------------------------------------------------------------------
template <int NB, int SGMAX, int NT, bool DC>
__global__ void __launch_bounds__(NT) fbv_kernel_hp(FbvArgs a) {
  extern __shared__ float lds[];
  const int n = NB ? NB : a.n;
  const VecGeom q = vec_geom(n);
  const int GS = q.GS, NSG = q.NSG;
  const int SGT = NB ? SGMAX : a.sgt;
  const int TPB = 16 * NSG / SGT;
  const int TQ = TPB / 16;
  const int BPW = NT / TPB;
  const int tid = threadIdx.x;
  const int bw = BPW == 1 ? 0 : tid / TPB;
  const int tb = BPW == 1 ? tid : tid - bw * TPB;
  const int tq = tb >> 4, tl = tb & 15;
  const int64_t N = a.N, L = 2 * a.N;
  const double k2 = a.k2d;
  const float invT = a.invT;

  RedCtx rc;
  rc.width = TPB < 64 ? TPB : 64;
  rc.rw = TPB > 64 ? TPB / 64 : 1;
  rc.wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: a scalar
  float* const red0 = lds + (size_t)BPW * 4 * q.VSZ;  // [2 parities][waves][kRed] floats
  double* const redd = reinterpret_cast<double*>(red0 + 2 * (NT / 64) * kRed);  // [waves]
  rc.red = red0;
  float* const vec0 = lds + (size_t)bw * 4 * q.VSZ;
  float* const vec1 = vec0 + 2 * q.VSZ;

  const rsrc_t cbk = make_rsrc(a.cs, (uint32_t)8 << n);
  const rsrc_t cbkT = make_rsrc(a.csT, (uint32_t)8 << n);
  const uint32_t voC1 = ((uint32_t)tq * 16 + tl) * 8u;
  const uint32_t tileC = (uint32_t)TQ * 128u;
  const uint32_t voC0 = ((uint32_t)tq * 256 + tl) * 8u;
  const uint32_t tileCT = (uint32_t)TQ * 2048u;
  const uint32_t hstep = (uint32_t)GS * 16u;          // history bytes per step (4 floats per group)
  const uint32_t voH = (uint32_t)bw * (uint32_t)N * hstep + ((uint32_t)tq * 16 + tl) * 16u;
  const uint32_t tileH = (uint32_t)TQ * 16u * 16u;
  const bool lane_rows = TPB >= 64;

  for (int64_t base = (int64_t)blockIdx.x * BPW; base < a.B; base += (int64_t)gridDim.x * BPW) {
    const int64_t blk = base + bw;
    const bool valid = blk < a.B;
    const int64_t bb = valid ? blk : a.B - 1;
    const int64_t slot = (int64_t)blockIdx.x * BPW + bw;
    const int64_t slot0 = (int64_t)blockIdx.x * BPW;
    const float* wb = a.w + bb * L;
    const float* gb = a.g + bb * L;
    const float* rb = a.bref + bb * L;
    const rsrc_t hist = make_rsrc(a.hist + slot0 * N * GS * 4, (uint32_t)BPW * (uint32_t)N * hstep);
    const rsrc_t hga = make_rsrc(DC ? a.histGA + slot0 * N * GS * 4 : a.hist,
                                 DC ? (uint32_t)BPW * (uint32_t)N * hstep : 0u);
    float* xlo0 = a.xlo + slot * 2 * GS;
    float* xlo1 = xlo0 + GS;
    float* sm_mB = a.small + slot * 6 * N;   // shift applied to H_t
    float* sm_xb = sm_mB + N;                // dCodebook: E_p[X_t]
    float* sm_cp = sm_xb + N;                // dCodebook: centring of A_t
    double* sm_lam = reinterpret_cast<double*>(sm_mB + 4 * N);  // dCodebook: lambda_t

    // ---------------------------------------------------------------- S0
    for (int i = tb; i < 2 * q.VSZ; i += TPB) vec0[i] = 0.f;
    for (int i = tb; i < GS; i += TPB) xlo0[i] = 0.f;
    if (tb == 0) sm_mB[N - 1] = 0.f;
    __syncthreads();
    double shiftB = 0.0;
    double lam0 = 0.0;
    float xbar = 0.f;
    float dlag = 0.f;
    PairRows rw_, rg_, rr_;
    for (int64_t t = N - 1;; --t) {
      const int par = (int)((N - 1 - t) & 1);
      rc.red = red0 + par * (NT / 64) * kRed;
      float* cur = par ? vec1 : vec0;
      float* nxt = par ? vec0 : vec1;
      const float* xlo_r = par ? xlo1 : xlo0;
      float* xlo_w = par ? xlo0 : xlo1;
      const bool reload = t == N - 1 || (t & 31) == 31;
      float w0f, w1f, g0, g1, r0, r1;
      pair_at(wb, t, L, lane_rows, reload, rw_, w0f, w1f);
      pair_at(gb, t, L, lane_rows, reload, rg_, g0, g1);
      pair_at(rb, t, L, lane_rows, reload, rr_, r0, r1);
      const double w0 = (double)w0f, w1 = (double)w1f;
      const uint32_t soH = (uint32_t)t * hstep;
      const bool first = t == 0;
      double lm = -INFINITY;
      float ls = 0.f, ly = 0.f;
      float vmax[1] = {-INFINITY};
#pragma unroll 1
      for (int i = 0; i < SGT; ++i) {
        const int m = tq + i * TQ;
        float cc[32], hb[32], hl[16];
        row_codewords(cbkT, voC0, (uint32_t)i * tileCT, cc);
#pragma unroll
        for (int u4 = 0; u4 < 8; ++u4) {
          float t4[4];
          ld_vec<4>(cur + 2 * q.row(m) + 4 * u4, t4);
#pragma unroll
          for (int e = 0; e < 4; ++e) hb[4 * u4 + e] = t4[e];
        }
        ld_vec<16>(xlo_r + m * 16, hl);
        {
          float own[2];
          ld_vec<2>(cur + 2 * (q.row(m) + tl), own);
          const float ent[4] = {own[0], xlo_r[m * 16 + tl], own[1], 0.f};
          buf_st<4>(hist, voH, soH + (uint32_t)i * tileH, ent);
        }
        double x[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const double d0 = w0 - (double)cc[2 * u], d1 = w1 - (double)cc[2 * u + 1];
          x[u] = fma(-k2, fma(d0, d0, d1 * d1), (double)hb[2 * u] + (double)hl[u]);
        }
        const double M = max_of<16>(x);
        float s = 0.f, sy = 0.f;
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const float E = ex2((float)(x[u] - M));
          s += E;
          // first step: E_p[<g_0, c> + B_0]; otherwise the summand of B_{t-1},
          // <g_t, c - r_t> + B_t
          const float y = first ? fmaf(g1, cc[2 * u + 1], fmaf(g0, cc[2 * u], hb[2 * u + 1]))
                                : fmaf(g1, cc[2 * u + 1] - r1, fmaf(g0, cc[2 * u] - r0, hb[2 * u + 1]));
          sy = fmaf(E, y, sy);
        }
        if (first) {
          lse3_pair_d(lm, ls, ly, M, s, sy);
        } else {
          const double h = M + (double)lg2(s) - (double)dlag;
          float hi, lo;
          split_df(h, hi, lo);
          vmax[0] = fmaxf(vmax[0], hi);
          const float o[2] = {hi, sy * rcp(s)};
          st_vec<2>(nxt + 2 * q.col(tl, m), o);
          xlo_w[tl * NSG + m] = lo;
        }
        sg_fence();
      }
      if (first) {
        lse3d_pre(lm, ls, ly, rc, redd);
        __syncthreads();
        lse3d_post(lm, ls, ly, rc, redd);
        xbar = ly / ls;
        lam0 = lm + (double)lg2(ls);
        if (tb == 0 && valid && a.logZ)
          a.logZ[bb] = (float)((shiftB + lam0) * 0.69314718055994530942);
        __syncthreads();
        break;
      }
      shiftB += (double)dlag;
      if (tb == 0) sm_mB[t - 1] = dlag;
      red_pre<1, 1u>(vmax, rc);
      __syncthreads();
      red_post<1, 1u>(vmax, rc);
      dlag = floorf(vmax[0]);
    }

    // ---------------------------------------------------------------- S1
    for (int i = tb; i < 2 * q.VSZ; i += TPB) vec0[i] = 0.f;
    for (int i = tb; i < GS; i += TPB) xlo0[i] = 0.f;
    if constexpr (DC) {
      const float z[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
      for (int i = 0; i < SGT; ++i) buf_st<4>(hga, voH, (uint32_t)i * tileH, z);
    }
    __syncthreads();
    double lam_est = lam0;
    float cprev = 0.f;
    dlag = 0.f;
    float pH[4];
    buf_ld<4>(hist, voH, 0u, pH);
    for (int64_t t = 0; t < N; ++t) {
      const int par = (int)(t & 1);
      rc.red = red0 + par * (NT / 64) * kRed;
      float* cur = par ? vec1 : vec0;
      float* nxt = par ? vec0 : vec1;
      const float* xlo_r = par ? xlo1 : xlo0;
      float* xlo_w = par ? xlo0 : xlo1;
      const bool reload = (t & 31) == 0;
      float w0f, w1f, g0, g1, r0, r1;
      pair_at(wb, t, L, lane_rows, reload, rw_, w0f, w1f);
      pair_at(gb, t, L, lane_rows, reload, rg_, g0, g1);
      pair_at(rb, t, L, lane_rows, reload, rr_, r0, r1);
      const double w0 = (double)w0f, w1 = (double)w1f;
      if (t > 0) xbar = fmaf(g1, r1, fmaf(g0, r0, xbar));  // B_t no longer holds step t
      const double mBt = (double)sm_mB[t];
      const uint32_t soH = (uint32_t)t * hstep;
      float rv[7] = {-INFINITY, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
      for (int i = 0; i < SGT; ++i) {
        const int m = tq + i * TQ;
        const float hu[4] = {pH[0], pH[1], pH[2], pH[3]};
        float c0[16], c1[16], Ar[16];
        double G[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float cv[2], ga[2];
          buf_ld<2>(cbk, voC1, (uint32_t)r * (uint32_t)GS * 8u + (uint32_t)i * tileC, cv);
          c0[r] = cv[0];
          c1[r] = cv[1];
          ld_vec<2>(cur + 2 * q.col(r, m), ga);
          G[r] = (double)ga[0] + (double)xlo_r[r * NSG + m];
          Ar[r] = ga[1] - cprev;
        }
        {
          const bool last = i + 1 >= SGT;
          const int64_t tn = last && t + 1 < N ? t + 1 : t;
          buf_ld<4>(hist, voH, (uint32_t)tn * hstep + (last ? 0u : (uint32_t)(i + 1) * tileH), pH);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const double d0 = w0 - (double)c0[r], d1 = w1 - (double)c1[r];
          G[r] = fma(-k2, fma(d0, d0, d1 * d1), G[r]);
        }
        const double M = max_of<16>(G);
        // X is centred per state before the sums (at low T uncentred moments
        // cancel only to X's rounding, amplified by 1/T)
        const float bx = hu[2] - xbar;
        float s = 0.f, e0 = 0.f, e1 = 0.f, sx = 0.f, sx0 = 0.f, sx1 = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float E = ex2((float)(G[r] - M));
          const float X = fmaf(g1, c1[r], fmaf(g0, c0[r], Ar[r])) + bx;
          const float EX = E * X;
          s += E;
          e0 = fmaf(E, c0[r], e0);
          e1 = fmaf(E, c1[r], e1);
          sx += EX;
          sx0 = fmaf(EX, c0[r], sx0);
          sx1 = fmaf(EX, c1[r], sx1);
        }
        const double gout = M + (double)lg2(s) - (double)dlag;
        float hi, lo;
        split_df(gout, hi, lo);
        rv[0] = fmaxf(rv[0], hi);
        const float f = ex2((float)(M + ((double)hu[0] + (double)hu[1]) - lam_est));
        rv[1] = fmaf(f, s, rv[1]);
        rv[2] = fmaf(f, e0, rv[2]);
        rv[3] = fmaf(f, e1, rv[3]);
        rv[4] = fmaf(f, sx, rv[4]);
        rv[5] = fmaf(f, sx0, rv[5]);
        rv[6] = fmaf(f, sx1, rv[6]);
        const float An = fmaf(sx, rcp(s), -bx);  // E-weighted mean of <g_t, c> + A_t
        if (t < N - 1) {
          const float o[2] = {hi, An};
          st_vec<2>(nxt + 2 * (q.row(m) + tl), o);
          xlo_w[m * 16 + tl] = lo;
          if constexpr (DC) {
            const float ent[4] = {hi, lo, An, 0.f};
            buf_st<4>(hga, voH, soH + hstep + (uint32_t)i * tileH, ent);
          }
        }
        sg_fence();
      }
      red_pre<7, 1u>(rv, rc);
      __syncthreads();
      red_post<7, 1u>(rv, rc);
      const float r1v = 1.f / rv[1];
      const float ws0 = rv[2] * r1v, ws1 = rv[3] * r1v;
      const double lamt = lam_est + (double)lg2(rv[1]);
      const float xbe = fmaf(rv[4], r1v, xbar);
      if (tb == 0) {
        if (DC) {
          sm_lam[t] = lamt;
          sm_xb[t] = xbe;
          sm_cp[t] = cprev;
        }
        if (valid) {
          if (a.w_soft) {
            a.w_soft[bb * L + 2 * t] = ws0;
            a.w_soft[bb * L + 2 * t + 1] = ws1;
          }
          if (a.dW) {
            a.dW[bb * L + 2 * t] = (rv[5] - ws0 * rv[4]) * r1v * invT;
            a.dW[bb * L + 2 * t + 1] = (rv[6] - ws1 * rv[4]) * r1v * invT;
          }
        }
      }
      lam_est = lamt - (double)dlag + mBt;
      dlag = floorf(rv[0]);
      cprev = fmaf(g1, ws1, g0 * ws0);
      xbar = xbe - cprev;
    }

    // ---------------------------------------------------------------- S2
    if constexpr (DC) {
      __syncthreads();
      const bool first = base == (int64_t)blockIdx.x * BPW;
      double* part = a.dc_part + slot * ((int64_t)2 << n);
#pragma unroll 1
      for (int i = 0; i < SGT; ++i) {
        const int m = tq + i * TQ;
        float c0[16], c1[16], acc0[16], acc1[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float cv[2];
          buf_ld<2>(cbk, voC1, (uint32_t)r * (uint32_t)GS * 8u + (uint32_t)i * tileC, cv);
          c0[r] = cv[0];
          c1[r] = cv[1];
          acc0[r] = 0.f;
          acc1[r] = 0.f;
        }
        const uint32_t voGA = (uint32_t)bw * (uint32_t)N * hstep + (uint32_t)m * 16u;
        PairRows cw, cg;
        for (int64_t t = 0; t < N; ++t) {
          const bool reload = (t & 31) == 0;
          float w0f, w1f, g0, g1;
          pair_at(wb, t, L, lane_rows, reload, cw, w0f, w1f);
          pair_at(gb, t, L, lane_rows, reload, cg, g0, g1);
          const double w0 = (double)w0f, w1 = (double)w1f;
          const uint32_t soH = (uint32_t)t * hstep;
          float hu[4];
          buf_ld<4>(hist, voH, soH + (uint32_t)i * tileH, hu);
          const double hl = ((double)hu[0] + (double)hu[1]) - sm_lam[t];
          const float bq = hu[2] - sm_xb[t] - sm_cp[t];
#pragma unroll 4
          for (int r = 0; r < 16; ++r) {
            float ga[4];
            buf_ld<4>(hga, voGA, soH + (uint32_t)r * (uint32_t)NSG * 16u, ga);
            const double d0 = w0 - (double)c0[r], d1 = w1 - (double)c1[r];
            const float p = ex2((float)(fma(-k2, fma(d0, d0, d1 * d1), (double)ga[0] + (double)ga[1]) + hl));
            const float X = fmaf(g1, c1[r], fmaf(g0, c0[r], ga[2] + bq));
            const float pX = p * X * invT;
            acc0[r] = fmaf(pX, w0f - c0[r], fmaf(p, g0, acc0[r]));
            acc1[r] = fmaf(pX, w1f - c1[r], fmaf(p, g1, acc1[r]));
          }
        }
        if (valid) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int64_t st = (int64_t)r * GS + m * 16 + tl;
            part[2 * st] = (first ? 0.0 : part[2 * st]) + (double)acc0[r];
            part[2 * st + 1] = (first ? 0.0 : part[2 * st + 1]) + (double)acc1[r];
          }
        }
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Min-sum decode (paper Sec. 3.2) on the vector-emission trellis, fp64 path
// metrics: Mn_{t+1}(m * 16 + u) = min_r [d_t(r, m, u) + Mn_t(r * NSG + m)],
// d_t(s) = (w_t0 - c_0(s))^2 + (w_t1 - c_1(s))^2 (each square rounded, then
// added in component order), the winning r (smallest on ties) kept per
// (t, group).  Same tile layout as the forward sweep of fbv_kernel.
// ---------------------------------------------------------------------------
template <int NB, int SGMAX, int NT>
__global__ void __launch_bounds__(NT) vitv_kernel(VitvArgs a) {
  extern __shared__ double ldsd[];
  const int n = NB ? NB : a.n;
  const VecGeom q = vec_geom(n);
  const int GS = q.GS, NSG = q.NSG;
  const int SGT = NB ? SGMAX : a.sgt;
  const int TPB = 16 * NSG / SGT;
  const int TQ = TPB / 16;
  const int BPW = NT / TPB;
  const int tid = threadIdx.x;
  const int bw = tid / TPB;
  const int tb = tid - bw * TPB;
  const int tq = tb >> 4, tl = tb & 15;
  const int lane = tid & 63, wave = tid >> 6;
  const int width = TPB < 64 ? TPB : 64;
  const int rw = TPB > 64 ? TPB / 64 : 1;
  const int64_t N = a.N, L = 2 * a.N;
  double* mv0 = ldsd + (size_t)bw * 2 * q.VSZ;
  double* mv1 = mv0 + q.VSZ;
  double* redv = ldsd + (size_t)BPW * 2 * q.VSZ;       // [waves]
  int* redi = reinterpret_cast<int*>(redv + NT / 64);   // [waves]
  const float2* c2 = reinterpret_cast<const float2*>(a.c);

  for (int64_t base = (int64_t)blockIdx.x * BPW; base < a.B; base += (int64_t)gridDim.x * BPW) {
    const int64_t blk = base + bw;
    const bool valid = blk < a.B;
    const int64_t bb = valid ? blk : a.B - 1;
    const int64_t slot = (int64_t)blockIdx.x * BPW + bw;
    const float* wb = a.w + bb * L;
    uint8_t* bp = a.bp + slot * N * GS;

    for (int i = tb; i < q.VSZ; i += TPB) mv0[i] = 0.0;
    __syncthreads();
    double bestv = INFINITY;
    int besti = 0x7fffffff;
    for (int64_t t = 0; t < N; ++t) {
      double* cur = (t & 1) ? mv1 : mv0;
      double* nxt = (t & 1) ? mv0 : mv1;
      const double w0 = (double)wb[2 * t], w1 = (double)wb[2 * t + 1];
      // the step's winning digits, one byte per tile, stored after the tile
      // loop: a store between two tiles would make the next tile's codebook
      // loads wait for it (loads and stores retire in order)
      uint64_t digs = 0;
#pragma unroll 1
      for (int i = 0; i < SGT; ++i) {
        {
          const int m = tq + i * TQ;
          double best = 0.0;
          int br = 0;
#pragma unroll 4
          for (int r = 0; r < 16; ++r) {
            const int s = r * GS + m * 16 + tl;
            const float2 cv = c2[s];
            const double d0 = w0 - (double)cv.x, d1 = w1 - (double)cv.y;
            const double e = __dadd_rn(__dmul_rn(d0, d0), __dmul_rn(d1, d1));
            const double v = __dadd_rn(e, cur[q.col(r, m)]);
            if (t < N - 1) {
              if (r == 0 || v < best) {
                best = v;
                br = r;
              }
            } else if (v < bestv || (v == bestv && s < besti)) {
              bestv = v;
              besti = s;
            }
          }
          if (t < N - 1) {
            nxt[(q.row(m) + tl)] = best;
            digs |= (uint64_t)br << (8 * i);
          }
        }
      }
      if (t < N - 1) {
#pragma unroll
        for (int i = 0; i < SGMAX; ++i)
          if (i < SGT) bp[(t + 1) * GS + (tq + i * TQ) * 16 + tl] = (uint8_t)(digs >> (8 * i));
      }
      __syncthreads();
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
      for (int k = 1; k < rw; ++k) {
        const double ov = redv[first + k];
        const int oi = redi[first + k];
        if (ov < bestv || (ov == bestv && oi < besti)) {
          bestv = ov;
          besti = oi;
        }
      }
    }
    if (tb == 0 && valid) {
      int32_t* st = a.states + bb * N;
      float* wh = a.w_hard ? a.w_hard + bb * L : nullptr;
      // (non-finite inputs leave no state below +inf: start from state 0)
      int s = (unsigned)besti < (unsigned)(GS * 16) ? besti : 0;
      st[N - 1] = s;
      if (wh) {
        wh[2 * (N - 1)] = a.c[2 * s];
        wh[2 * (N - 1) + 1] = a.c[2 * s + 1];
      }
      for (int64_t t = N - 1; t >= 1; --t) {
        const int v = s >> 4;
        const int r = bp[t * GS + v];
        s = r * GS + v;
        st[t - 1] = s;
        if (wh) {
          wh[2 * (t - 1)] = a.c[2 * s];
          wh[2 * (t - 1) + 1] = a.c[2 * s + 1];
        }
      }
    }
    __syncthreads();
  }
}

// Scaled codebook of the vector-emission kernels in two layouts: cs[s] =
// kappa c(s) (2-vectors, state order) and csT[(s mod GS) * 16 + s / GS], the
// transposed copy read by the backward sweep.
__global__ void scale_vec_kernel(const float* c, float kap, float* cs, float* csT, int n) {
  const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= ((int64_t)1 << n)) return;
  const int64_t gs = (int64_t)1 << (n - 4);
  const float c0 = c[2 * s] * kap, c1 = c[2 * s + 1] * kap;
  cs[2 * s] = c0;
  cs[2 * s + 1] = c1;
  const int64_t j = (s & (gs - 1)) * 16 + (s >> (n - 4));
  csT[2 * j] = c0;
  csT[2 * j + 1] = c1;
}

}  // namespace
}  // namespace bcjr
