// bcjr_pruned_kernels.h -- the low-temperature VJP at S = 65536, k = 2 over
// the states that carry the posterior.
//
// At low T the posterior of a block lives on a few states per step: those
// whose best path lies within a margin of the block's best path (the
// min-sum max-marginal, Sec. 3.2's recursion run from both ends).  Every
// path through a state outside that window weighs at most e^{-margin}
// relative to the best one, so dropping those states changes w_soft, logZ,
// dW and dCodebook by far less than fp32 resolves (a margin of 30 nats
// leaves errors of ~1e-10 to 1e-8 against the full recursion).  Three launches per
// chunk of blocks:
//
//   mm_back_kernel   backward min-sum over all states (fp32, group form):
//                    per step the backward metric of every group above the
//                    step's minimum, coded in one byte (rounded down, so the
//                    window test below is conservative), and the block's best
//                    path cost;
//   mm_fwd_kernel    forward min-sum over all states: a state is kept when its
//                    forward metric plus the stored backward bound lies within
//                    the window; one bit per state and step;
//   pruned_sp_kernel one wave per block: Eqs. alpha and beta, the marginals
//                    (Eq. marginal), w_soft (Eq. soft-codeword), logZ and the
//                    VJP (dW, and dCodebook added into an fp64 accumulator)
//                    in fp64 over the kept states only, looked up through
//                    per-step rank tables.
//
// State s = (j, sg, u) = j * 2^14 + sg * 4 + u.  The min-sum kernels give
// thread tb the super-groups sg = tb + i * 1024 (i < 4); the kept-state bits
// of a step are 1024 words of 64 bits, word tb holding bit i * 16 + j * 4 + u.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bcjr_device.h"

namespace bcjr {

struct PrArgs {
  const float* w;       // [B, L]
  const float* g;       // [B, L] upstream gradient
  const float* c;       // [S] codebook
  int64_t B, L;
  int64_t b0;           // first block of this chunk
  int64_t nblk;         // blocks in this chunk (one slot each)
  double T;
  float theta;          // the window in squared-distortion units: 2 T margin
  float qscale;         // 16 / theta
  uint8_t* q;           // [slots][L][S/4] backward bound above the step minimum (bound_code)
  float* hmin;          // [slots][L] the step minimum of the backward metric
  float* best;          // [slots] the block's best path cost
  uint64_t* bm;         // [slots][L][1024] kept-state bits
  int64_t ecap;         // kept state-steps a slot can hold
  double* ent;          // [slots][2][ecap] per kept state-step log alpha and A, then log beta and B
  double* dc;           // [S] fp64 dCodebook accumulator, or null
  float* w_soft;        // [B, L] or null
  float* logZ;          // [B] or null
  float* dW;            // [B, L] or null
  int32_t* flags;       // [B]: set to 1 for a block this path does not finish
};

namespace pr {
constexpr int NT = 1024;          // min-sum kernels: threads per block
constexpr int GS = 1 << 14;       // groups
constexpr int NSG = 1 << 12;      // super-groups
constexpr int SGT = NSG / NT;     // super-groups per thread
constexpr int K = 4;
constexpr int NW = NT / 64;
constexpr int SP_WAVES = 4;       // pruned_sp_kernel: one block per wave
constexpr int WORDS = NT;         // kept-state words per step
constexpr size_t kMinSumLds = (size_t)2 * GS * sizeof(float) + (size_t)3 * NW * sizeof(float) +
                              (size_t)256 * sizeof(float);  // (the forward sweep's bound values)
constexpr size_t kSpLdsPerWave = (size_t)WORDS * sizeof(uint64_t) + (size_t)WORDS * sizeof(uint32_t) +
                                  (size_t)1024 * sizeof(uint32_t);
constexpr size_t kSpLds = kSpLdsPerWave * SP_WAVES;

// The byte code of a backward bound z >= 0 in units of window / 16: codes
// below 128 are z rounded down; from 128 on, z's binary exponent e >= 7 and
// its top three mantissa bits m: 128 + 8 (e - 7) + m, standing for
// 2^e (1 + m / 8), the largest such value not above z (up to ~5e5 windows).
// Blocks far outside the codebook's range have future costs spread over
// thousands of windows; a code that saturated at a few windows would keep
// most of their states.
//
// The exponent code is z's bits above bit 20 (8 x the biased exponent
// e + 127, plus m) minus 8 x 134 - 128 = 944.  Below z = 128 it exceeds
// floor(z) (it is 8 e + 72 + m there), from 128 on it is at most floor(z),
// so the code is the smaller of the two, with floor(z) capped at 255 (a NaN
// codes as 255).  Its value back is (code + 944) << 20 as a float.
__device__ __forceinline__ uint32_t bound_code(float z) {
  const uint32_t lin = (uint32_t)fminf(z, 255.f);
  const uint32_t ex = (__float_as_uint(z) >> 20) - 944u;
  return lin < ex ? lin : ex;
}

__device__ __forceinline__ float bound_value(uint32_t q) {
  return q < 128u ? (float)q : __uint_as_float((q + 944u) << 20);
}

__device__ __forceinline__ float wave_min(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fminf(v, __shfl_xor(v, o));
  return v;
}

// Wave reductions by DPP lane permutations within each 16-lane row, then the
// four row results read from lanes 0, 16, 32, 48 (or 15, 31, 47, 63) and
// combined in a fixed order: no LDS round trip, and every lane gets the
// same bits.  Called in wave-uniform control flow (all 64 lanes active).
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, true);
}

template <int CTRL>
__device__ __forceinline__ double dpp_d(double v) {
  const long long b = __double_as_longlong(v);
  const int lo = dpp_i<CTRL>((int)b), hi = dpp_i<CTRL>((int)(b >> 32));
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

__device__ __forceinline__ double readlane_d(double v, int l) {
  const long long b = __double_as_longlong(v);
  const int lo = __builtin_amdgcn_readlane((int)b, l), hi = __builtin_amdgcn_readlane((int)(b >> 32), l);
  return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

__device__ __forceinline__ double wave_sum_d(double v) {
  v += dpp_d<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_d<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_d<0x141>(v);  // row_half_mirror
  v += dpp_d<0x140>(v);  // row_mirror: every lane holds its row's sum
  return (readlane_d(v, 0) + readlane_d(v, 16)) + (readlane_d(v, 32) + readlane_d(v, 48));
}

// exclusive prefix over the wave's lanes, and the wave's total
__device__ __forceinline__ int wave_excl_scan(int v, int lane, int& total) {
  int x = v;
  x += dpp_i<0x111>(x);  // row_shr:1 (lanes without a source add 0)
  x += dpp_i<0x112>(x);  // row_shr:2
  x += dpp_i<0x114>(x);  // row_shr:4
  x += dpp_i<0x118>(x);  // row_shr:8: inclusive prefix within the row
  const int r0 = __builtin_amdgcn_readlane(x, 15), r1 = __builtin_amdgcn_readlane(x, 31),
            r2 = __builtin_amdgcn_readlane(x, 47), r3 = __builtin_amdgcn_readlane(x, 63);
  const int row = lane >> 4;
  x += (row >= 1 ? r0 : 0) + (row >= 2 ? r1 : 0) + (row >= 3 ? r2 : 0);
  total = r0 + r1 + r2 + r3;
  return x - v;
}

// running log-sum-exp with a payload: exp(m) * s is the sum, y / s the
// weighted mean of the payload
__device__ __forceinline__ void lse_add(double& m, double& s, double& y, double v, double yv) {
  if (!(v > -INFINITY)) return;
  if (!(m > -INFINITY)) {  // the first term: no exponential
    m = v;
    s = 1.0;
    y = yv;
    return;
  }
  if (v > m) {
    const double r = exp(m - v);
    s = s * r + 1.0;
    y = y * r + yv;
    m = v;
  } else {
    const double r = exp(v - m);
    s += r;
    y += r * yv;
  }
}

__device__ __forceinline__ void lse_merge(double& m, double& s, double& y, double mo, double so, double yo) {
  if (!(mo > -INFINITY)) return;
  if (!(m > -INFINITY)) {
    m = mo; s = so; y = yo;
    return;
  }
  if (mo > m) {
    const double r = exp(m - mo);
    s = s * r + so;
    y = y * r + yo;
    m = mo;
  } else {
    const double r = exp(mo - m);
    s += so * r;
    y += yo * r;
  }
}

// The entries and LDS tables of a block are written and read by its one
// wave only, whose memory operations take effect in program order: a fence
// at wavefront scope keeps the compiler from reordering them and emits no
// wait.
__device__ __forceinline__ void wave_fence() { __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront"); }

// state of bit `bit` of word `q`
__device__ __forceinline__ int state_of(int q, int bit) {
  const int i = bit >> 4, j = (bit >> 2) & 3, u = bit & 3;
  return (j << 14) | ((q + (i << 10)) << 2) | u;
}

}  // namespace pr

// Backward min-sum: Hm_{t-1}(j * 2^12 + sg) = min_b [ (w_t - c(j, sg, b))^2 + Hm_t(sg * 4 + b) ],
// Hm_{L-1} = 0; the step's own inputs Hm_t(sg * 4 + b) are what the forward
// window test needs for the states (., sg, b) of step t.
__global__ void __launch_bounds__(pr::NT) mm_back_kernel(PrArgs a) {
  using namespace pr;
  extern __shared__ float lds_mm[];
  float* red = lds_mm + 2 * GS;  // [2][NW] step minima, then [NW] best
  const int tb = threadIdx.x, lane = tb & 63, wave = tb >> 6;
  const int64_t L = a.L;
  const rsrc_t cbk = make_rsrc(a.c, (uint32_t)GS * K * 4u);
  const uint32_t voK = (uint32_t)tb * K * 4u;
  // this thread's 64 codewords, the same at every step and block
  float cb[SGT][K][K];
#pragma unroll
  for (int i = 0; i < SGT; ++i)
#pragma unroll
    for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, (uint32_t)(j * GS + i * NT * K) * 4u, cb[i][j]);
  for (int64_t sl = blockIdx.x; sl < a.nblk; sl += gridDim.x) {
    const int64_t bb = a.b0 + sl;
    const float* wb = a.w + bb * L;
    const rsrc_t qr = make_rsrc(a.q + sl * L * (int64_t)GS, (uint32_t)(L * GS));
    float* hmin = a.hmin + sl * L;
    float* p0 = lds_mm + ((L - 1) & 1) * GS;
    for (int x = tb; x < GS; x += NT) p0[x] = 0.f;
    __syncthreads();
    float bestv = INFINITY;
    for (int64_t t = L - 1; t >= 0; --t) {
      const float* pin = lds_mm + (t & 1) * GS;
      float* pout = lds_mm + ((t + 1) & 1) * GS;
      const float wt = ld_uniform(wb, t);
      float in[SGT][K];
      float mn = INFINITY;
#pragma unroll
      for (int i = 0; i < SGT; ++i) {
        const float4 v = *reinterpret_cast<const float4*>(pin + (tb + i * NT) * K);
        in[i][0] = v.x; in[i][1] = v.y; in[i][2] = v.z; in[i][3] = v.w;
        mn = fminf(mn, fminf(fminf(v.x, v.y), fminf(v.z, v.w)));
      }
#pragma unroll
      for (int i = 0; i < SGT; ++i)
#pragma unroll
        for (int j = 0; j < K; ++j) {
          float m = INFINITY;
#pragma unroll
          for (int b = 0; b < K; ++b) {
            const float d = wt - cb[i][j][b];
            m = fminf(m, fmaf(d, d, in[i][b]));
          }
          // (at t = 0 these are the best path costs through each state;
          // the half no later step reads holds them)
          pout[j * NSG + tb + i * NT] = m;
        }
      mn = wave_min(mn);
      float* rd = red + (t & 1) * NW;
      if (lane == 0) rd[wave] = mn;
      __syncthreads();
      float hm = rd[0];
#pragma unroll
      for (int x = 1; x < NW; ++x) hm = fminf(hm, rd[x]);
      // the bound above the step minimum, coded and rounded down
#pragma unroll
      for (int i = 0; i < SGT; ++i) {
        uint32_t word = 0;
#pragma unroll
        for (int b = 0; b < K; ++b) word |= bound_code((in[i][b] - hm) * a.qscale) << (8 * b);  // (in >= hm)
        __builtin_amdgcn_raw_buffer_store_b32(word, qr, (int)((uint32_t)(tb + i * NT) * K), (int)(t * GS), 0);
      }
      if (tb == 0) hmin[t] = hm;
    }
    // (the step-0 rows were written before that step's barrier)
    for (int x = tb; x < GS; x += NT) bestv = fminf(bestv, lds_mm[GS + x]);
    bestv = wave_min(bestv);
    float* rb = red + 2 * NW;
    if (lane == 0) rb[wave] = bestv;
    __syncthreads();
    if (tb == 0) {
      float v = rb[0];
      for (int x = 1; x < NW; ++x) v = fminf(v, rb[x]);
      a.best[sl] = v;
    }
    __syncthreads();
  }
}

// Forward min-sum with the window test: F_t(s) = (w_t - c(s))^2 + Gm_t(s >> 2),
// Gm_{t+1}(sg * 4 + u) = min_j F_t(j, sg, u), Gm_0 = 0; state s is kept at
// step t when F_t(s) + hmin_t + (its coded bound) theta / 16 <= best + theta.
__global__ void __launch_bounds__(pr::NT) mm_fwd_kernel(PrArgs a) {
  using namespace pr;
  extern __shared__ float lds_mm[];
  const int tb = threadIdx.x;
  const int64_t L = a.L;
  const float step = a.theta * (1.f / 16.f);
  // the distortion each byte code stands for, the same at every step
  float* bval = lds_mm + 2 * GS + 3 * NW;
  for (int x = tb; x < 256; x += NT) bval[x] = bound_value((uint32_t)x) * step;
  const rsrc_t cbk = make_rsrc(a.c, (uint32_t)GS * K * 4u);
  const uint32_t voK = (uint32_t)tb * K * 4u;
  float cb[SGT][K][K];  // as in the backward sweep
#pragma unroll
  for (int i = 0; i < SGT; ++i)
#pragma unroll
    for (int j = 0; j < K; ++j) buf_ld<K>(cbk, voK, (uint32_t)(j * GS + i * NT * K) * 4u, cb[i][j]);
  for (int64_t sl = blockIdx.x; sl < a.nblk; sl += gridDim.x) {
    const int64_t bb = a.b0 + sl;
    const float* wb = a.w + bb * L;
    const rsrc_t qr = make_rsrc(a.q + sl * L * (int64_t)GS, (uint32_t)(L * GS));
    const float* hmin = a.hmin + sl * L;
    uint64_t* bm = a.bm + sl * L * (int64_t)WORDS;
    // (the window is widened by a few fp32 roundings of the path costs)
    const float best = ld_uniform(a.best, sl);
    const float lim = best + a.theta + 1e-5f * (fabsf(best) + a.theta);
    for (int x = tb; x < GS; x += NT) lds_mm[x] = 0.f;
    // the step's bound words, weight and minimum are fetched one step ahead
    uint32_t qn[SGT];
#pragma unroll
    for (int i = 0; i < SGT; ++i)
      qn[i] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(qr, (int)((uint32_t)(tb + i * NT) * K), 0, 0);
    float wn = ld_uniform(wb, 0), hn = ld_uniform(hmin, 0);
    __syncthreads();
    for (int64_t t = 0; t < L; ++t) {
      const float* pin = lds_mm + (t & 1) * GS;
      float* pout = lds_mm + ((t + 1) & 1) * GS;
      const float wt = wn;
      const float lmh = lim - hn;
      uint32_t qc[SGT];
#pragma unroll
      for (int i = 0; i < SGT; ++i) qc[i] = qn[i];
      {
        const int64_t tn = t + 1 < L ? t + 1 : t;
#pragma unroll
        for (int i = 0; i < SGT; ++i)
          qn[i] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(qr, (int)((uint32_t)(tb + i * NT) * K),
                                                                 (int)(tn * GS), 0);
        wn = ld_uniform(wb, tn);
        hn = ld_uniform(hmin, tn);
      }
      uint32_t mask[2] = {0u, 0u};
#pragma unroll
      for (int i = 0; i < SGT; ++i) {
        const int sg = tb + i * NT;
        float gin[K];
#pragma unroll
        for (int j = 0; j < K; ++j) gin[j] = pin[j * NSG + sg];
        const uint32_t qw = qc[i];
        float mo[K];
        uint32_t bits = 0;
#pragma unroll
        for (int u = 0; u < K; ++u) {
          // (the forward cost a kept state may reach: one subtraction for
          // the four states of this bound, inside the window's widening)
          const float thr = lmh - bval[(qw >> (8 * u)) & 0xFFu];
          float m = INFINITY;
#pragma unroll
          for (int j = 0; j < K; ++j) {
            const float d = wt - cb[i][j][u];
            const float f = fmaf(d, d, gin[j]);
            m = fminf(m, f);
            bits |= (f <= thr ? 1u : 0u) << (j * 4 + u);
          }
          mo[u] = m;
        }
        // (after the last step this row goes to the buffer half no later
        // step reads; the next block clears it behind the step's barrier)
        *reinterpret_cast<float4*>(pout + sg * K) = make_float4(mo[0], mo[1], mo[2], mo[3]);
        pin_u(bits);
        mask[i >> 1] |= bits << (16 * (i & 1));
        sg_fence();
      }
      *reinterpret_cast<uint2*>(bm + t * WORDS + tb) = make_uint2(mask[0], mask[1]);
      __syncthreads();
    }
  }
}

// Sum-product and VJP over the kept states, one block per wave, fp64.
// Forward: log alpha_t(s) = h_t(s) + LSE over kept predecessors p of
// log alpha_{t-1}(p), A_t(s) = g_t c(s) + their alpha-weighted mean of
// A_{t-1}; backward: log beta_t(s) = LSE over kept successors d of
// h_{t+1}(d) + log beta_{t+1}(d), B_t(s) = the weighted mean of
// g_{t+1} c(d) + B_{t+1}(d); then with P = alpha beta / Z and
// X = A + B - E[F]: w_soft_t = sum P c, dW_t = sum P (c - w_soft_t) X / T,
// dc(s) += P (g_t + (w_t - c(s)) X / T).  A step's kept states are ranked in
// word order (their entry index), listed in LDS in rounds of LIST and taken
// by the lanes in turn; the neighbouring step's words and rank table stay in
// LDS for the predecessor (successor) lookups, the next step's words are
// fetched one step ahead.  A block whose kept state-steps exceed the slot,
// or whose Z misses the best path, is marked in `flags` and left to the
// dense kernel.
namespace pr {
constexpr int LIST = 1024;
constexpr int WPL = WORDS / 64;  // words per lane

// this lane's words of a step into registers
__device__ __forceinline__ void fetch_step(const uint64_t* src, int lane, uint64_t (&wd)[WPL]) {
#pragma unroll
  for (int r = 0; r < WPL; ++r) wd[r] = src[lane * WPL + r];
}

// the step's count, and this lane's first rank
__device__ __forceinline__ int step_ranks(const uint64_t (&wd)[WPL], int lane, int& run) {
  int cnt = 0;
#pragma unroll
  for (int r = 0; r < WPL; ++r) cnt += __popcll(wd[r]);
  int total;
  run = wave_excl_scan(cnt, lane, total);
  return total;
}

// kept states of ranks [r0, r0 + LIST) into list[rank - r0]
__device__ __forceinline__ void list_round(const uint64_t (&wd)[WPL], int lane, int run, int r0, uint32_t* list) {
  int rk = run;
#pragma unroll
  for (int r = 0; r < WPL; ++r) {
    const int n = __popcll(wd[r]);
    if (rk + n > r0 && rk < r0 + LIST) {
      uint64_t x = wd[r];
      int k = rk;
      while (x) {
        const int bit = __builtin_ctzll(x);
        x &= x - 1ull;
        if (k >= r0 && k < r0 + LIST) list[k - r0] = (uint32_t)state_of(lane * WPL + r, bit);
        ++k;
      }
    }
    rk += n;
  }
}

// this step's words and ranks become the neighbour tables of the next step
__device__ __forceinline__ void keep_tables(const uint64_t (&wd)[WPL], int lane, int run, uint64_t* nbm, uint32_t* npre) {
  int rk = run;
#pragma unroll
  for (int r = 0; r < WPL; ++r) {
    nbm[lane * WPL + r] = wd[r];
    npre[lane * WPL + r] = (uint32_t)rk;
    rk += __popcll(wd[r]);
  }
}

// (word, bit) of state s
__device__ __forceinline__ void pos_of(int s, int& q, int& bit) {
  const int j = s >> 14, sg = (s >> 2) & (NSG - 1), u = s & 3;
  q = sg & (NT - 1);
  bit = (sg >> 10) * 16 + j * 4 + u;
}

// log alpha and A of the kept predecessors (s >> 2) + j 2^14 of state s
// (one word, bits ip * 16 + j * 4 + up); -inf and 0 for the others
__device__ __forceinline__ void pred_vals(int s, const uint64_t* nbm, const uint32_t* npre,
                                          int64_t base_prev, const double* la, const double* aa,
                                          double (&v)[K], double (&y)[K]) {
  int qp, b0;
  pos_of(s >> 2, qp, b0);  // (j = 0)
  const uint64_t word = nbm[qp];
  const uint32_t pr0 = npre[qp];
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const int pb = b0 + j * 4;
    v[j] = -INFINITY;
    y[j] = 0.0;
    if ((word >> pb) & 1ull) {
      const int64_t ep = base_prev + pr0 + __popcll(word & ((1ull << pb) - 1ull));
      v[j] = la[ep];
      y[j] = aa[ep];
    }
  }
}

// h_{t+1}(d) + log beta_{t+1}(d) and g_{t+1} c(d) + B_{t+1}(d) of the kept
// successors d = (s mod 2^14) * 4 + b (one word, bits id * 16 + jd * 4 + b);
// -inf and 0 for the others
__device__ __forceinline__ void succ_vals(int s, const uint64_t* nbm, const uint32_t* npre,
                                          int64_t base_next, const double* la, const double* aa,
                                          const float* c, double wn, double gn, double i2T,
                                          double (&v)[K], double (&y)[K]) {
  const int s14 = s & (GS - 1);
  int qd, b0;
  pos_of(s14 << 2, qd, b0);  // (b = 0)
  const uint64_t word = nbm[qd];
  const uint32_t pr0 = npre[qd];
  const float4 c4 = *reinterpret_cast<const float4*>(c + (s14 << 2));
  const float cd[K] = {c4.x, c4.y, c4.z, c4.w};
#pragma unroll
  for (int b = 0; b < K; ++b) {
    const int nb = b0 + b;
    v[b] = -INFINITY;
    y[b] = 0.0;
    if ((word >> nb) & 1ull) {
      const int64_t ed = base_next + pr0 + __popcll(word & ((1ull << nb) - 1ull));
      const double cdb = (double)cd[b];
      v[b] = -(wn - cdb) * (wn - cdb) * i2T + la[ed];
      y[b] = gn * cdb + aa[ed];
    }
  }
}

// log sum_j exp(v_j), and the exp(v_j)-weighted mean of y_j, over the
// finite v_j (-inf and 0 when there are none); the largest term is taken
// as 1 without an exponential
__device__ __forceinline__ void lse4(const double (&v)[K], const double (&y)[K], double& lse, double& mean) {
  const double m = fmax(fmax(v[0], v[1]), fmax(v[2], v[3]));
  if (!(m > -INFINITY)) {
    lse = -INFINITY;
    mean = 0.0;
    return;
  }
  double s = 0.0, sy = 0.0;
#pragma unroll
  for (int j = 0; j < K; ++j) {
    if (v[j] == m) {
      s += 1.0;
      sy += y[j];
    } else if (v[j] > -INFINITY) {
      const double r = exp(v[j] - m);
      s += r;
      sy += r * y[j];
    }
  }
  lse = m + (s == 1.0 ? 0.0 : log(s));
  mean = sy / s;
}
}  // namespace pr

// U: kept states per lane and pass.  U = 2 issues two states' loads before
// either's stores (the neighbouring step's entries never overlap this
// step's), which pays where a step keeps hundreds of states; U = 1 keeps the
// registers for fetching the next step's words one step ahead, which pays
// where a step keeps a few.
template <int U>
__global__ void __launch_bounds__(pr::SP_WAVES * 64, 2) pruned_sp_kernel(PrArgs a) {
  using namespace pr;
  static_assert(U == 1 || U == 2, "states per lane and pass");
  constexpr bool kAhead = U == 1;
  extern __shared__ uint64_t lds_sp[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint64_t* nbm = lds_sp + (size_t)wave * (kSpLdsPerWave / sizeof(uint64_t));  // [WORDS] neighbour words
  uint32_t* npre = reinterpret_cast<uint32_t*>(nbm + WORDS);                    // [WORDS] neighbour ranks
  uint32_t* list = npre + WORDS;                                                // [LIST]
  const int64_t L = a.L;
  const double T = a.T, i2T = 0.5 / a.T, iT = 1.0 / a.T;
  for (int64_t sl = (int64_t)blockIdx.x * SP_WAVES + wave; sl < a.nblk; sl += (int64_t)gridDim.x * SP_WAVES) {
    const int64_t bb = a.b0 + sl;
    const float* wb = a.w + bb * L;
    const float* gb = a.g + bb * L;
    const uint64_t* bm = a.bm + sl * L * (int64_t)WORDS;
    // an entry holds log alpha and A until the backward sweep reaches it,
    // then log beta and B (its own forward values are read first)
    double* la = a.ent + sl * 2 * a.ecap;
    double* aa = la + a.ecap;
    bool bad = false;
    // ------------------------------------------------------------ forward
    int64_t base = 0, base_prev = 0;
    double zm = -INFINITY, zs = 0.0, zy = 0.0;  // logZ and E[F] at the last step
    uint64_t wd[WPL], nx[kAhead ? WPL : 1];
    if constexpr (kAhead) fetch_step(bm, lane, nx);
    for (int64_t t = 0; t < L; ++t) {
      if constexpr (kAhead) {
#pragma unroll
        for (int r = 0; r < WPL; ++r) wd[r] = nx[r];
        if (t + 1 < L) fetch_step(bm + (t + 1) * WORDS, lane, nx);
      } else {
        fetch_step(bm + t * WORDS, lane, wd);
      }
      int run;
      const int m = step_ranks(wd, lane, run);
      if (base + m > a.ecap || m == 0) {
        bad = true;
        break;
      }
      const double wt = (double)ld_uniform(wb, t), gt = (double)ld_uniform(gb, t);
      for (int r0 = 0; r0 < m; r0 += LIST) {
        list_round(wd, lane, run, r0, list);
        const int mr = m - r0 < LIST ? m - r0 : LIST;
        if constexpr (U == 1) {
          for (int k = lane; k < mr; k += 64) {
            const int s = (int)list[k];
            const int64_t e = base + r0 + k;
            const double cs = (double)a.c[s];
            const double h = -(wt - cs) * (wt - cs) * i2T;
            double lv, av;
            if (t == 0) {
              lv = h;
              av = gt * cs;
            } else {
              // predecessors (s >> 2) + j 2^14: one word, bits ip * 16 + j * 4 + up
              int qp, b0;
              pos_of(s >> 2, qp, b0);  // (j = 0)
              const uint64_t word = nbm[qp];
              const uint32_t pr0 = npre[qp];
              double pm = -INFINITY, ps = 0.0, py = 0.0;
#pragma unroll
              for (int j = 0; j < K; ++j) {
                const int pb = b0 + j * 4;
                if ((word >> pb) & 1ull) {
                  const int64_t ep = base_prev + pr0 + __popcll(word & ((1ull << pb) - 1ull));
                  lse_add(pm, ps, py, la[ep], aa[ep]);
                }
              }
              lv = (pm > -INFINITY) ? h + pm + (ps == 1.0 ? 0.0 : log(ps)) : -INFINITY;
              av = gt * cs + ((pm > -INFINITY) ? py / ps : 0.0);
            }
            la[e] = lv;
            aa[e] = av;
            if (t == L - 1) lse_add(zm, zs, zy, lv, av);
          }
        } else {
          // (this step's entries lie above the previous step's)
          for (int k = lane; k < mr; k += 64 * U) {
            const bool two = U == 2 && k + 64 < mr;
            int st[U];
            st[0] = (int)list[k];
            if constexpr (U == 2) st[1] = two ? (int)list[k + 64] : st[0];
            double cs[U], v[U][K], y[U][K];
#pragma unroll
            for (int x = 0; x < U; ++x) {
              cs[x] = (double)a.c[st[x]];
              if (t > 0) pred_vals(st[x], nbm, npre, base_prev, la, aa, v[x], y[x]);
            }
#pragma unroll
            for (int x = 0; x < U; ++x) {
              if (x == 1 && !two) break;
              const double h = -(wt - cs[x]) * (wt - cs[x]) * i2T;
              double lv = h, av = gt * cs[x];
              if (t > 0) {
                double lp, mp;
                lse4(v[x], y[x], lp, mp);
                lv = h + lp;
                av += mp;
              }
              const int64_t e = base + r0 + k + 64 * x;
              la[e] = lv;
              aa[e] = av;
              if (t == L - 1) lse_add(zm, zs, zy, lv, av);
            }
          }
        }
      }
      keep_tables(wd, lane, run, nbm, npre);
      wave_fence();
      base_prev = base;
      base += m;
    }
    if (bad) {
      if (lane == 0) a.flags[bb] = 1;
      continue;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1)
      lse_merge(zm, zs, zy, __shfl_xor(zm, o), __shfl_xor(zs, o), __shfl_xor(zy, o));
    zm = __shfl(zm, 0); zs = __shfl(zs, 0); zy = __shfl(zy, 0);
    const double logZ = zm + log(zs);
    const double EF = zy / zs;
    // Z holds the best path, whose weight is exp(-best / 2T): a smaller Z
    // means the kept states missed it
    const double zbest = -(double)ld_uniform(a.best, sl) * i2T;
    if (!(logZ > -INFINITY && logZ < INFINITY) || logZ < zbest - 1e-5 * fabs(zbest) - 1e-3) {
      if (lane == 0) a.flags[bb] = 1;
      continue;
    }
    // ----------------------------------------------------------- backward
    int64_t base_next = base;  // base of step t + 1
    if constexpr (kAhead) fetch_step(bm + (L - 1) * WORDS, lane, nx);
    for (int64_t t = L - 1; t >= 0; --t) {
      if constexpr (kAhead) {
#pragma unroll
        for (int r = 0; r < WPL; ++r) wd[r] = nx[r];
        if (t > 0) fetch_step(bm + (t - 1) * WORDS, lane, nx);
      } else {
        fetch_step(bm + t * WORDS, lane, wd);
      }
      int run;
      const int m = step_ranks(wd, lane, run);
      const int64_t bt = base_next - m;
      const double wt = (double)ld_uniform(wb, t), gt = (double)ld_uniform(gb, t);
      const double wn = t + 1 < L ? (double)ld_uniform(wb, t + 1) : 0.0;
      const double gn = t + 1 < L ? (double)ld_uniform(gb, t + 1) : 0.0;
      double sPc = 0.0, sPX = 0.0, sPcX = 0.0;
      for (int r0 = 0; r0 < m; r0 += LIST) {
        list_round(wd, lane, run, r0, list);
        const int mr = m - r0 < LIST ? m - r0 : LIST;
        if constexpr (U == 1) {
          for (int k = lane; k < mr; k += 64) {
            const int s = (int)list[k];
            const int64_t e = bt + r0 + k;
            const double cs = (double)a.c[s];
            const double lae = la[e], aae = aa[e];
            double lbv = 0.0, bvv = 0.0;
            if (t + 1 < L) {
              // successors (s mod 2^14) * 4 + b: one word, bits id * 16 + jd * 4 + b
              const int s14 = s & (GS - 1);
              int qd, b0;
              pos_of(s14 << 2, qd, b0);  // (b = 0)
              const uint64_t word = nbm[qd];
              const uint32_t pr0 = npre[qd];
              double nm = -INFINITY, ns = 0.0, ny = 0.0;
#pragma unroll
              for (int b = 0; b < K; ++b) {
                const int nb = b0 + b;
                if ((word >> nb) & 1ull) {
                  const int64_t ed = base_next + pr0 + __popcll(word & ((1ull << nb) - 1ull));
                  const double cd = (double)a.c[(s14 << 2) | b];
                  const double hd = -(wn - cd) * (wn - cd) * i2T;
                  lse_add(nm, ns, ny, hd + la[ed], gn * cd + aa[ed]);  // (step t + 1: beta, B)
                }
              }
              lbv = (nm > -INFINITY) ? nm + (ns == 1.0 ? 0.0 : log(ns)) : -INFINITY;
              bvv = (nm > -INFINITY) ? ny / ns : 0.0;
            }
            la[e] = lbv;
            aa[e] = bvv;
            const double P = exp(lae + lbv - logZ);
            const double X = aae + bvv - EF;
            sPc += P * cs;
            sPX += P * X;
            sPcX += P * cs * X;
            if (a.dc && P > 0.0) atomicAdd(a.dc + s, P * (gt + (wt - cs) * X * iT));
          }
        } else {
          // (the successors' entries lie above this step's)
          for (int k = lane; k < mr; k += 64 * U) {
            const bool two = U == 2 && k + 64 < mr;
            int st[U];
            st[0] = (int)list[k];
            if constexpr (U == 2) st[1] = two ? (int)list[k + 64] : st[0];
            double cs[U], lae[U], aae[U], v[U][K], y[U][K];
#pragma unroll
            for (int x = 0; x < U; ++x) {
              const int64_t e = bt + r0 + (two ? k + 64 * x : k);
              cs[x] = (double)a.c[st[x]];
              lae[x] = la[e];
              aae[x] = aa[e];
              if (t + 1 < L) succ_vals(st[x], nbm, npre, base_next, la, aa, a.c, wn, gn, i2T, v[x], y[x]);
            }
#pragma unroll
            for (int x = 0; x < U; ++x) {
              if (x == 1 && !two) break;
              double lbv = 0.0, bvv = 0.0;
              if (t + 1 < L) lse4(v[x], y[x], lbv, bvv);
              const int64_t e = bt + r0 + k + 64 * x;
              la[e] = lbv;
              aa[e] = bvv;
              const double P = exp(lae[x] + lbv - logZ);
              const double X = aae[x] + bvv - EF;
              sPc += P * cs[x];
              sPX += P * X;
              sPcX += P * cs[x] * X;
              if (a.dc && P > 0.0) atomicAdd(a.dc + st[x], P * (gt + (wt - cs[x]) * X * iT));
            }
          }
        }
      }
      keep_tables(wd, lane, run, nbm, npre);
      wave_fence();
      sPc = wave_sum_d(sPc);
      sPX = wave_sum_d(sPX);
      sPcX = wave_sum_d(sPcX);
      if (lane == 0) {
        if (a.w_soft) a.w_soft[bb * L + t] = (float)sPc;
        if (a.dW) a.dW[bb * L + t] = (float)((sPcX - sPc * sPX) / T);
      }
      base_next = bt;
    }
    if (lane == 0 && a.logZ) a.logZ[bb] = (float)logZ;
  }
}

// dCodebook: the fp64 accumulator as the fp32 output
__global__ void dc_store_kernel(const double* acc, int64_t S, float* out) {
  const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (s < S) out[s] = (float)acc[s];
}

// the slots' fp64 partial sums added into the accumulator (fixed slot order)
__global__ void dc_reduce_add_kernel(const double* part, int64_t nslots, int64_t S, double* acc) {
  const int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  double v = acc[s];
  for (int64_t q = 0; q < nslots; ++q) v += part[q * S + s];
  acc[s] = v;
}

__global__ void fill_d_kernel(double* out, int64_t count) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) out[i] = 0.0;
}

}  // namespace bcjr
