// bcjr_internal.h -- kernel argument blocks shared by the host dispatcher and
// the kernels.  Not part of the public ABI.
#pragma once
#include <stdint.h>

namespace bcjr {

struct FbArgs {
  const float* w;      // [B, L]
  const float* g;      // [B, L] upstream gradient (VJP only)
  const float* c;      // [S] codebook
  const float* cs;     // [S] codebook times kappa (fp32 forward-backward kernel)
  int64_t B, L;
  int n;               // state bits
  int sgt;             // super-groups per thread
  float k2;            // log2(e) / (2T): h_t(s) in log2 units = -(w_t - c(s))^2 * k2
  float invT;          // 1 / T
  float kap, inv_kap;  // kappa = sqrt(k2) and 1 / kappa
  float dws;           // 1 / (kappa^2 T)
  float* w_soft;       // [B, L] or null
  float* logZ;         // [B] or null
  float* dW;           // [B, L] or null
  double* dc_part;     // [slots][S] fp64 partial sums of dCodebook, or null
  float* histH;        // [slots][L][S/K]   H_t as read by each super-group (soft codeword)
  float* histHB;       // [slots][L][2 S/K] H_t, then the B tangent, as [S/K] vectors (VJP)
  float* histGA;       // [slots][L][2 S/K] G_t and the A tangent per super-group (dCodebook)
  // (per step an H (G) vector then a B (A) vector of S/K floats, indexed by
  // group, written from the sweeps' exchange-write phases: the backward
  // sweep one dword per lane (column form), the forward sweep one 16-byte
  // row per super-group; the entries of step L - 1 (H, B) and step 0 (G, A)
  // are zero and filled before the launch)
  float* small;        // [slots][3][L]     shifts of H, lambda_t, E_p[X_t]
  // low-temperature variant (log vectors as hi + 8-bit lo pairs): steps of
  // hp_step_bytes(); histHB holds, per step and super-group, three planes
  // (hi, tangent as [threads][K] floats, lo as [threads][K] bytes), so that
  // one store of a wave fills whole cache lines; histGA per step three [S/K]
  // vectors (G hi, A floats, G lo bytes), stored by the forward sweep's
  // write phase for the next step (step 0 filled with zeros before the
  // launch); small is [slots][4][L]
  double k2d;          // log2(e) / (2T) in fp64
  const float* bref;   // [B, L] centring reference of the backward tangent
  // linear-domain kernel: per block 1 when its group vectors left the fp32
  // range (the block is then recomputed by the log-domain kernel), else 0;
  // with `repair` set, the log-domain kernel runs only the blocks marked 1
  int32_t* flags;      // [B] or null
  int repair;
};

// Bytes of one history step of the low-temperature kernel: 9 per group
// (hi and tangent floats, one lo byte), rounded up to 16.
inline uint32_t hp_step_bytes(int n, int k) { return (9u * (1u << (n - k)) + 15u) & ~15u; }

// Vector-emission trellis: k = 4 bits per step (K = 16), V = 2 weights per
// step.  Blocks hold L = 2 N weights.
struct FbvArgs {
  const float* w;      // [B, 2N]
  const float* g;      // [B, 2N] upstream gradient (VJP only)
  const float* cs;     // [S][2] codebook times kappa
  const float* csT;    // the same, transposed: entry (s mod (S/16)) * 16 + s / (S/16)
  int64_t B, N;        // blocks, steps per block
  int n;               // state bits
  int sgt;             // tiles per thread
  float kap, inv_kap;  // kappa = sqrt(log2(e) / (2T)) and 1 / kappa
  float dws;           // 1 / (kappa^2 T)
  float* w_soft;       // [B, 2N] or null
  float* logZ;         // [B] or null
  float* dW;           // [B, 2N] or null
  double* dc_part;     // [slots][S][2] fp64 partial sums of dCodebook, or null
  float* hist;         // [slots][N][S/16] H_t, or [slots][N][S/16][2] (H_t, B_t) with the VJP
  float* histGA;       // [slots][N][S/16][2] (G_t, A_t) (dCodebook)
  float* small;        // [slots][4][N] shifts of H, lambda_t, E_p[X_t], A centring
  // low-temperature variant (double-float log vectors, unscaled codebook in
  // cs / csT): hist and histGA hold [slots][N][S/16][4] (hi, lo, tangent, 0),
  // small [slots][6][N] (shift, E_p[X_t], A centring, -, lambda_t as fp64)
  double k2d;          // log2(e) / (2T)
  float invT;          // 1 / T
  const float* bref;   // [B, 2N] centring reference of the backward tangent
  float* xlo;          // [slots][2][S/16] lo words of the group vector being exchanged
};

struct VitvArgs {
  const float* w;      // [B, 2N]
  const float* c;      // [S][2]
  int64_t B, N;
  int n;
  int sgt;
  int32_t* states;     // [B, N]
  float* w_hard;       // [B, 2N] or null
  uint8_t* bp;         // [slots][N][S/16] winning predecessor digit
};

struct VitArgs {
  const float* w;
  const float* c;
  int64_t B, L;
  int n;
  int sgt;
  int32_t* states;     // [B, L]
  float* w_hard;       // [B, L] or null
  uint8_t* bp;         // [slots][L][S/K] winning predecessor digit
  // fp32 decode (one block per workgroup): when set, only the blocks marked
  // 1 here are decoded (the centring reference of a repair pass)
  const int32_t* flags;
};

}  // namespace bcjr
