// issue_rates.hip -- gfx950 VALU issue-rate probe (measurement only; not
// part of the BCJR library's ABI).
//
// Every lane runs NCH independent chains of one operation (or an interleave
// of two), so that no instruction waits on the result of the one before it
// and, at full occupancy, the issue rate of the SIMD is what limits the
// kernel.  A second kernel (chain_kernel) varies the number of chains at low
// occupancy: with few chains per lane a wave waits on VALU results, which
// exposes the result latency and the per-wave instruction interval a
// kernel with that much independent work can reach.  The host times
// one launch with HIP events; the kernel also reads the shader clock
// counter (s_memtime) and the constant 100 MHz counter (s_memrealtime) at
// the start and end of every wave, from which the shader clock during the
// run follows.  Rates are lane-operations per clock per CU.
//
//   op 0  v_fma_f32            x = fma(x, a, b)
//   op 1  v_exp_f32            x = exp2(-x)
//   op 2  v_log_f32            x = log2(|x|)
//   op 3  v_rcp_f32            x = 1 / x
//   op 4  v_fma_f64            x = fma(x, a, b)   (fp64)
//   op 5  fma + exp, 1 : 1     one chain of each per step
//   op 6  fma + exp, 4 : 1
//   op 7  fma + exp, 8 : 1
//   op 8  v_add_f32            x = x + b
//   op 9  v_max_f32            x = max(x, y), y the neighbouring chain (fmaxf also
//                              quiets its operand: two v_max_f32 per step)
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <algorithm>
#include <vector>

namespace {

constexpr int NCH = 8;  // independent chains per operation type and lane

__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float lg2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float rcp(float x) { return __builtin_amdgcn_rcpf(x); }

template <int OP>
__global__ void __launch_bounds__(256) probe_kernel(int iters, float seed, float* sink, int64_t* clocks) {
  const int tid = threadIdx.x;
  uint64_t c0 = 0, r0 = 0;
  if ((tid & 63) == 0) {
    c0 = clock64();
    r0 = wall_clock64();
  }
  float x[NCH], y[NCH];
  double xd[NCH];
#pragma unroll
  for (int i = 0; i < NCH; ++i) {
    x[i] = seed + 0.01f * (float)(i + 1) + 1e-6f * (float)tid;
    y[i] = 0.5f + 0.01f * (float)i;
    xd[i] = (double)x[i];
  }
  const float a = 0.999f, b = 1e-3f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      if constexpr (OP == 0) x[i] = fmaf(x[i], a, b);
      if constexpr (OP == 1) x[i] = ex2(-x[i]);
      if constexpr (OP == 2) x[i] = lg2(fabsf(x[i]));
      if constexpr (OP == 3) x[i] = rcp(x[i]);
      if constexpr (OP == 4) xd[i] = fma(xd[i], 0.999, 1e-3);
      if constexpr (OP >= 5 && OP <= 7) {
        constexpr int R = OP == 5 ? 1 : (OP == 6 ? 4 : 8);
#pragma unroll
        for (int q = 0; q < R; ++q) y[i] = fmaf(y[i], a, b);
        x[i] = ex2(-x[i]);
      }
      if constexpr (OP == 8) x[i] = x[i] + b;
      if constexpr (OP == 9) x[i] = fmaxf(x[i], x[(i + 1) % NCH]);
    }
  }
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < NCH; ++i) acc += x[i] + y[i] + (float)xd[i];
  // never true for the seeds the host passes: keeps the chains live
  if (acc == 1234.5f) sink[blockIdx.x * blockDim.x + tid] = acc;
  if ((tid & 63) == 0) {
    const uint64_t c1 = clock64(), r1 = wall_clock64();
    const int wave = blockIdx.x * (blockDim.x >> 6) + (tid >> 6);
    clocks[2 * wave + 0] = (int64_t)(c1 - c0);
    clocks[2 * wave + 1] = (int64_t)(r1 - r0);
  }
}

// Dependency-latency probe: NC independent chains per lane of one operation
// whose constants come from kernel arguments (no literal operands), 4 chain
// steps per loop iteration.  OP 0: v_fma_f32 (VOP3, 8-byte encoding),
// OP 1: v_add_f32 (VOP2, 4 bytes).  With few chains every instruction waits
// on the result of one NC instructions earlier, so the per-wave interval
// exposes the VALU result latency; with many it approaches the issue limit.
template <int NC, int OP>
__global__ void __launch_bounds__(256) chain_kernel(int iters, float seed, float a, float b, float* sink,
                                                     int64_t* clocks) {
  const int tid = threadIdx.x;
  uint64_t c0 = 0, r0 = 0;
  if ((tid & 63) == 0) {
    c0 = clock64();
    r0 = wall_clock64();
  }
  float x[NC];
#pragma unroll
  for (int i = 0; i < NC; ++i) x[i] = seed + 0.01f * (float)(i + 1) + 1e-6f * (float)tid;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        if constexpr (OP == 0) x[i] = fmaf(x[i], a, b);
        if constexpr (OP == 1) x[i] = x[i] + b;
      }
    }
  }
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < NC; ++i) acc += x[i];
  if (acc == 1234.5f) sink[blockIdx.x * blockDim.x + tid] = acc;
  if ((tid & 63) == 0) {
    const uint64_t c1 = clock64(), r1 = wall_clock64();
    const int wave = blockIdx.x * (blockDim.x >> 6) + (tid >> 6);
    clocks[2 * wave + 0] = (int64_t)(c1 - c0);
    clocks[2 * wave + 1] = (int64_t)(r1 - r0);
  }
}

using ChainFn = void (*)(int, float, float, float, float*, int64_t*);

ChainFn pick_chain(int op, int chains) {
  switch (op * 100 + chains) {
    case 2: return chain_kernel<2, 0>;
    case 4: return chain_kernel<4, 0>;
    case 8: return chain_kernel<8, 0>;
    case 16: return chain_kernel<16, 0>;
    case 32: return chain_kernel<32, 0>;
    case 102: return chain_kernel<2, 1>;
    case 104: return chain_kernel<4, 1>;
    case 108: return chain_kernel<8, 1>;
    case 116: return chain_kernel<16, 1>;
    case 132: return chain_kernel<32, 1>;
    default: return nullptr;
  }
}

using ProbeFn = void (*)(int, float, float*, int64_t*);

ProbeFn pick(int op) {
  switch (op) {
    case 0: return probe_kernel<0>;
    case 1: return probe_kernel<1>;
    case 2: return probe_kernel<2>;
    case 3: return probe_kernel<3>;
    case 4: return probe_kernel<4>;
    case 5: return probe_kernel<5>;
    case 6: return probe_kernel<6>;
    case 7: return probe_kernel<7>;
    case 8: return probe_kernel<8>;
    case 9: return probe_kernel<9>;
    default: return nullptr;
  }
}

// Launches `launch` once untimed and once timed (HIP events) on `grid`
// workgroups of 256 threads.  Outputs: ms, the median shader clock over
// waves (clock ticks / real time) and the mean shader cycles per wave.
template <class F>
int timed_launches(int grid, F launch, float* ms, double* clock_hz, double* cycles_per_wave) {
  const int waves = grid * 4;
  float* sink = nullptr;
  int64_t* clk = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  int rc = 0;
  if (hipMalloc(&sink, (size_t)grid * 256 * sizeof(float)) != hipSuccess ||
      hipMalloc(&clk, (size_t)waves * 2 * sizeof(int64_t)) != hipSuccess ||
      hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
    rc = -4;
  } else {
    launch(sink, clk);
    (void)hipEventRecord(e0, 0);
    launch(sink, clk);
    (void)hipEventRecord(e1, 0);
    if (hipEventSynchronize(e1) != hipSuccess || hipGetLastError() != hipSuccess) rc = -4;
  }
  if (rc == 0) {
    (void)hipEventElapsedTime(ms, e0, e1);
    int64_t* h = new int64_t[(size_t)waves * 2];
    if (hipMemcpy(h, clk, (size_t)waves * 2 * sizeof(int64_t), hipMemcpyDeviceToHost) != hipSuccess) {
      rc = -4;
    } else {
      int rate_khz = 100000;
      int dev = 0;
      if (hipGetDevice(&dev) != hipSuccess ||
          hipDeviceGetAttribute(&rate_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess)
        rate_khz = 100000;
      std::vector<double> f;
      double cyc = 0.0;
      for (int i = 0; i < waves; ++i) {
        cyc += (double)h[2 * i];
        if (h[2 * i + 1] > 0)
          f.push_back((double)h[2 * i] / ((double)h[2 * i + 1] / ((double)rate_khz * 1e3)));
      }
      std::sort(f.begin(), f.end());
      *clock_hz = f.empty() ? 0.0 : f[f.size() / 2];
      *cycles_per_wave = cyc / (double)waves;
    }
    delete[] h;
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (sink) (void)hipFree(sink);
  if (clk) (void)hipFree(clk);
  return rc;
}

}  // namespace

extern "C" {

// Lane-operations per chain step of `op`: (ordinary VALU, transcendental).
int issue_rate_ops_per_step(int op, double* valu, double* trans) {
  static const double v[10] = {1, 0, 0, 0, 1, 1, 4, 8, 1, 2};
  static const double t[10] = {0, 1, 1, 1, 0, 1, 1, 1, 0, 0};
  if (op < 0 || op > 9 || !valu || !trans) return -1;
  *valu = v[op];
  *trans = t[op];
  return 0;
}

// Runs probe `op` once untimed and once timed on `grid` workgroups of 256
// threads, `iters` chain steps per lane.  Outputs: ms (event time of the
// timed launch), lane_ops (VALU + transcendental lane-operations of that
// launch), clock_hz (median over waves of shader-clock ticks / real time).
// Allocates and frees its own small buffers.  0 on success, -1 on bad
// arguments, -4 on a HIP error.
int issue_rate_run(int op, int iters, int grid, float* ms, double* lane_ops, double* clock_hz) {
  ProbeFn fn = pick(op);
  if (!fn || iters < 1 || grid < 1 || !ms || !lane_ops || !clock_hz) return -1;
  double cyc = 0.0;
  const int rc = timed_launches(
      grid, [&](float* sink, int64_t* clk) {
        hipLaunchKernelGGL(fn, dim3(grid), dim3(256), 0, 0, iters, 0.25f, sink, clk);
      },
      ms, clock_hz, &cyc);
  if (rc == 0) {
    double v = 0, t = 0;
    issue_rate_ops_per_step(op, &v, &t);
    *lane_ops = (double)grid * 256.0 * (double)iters * NCH * (v + t);
  }
  return rc;
}

// Dependency-latency probe: `chains` (2, 4, 8, 16 or 32) independent chains
// per lane of v_fma_f32 (op 0) or v_add_f32 (op 1), `iters` x 4 steps each,
// on `grid` workgroups of 256 threads (grid / 256 waves per SIMD at 256
// CUs).  Output: ms, the shader clock, and the mean shader cycles per VALU
// instruction of one wave (cycles per wave / instructions per wave).
int issue_rate_chains(int op, int chains, int iters, int grid, float* ms, double* cycles_per_instr,
                      double* clock_hz) {
  ChainFn fn = pick_chain(op, chains);
  if (!fn || iters < 1 || grid < 1 || !ms || !cycles_per_instr || !clock_hz) return -1;
  double cyc = 0.0;
  const int rc = timed_launches(
      grid, [&](float* sink, int64_t* clk) {
        hipLaunchKernelGGL(fn, dim3(grid), dim3(256), 0, 0, iters, 0.25f, 0.999f, 1e-3f, sink, clk);
      },
      ms, clock_hz, &cyc);
  if (rc == 0) *cycles_per_instr = cyc / ((double)iters * 4.0 * (double)chains);
  return rc;
}

}  // extern "C"
