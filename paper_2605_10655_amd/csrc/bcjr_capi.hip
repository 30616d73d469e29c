// bcjr_capi.hip -- C ABI entry points (declared in include/bcjr.h): argument
// validation, kernel-family choice, workspace carving and launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstddef>
#include <cstdint>
#include <mutex>

#include "bcjr.h"
#include "bcjr_internal.h"
#include "bcjr_generic_kernels.h"
#include "bcjr_kernels.h"
#include "bcjr_ldlq_kernels.h"
#include "bcjr_pruned_kernels.h"
#include "bcjr_vec_kernels.h"
#include "bcjr_qat.h"

// Scratch memory of bcjr_soft_codeword_fwd_vjp_noalloc: one copy per GPU,
// allocated with the code object and held until the process ends.  In host
// code this name is only a stand-in for the symbol; the device address of a
// GPU's copy comes from hipGetSymbolAddress with that GPU current.
constexpr size_t kScratchBytes = BCJR_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace bcjr {

// The rotating-exchange kernel for S = 65536, k = 2 (bcjr_rot.hip, its own
// translation unit and instruction scheduler).
const void* fb_rot_kernel();
int fb_rot_launch(unsigned grid, size_t lds, hipStream_t stream, const FbArgs& a);
// its linear-domain form (blocks it marks are recomputed by the former)
const void* fb_lin_kernel(bool vjp);
int fb_lin_threads();
int fb_lin_launch(bool vjp, unsigned grid, size_t lds, hipStream_t stream, const FbArgs& a);

namespace {

constexpr int kDeviceCUs = 256;     // MI355X; used only to size the workspace query
constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Kernel family for a given (n, k): threads per workgroup, the super-group
// slots per thread compiled in, the runtime super-groups per thread.
struct Family {
  int nt = 0;       // threads per workgroup
  int sgmax = 0;    // compiled super-groups per thread
  int sgt = 0;      // super-groups per thread at run time
  int bpw = 0;      // blocks per workgroup
  int occ_est = 0;  // workgroups per CU assumed by the workspace query
};

// Shapes of the super-group families (fp32 / double-float, LDS-resident
// group vectors); every other 1 <= k <= n <= 16 runs the fp64 generic
// family of bcjr_generic_kernels.h.
bool supported(int n, int k) {
  if (k < 1 || k > 3 || n < 2 * k || n > 16) return false;
  const int nsg_bits = n - 2 * k;
  if (nsg_bits > 12) return false;           // at most 4096 super-groups
  if (k == 3 && nsg_bits > 8) return false;  // 64-state super-groups: one per thread
  return true;
}

Family family(int n, int k, bool dc) {
  Family f;
  const int nsg = 1 << (n - 2 * k);
  if (nsg <= 256) {
    f.nt = 256; f.sgmax = 1; f.sgt = 1; f.occ_est = 8;
  } else if (nsg <= 2048) {
    f.nt = 256; f.sgt = nsg / 256; f.sgmax = f.sgt; f.occ_est = 4;
  } else {
    f.nt = 1024; f.sgt = nsg / 1024; f.sgmax = f.sgt; f.occ_est = 1;
  }
  (void)dc;  // dCodebook runs as a separate sweep: same family
  const int tpb = nsg / f.sgt;
  f.bpw = f.nt / tpb;
  return f;
}

// The forward-backward kernels at 4096 super-groups run 512 threads of 8
// super-groups each (two waves per SIMD: room for the fp32 kernel's
// register-resident codebook and the low-temperature kernel's prefetched
// rows); the block count per workgroup and the slots are unchanged.
Family fb_family(int n, int k, bool dc) {
  Family f = family(n, k, dc);
  if (f.nt == 1024) {
    f.nt = 512;
    f.sgt = f.sgmax = 8;
  }
  return f;
}

// The VJP switches to fp64 log vectors when the field scale log2(e)/(2T)
// exceeds this value (T < 0.040 for unit-variance data).  The log values of
// the states that carry the posterior sit ~(field scale) x O(1) below the
// per-step maximum, and fp32 storage of them costs VJP accuracy roughly in
// proportion to 1/T (dCodebook error 2e-5 at T = 0.05, 5e-5 at 0.0245,
// 1.3e-4 at 0.014 for S = 65536); the switch keeps the fp32 path at >= 3x
// margin below the 1e-4 tolerance.
constexpr double kHighPrecisionK2 = 18.0;

bool use_high_precision(float T) { return 1.4426950408889634074 / (2.0 * (double)T) > kHighPrecisionK2; }

// The linear-domain kernel (S = 65536, k = 2, fwd + dW) serves the call up
// to this field scale (T >= 0.0206).  Its error grows steeply at lower T on
// blocks whose posterior is crisp everywhere (their dW is small, so the
// tolerance is tight): emulated on such a block of the q/o-projection
// matrix, dW is within 2.7e-6 of the oracle at T = 0.04, 2.9e-5 at 0.02,
// 7.7e-5 at 0.015 and 2.7e-4 at 0.0125.
constexpr double kLinearK2 = 35.0;

bool linear_ok(int n, int k, float T) {
  return n == 16 && k == 2 && 1.4426950408889634074 / (2.0 * (double)T) <= kLinearK2;
}

// The histories of one workgroup's blocks are addressed with 32-bit byte
// offsets: blocks per workgroup x L x (S/K x 8 bytes; for the VJP 12, or
// the low-temperature variant's hp_step_bytes where that is larger, at
// S/K = 2) below 2^31.
bool length_ok(int64_t L, int n, int k, bool vjp) {
  if (!supported(n, k)) return L <= ((int64_t)1 << 30);  // generic family: 64-bit offsets
  const Family f = family(n, k, false);
  const int64_t gs = (int64_t)1 << (n - k);
  const int64_t step = vjp ? std::max<int64_t>(12 * gs, hp_step_bytes(n, k)) : 8 * gs;
  return L <= 0x7FFFFFFF / ((int64_t)f.bpw * step);
}

// The fp32 forward-backward path keeps the scaled codebook at the front of
// its workspace.
size_t cs_bytes(int n) { return align_up(((size_t)4) << n); }

// Per-block flags of the linear-domain kernel (after the scaled codebook).
size_t flag_bytes(int64_t B) { return align_up((size_t)B * sizeof(int32_t)); }

struct FbLayout {
  size_t hist, histGA, small, dc, slot;
};

struct HpLayout {
  size_t hist, histGA, small, dc, slot;
};

HpLayout hp_layout(int64_t L, int n, int k, bool dc) {
  const size_t step = hp_step_bytes(n, k);
  HpLayout l;
  l.hist = align_up((size_t)L * step);
  l.histGA = dc ? align_up((size_t)L * step) : 0;
  l.small = align_up((size_t)4 * L * sizeof(float));
  l.dc = dc ? align_up(((size_t)1 << n) * sizeof(double)) : 0;
  l.slot = l.hist + l.histGA + l.small + l.dc;
  return l;
}

// per block [hi, tangent] floats and [lo] bytes of S/K each, then the
// cross-wave reduction area
size_t hp_lds_bytes(const Family& f, int n, int k) {
  const size_t gs = (size_t)1 << (n - k);
  return (size_t)f.bpw * 2 * gs * sizeof(float) + (((size_t)f.bpw * gs + 15) & ~(size_t)15) +
         (size_t)(f.nt / 64) * (2 * kRed * sizeof(float) + sizeof(double));
}

// The low-temperature VJP first decodes the minimum-distortion path (its
// codewords centre the backward tangent): [w_hard B*L f32][states B*L i32]
// [slots: Viterbi digits, then reused by the VJP kernel].
size_t hp_prefix_bytes(int64_t B, int64_t L) { return 2 * align_up((size_t)B * L * 4); }

FbLayout fb_layout(int64_t L, int n, int k, bool vjp, bool dc) {
  const size_t gs = (size_t)1 << (n - k);
  FbLayout l;
  l.hist = align_up((size_t)L * (vjp ? 2 : 1) * gs * sizeof(float));
  l.histGA = dc ? align_up((size_t)L * 2 * gs * sizeof(float)) : 0;
  l.small = align_up((size_t)3 * L * sizeof(float));
  l.dc = dc ? align_up(((size_t)1 << n) * sizeof(double)) : 0;
  l.slot = l.hist + l.histGA + l.small + l.dc;
  return l;
}

// The linear-domain kernel's slot: the same history and per-step vectors
// as the fp32 kernels (its repair pass reuses them).
FbLayout lin_layout(int64_t L, int n, int k, bool vjp) { return fb_layout(L, n, k, vjp, false); }

size_t vit_slot_bytes(int64_t L, int n, int k) {
  return align_up((size_t)L * ((size_t)1 << (n - k)));
}

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

size_t fb_lds_bytes(const Family& f, int n, int k) {
  const size_t gs = (size_t)1 << (n - k);
  return (size_t)f.bpw * 2 * gs * sizeof(float) + (size_t)(f.nt / 64) * 2 * kRed * sizeof(float);
}

size_t vit_lds_bytes(const Family& f, int n, int k) {
  const size_t gs = (size_t)1 << (n - k);
  return (size_t)f.bpw * gs * sizeof(double) + (size_t)(f.nt / 64) * (sizeof(double) + sizeof(int));
}

// ----------------------------------------------------------------- dispatch
using FbFn = void (*)(FbArgs);
using VitFn = void (*)(VitArgs);

// Families with one super-group per thread take the state bits at run time;
// the others are compiled per state-bit count so that every LDS and codebook
// offset folds into an immediate.
template <int KB, int NB, int SGM, int NT>
FbFn fb_variant(bool vjp, bool dc) {
  if (!vjp) return fb_kernel<KB, NB, SGM, NT, false, false>;
  if (!dc) return fb_kernel<KB, NB, SGM, NT, true, false>;
  return fb_kernel<KB, NB, SGM, NT, true, true>;
}

template <int KB>
FbFn fb_pick_kb(int n, const Family& f, bool vjp, bool dc) {
  if (f.sgmax == 1) return fb_variant<KB, 0, 1, 256>(vjp, dc);
  if constexpr (KB < 3) {
    // nsg = 2^(n - 2KB): 512, 1024, 2048 -> 256 threads; 4096 -> 512 (fb_family)
    constexpr int n512 = 2 * KB + 9;
    if (f.nt == 256) {
      if (n == n512) return fb_variant<KB, n512, 2, 256>(vjp, dc);
      if (n == n512 + 1) return fb_variant<KB, n512 + 1, 4, 256>(vjp, dc);
      if (n == n512 + 2) return fb_variant<KB, n512 + 2, 8, 256>(vjp, dc);
    }
    if (n == n512 + 3 && f.nt == 512) return fb_variant<KB, n512 + 3, 8, 512>(vjp, dc);
  }
  return nullptr;
}

template <int KB>
FbFn hp_pick_kb(int n, const Family& f, bool dc) {
  if (f.sgmax == 1) return dc ? fb_kernel_hp<KB, 0, 1, 256, true> : fb_kernel_hp<KB, 0, 1, 256, false>;
  if constexpr (KB < 3) {
    constexpr int n512 = 2 * KB + 9;
    if (n == n512) return dc ? fb_kernel_hp<KB, n512, 2, 256, true> : fb_kernel_hp<KB, n512, 2, 256, false>;
    if (n == n512 + 1)
      return dc ? fb_kernel_hp<KB, n512 + 1, 4, 256, true> : fb_kernel_hp<KB, n512 + 1, 4, 256, false>;
    if (n == n512 + 2)
      return dc ? fb_kernel_hp<KB, n512 + 2, 8, 256, true> : fb_kernel_hp<KB, n512 + 2, 8, 256, false>;
    if (n == n512 + 3 && f.nt == 512)
      return dc ? fb_kernel_hp<KB, n512 + 3, 8, 512, true> : fb_kernel_hp<KB, n512 + 3, 8, 512, false>;
  }
  return nullptr;
}

FbFn hp_pick(int n, int k, const Family& f, bool dc) {
  switch (k) {
    case 1: return hp_pick_kb<1>(n, f, dc);
    case 2: return hp_pick_kb<2>(n, f, dc);
    case 3: return hp_pick_kb<3>(n, f, dc);
    default: return nullptr;
  }
}

FbFn fb_pick(int n, int k, const Family& f, bool vjp, bool dc) {
  switch (k) {
    case 1: return fb_pick_kb<1>(n, f, vjp, dc);
    case 2: return fb_pick_kb<2>(n, f, vjp, dc);
    case 3: return fb_pick_kb<3>(n, f, vjp, dc);
    default: return nullptr;
  }
}

template <int KB>
VitFn vit_pick_kb(int n, const Family& f) {
  if (f.sgmax == 1) return viterbi_kernel<KB, 0, 1, 256>;
  if constexpr (KB < 3) {
    constexpr int n512 = 2 * KB + 9;
    if (n == n512) return viterbi_kernel<KB, n512, 2, 256>;
    if (n == n512 + 1) return viterbi_kernel<KB, n512 + 1, 4, 256>;
    if (n == n512 + 2) return viterbi_kernel<KB, n512 + 2, 8, 256>;
    if (n == n512 + 3) return viterbi_kernel<KB, n512 + 3, 4, 1024>;
  }
  return nullptr;
}

VitFn vit_pick(int n, int k, const Family& f) {
  switch (k) {
    case 1: return vit_pick_kb<1>(n, f);
    case 2: return vit_pick_kb<2>(n, f);
    case 3: return vit_pick_kb<3>(n, f);
    default: return nullptr;
  }
}

// the fp32 min-sum decode of the centring reference, same families
template <int KB>
VitFn vit_ref_pick_kb(int n, const Family& f) {
  if (f.sgmax == 1) return viterbi_ref_kernel<KB, 0, 1, 256>;
  if constexpr (KB < 3) {
    constexpr int n512 = 2 * KB + 9;
    if (n == n512) return viterbi_ref_kernel<KB, n512, 2, 256>;
    if (n == n512 + 1) return viterbi_ref_kernel<KB, n512 + 1, 4, 256>;
    if (n == n512 + 2) return viterbi_ref_kernel<KB, n512 + 2, 8, 256>;
    if (n == n512 + 3) return viterbi_ref_kernel<KB, n512 + 3, 4, 1024>;
  }
  return nullptr;
}

VitFn vit_ref_pick(int n, int k, const Family& f) {
  switch (k) {
    case 1: return vit_ref_pick_kb<1>(n, f);
    case 2: return vit_ref_pick_kb<2>(n, f);
    case 3: return vit_ref_pick_kb<3>(n, f);
    default: return nullptr;
  }
}

int common_checks(const float* w, int64_t B, int64_t L, const float* codebook, int n, int k,
                  bool vjp) {
  if (B < 0 || L < 1 || k < 1 || n < k || n > 16) return BCJR_ERR_INVALID_ARG;
  if (B > 0 && (!w || !codebook)) return BCJR_ERR_INVALID_ARG;
  if (codebook && ((uintptr_t)codebook & 15u)) return BCJR_ERR_INVALID_ARG;
  if (w && ((uintptr_t)w & 3u)) return BCJR_ERR_INVALID_ARG;
  if (!length_ok(L, n, k, vjp)) return BCJR_ERR_UNSUPPORTED;
  return BCJR_OK;
}

bool temperature_ok(float T) { return std::isfinite(T) && T > 0.f; }

// Number of workgroups to launch.  0 means the workspace holds less than one
// workgroup's slots.
int64_t grid_size(const void* kernel, const Family& f, size_t lds, int64_t B, size_t ws_bytes,
                  size_t slot_bytes, int* hip_err) {
  *hip_err = 0;
  int dev = 0, cus = kDeviceCUs, occ = 1;
  if (hipGetDevice(&dev) != hipSuccess) { *hip_err = 1; return 0; }
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
    *hip_err = 1;
    return 0;
  }
  if (hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
      hipSuccess) {
    *hip_err = 1;
    return 0;
  }
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, f.nt, lds) != hipSuccess ||
      occ < 1)
    occ = 1;
  const int64_t want = ceil_div(B, f.bpw);
  const int64_t fit = (int64_t)(ws_bytes / slot_bytes) / f.bpw;
  int64_t grid = want < (int64_t)cus * occ ? want : (int64_t)cus * occ;
  if (grid > fit) grid = fit;
  return grid;
}

int fill_zero(float* p, int64_t count, hipStream_t stream) {
  if (!p || count <= 0) return BCJR_OK;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)ceil_div(count, 256)), dim3(256), 0, stream, p,
                     count, 0.f);
  return hipGetLastError() == hipSuccess ? BCJR_OK : BCJR_ERR_HIP;
}

// ------------------------------------------------------------ generic family
constexpr int kGenOccEst = 4;  // workgroups per CU assumed by the workspace query

// doubles per slot: H and (VJP) B histories, four group vectors, and with
// the VJP the fp64 dCodebook partial (a VJP workspace always has room for it)
int64_t gen_slot_doubles(int64_t L, int n, int k, bool vjp) {
  const int64_t GS = (int64_t)1 << (n - k);
  return (vjp ? 2 : 1) * L * GS + 4 * GS + (vjp ? ((int64_t)1 << n) : 0);
}

// Viterbi: two metric vectors of doubles, then the digits of every slot
int64_t gen_vit_slot_bytes(int64_t L, int n, int k) {
  const int64_t GS = (int64_t)1 << (n - k);
  return 2 * GS * (int64_t)sizeof(double) + L * GS * (int64_t)sizeof(uint16_t);
}

int run_gen(const float* w, int64_t B, int64_t L, const float* codebook, int n, int k, float T,
            const float* g, float* w_soft, float* logZ, float* dW, float* dCodebook,
            void* workspace, size_t ws_bytes, hipStream_t stream, bool vjp) {
  const bool dc = vjp && dCodebook != nullptr;
  using Fn = void (*)(GenArgs);
  Fn fn = !vjp ? gen_fb_kernel<false, false> : (dc ? gen_fb_kernel<true, true> : gen_fb_kernel<true, false>);
  Family f;
  f.nt = kGenThreads;
  f.bpw = 1;
  const int64_t slot_d = gen_slot_doubles(L, n, k, vjp);
  int herr = 0;
  const int64_t grid = grid_size((const void*)fn, f, 0, B, ws_bytes, (size_t)slot_d * sizeof(double), &herr);
  if (herr) return BCJR_ERR_HIP;
  if (grid < 1) return BCJR_ERR_WORKSPACE;
  GenArgs a = {};
  a.w = w; a.g = g; a.c = codebook; a.B = B; a.L = L; a.n = n; a.k = k;
  a.inv2T = 1.0 / (2.0 * (double)T);
  a.invT = 1.0 / (double)T;
  a.w_soft = w_soft; a.logZ = logZ; a.dW = dW; a.dc = dCodebook;
  a.ws = static_cast<double*>(workspace);
  a.slot_doubles = slot_d;
  hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(kGenThreads), 0, stream, a);
  if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  if (dc) {
    const int64_t S = (int64_t)1 << n;
    hipLaunchKernelGGL(gen_dc_reduce_kernel, dim3((unsigned)ceil_div(S, 256)), dim3(256), 0, stream, a,
                       grid);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  }
  return BCJR_OK;
}

int run_gen_viterbi(const float* w, int64_t B, int64_t L, const float* codebook, int n, int k,
                    int32_t* states, float* w_hard, void* workspace, size_t ws_bytes,
                    hipStream_t stream) {
  Family f;
  f.nt = kGenThreads;
  f.bpw = 1;
  const int64_t slot = gen_vit_slot_bytes(L, n, k);
  int herr = 0;
  const int64_t grid = grid_size((const void*)gen_viterbi_kernel, f, 0, B, ws_bytes, (size_t)slot, &herr);
  if (herr) return BCJR_ERR_HIP;
  if (grid < 1) return BCJR_ERR_WORKSPACE;
  const int64_t GS = (int64_t)1 << (n - k);
  GenArgs a = {};
  a.w = w; a.c = codebook; a.B = B; a.L = L; a.n = n; a.k = k;
  a.states = states; a.w_hard = w_hard;
  a.ws = static_cast<double*>(workspace);
  a.slot_doubles = 2 * GS;
  a.bp = reinterpret_cast<uint16_t*>(static_cast<char*>(workspace) + grid * 2 * GS * (int64_t)sizeof(double));
  hipLaunchKernelGGL(gen_viterbi_kernel, dim3((unsigned)grid), dim3(kGenThreads), 0, stream, a);
  return hipGetLastError() == hipSuccess ? BCJR_OK : BCJR_ERR_HIP;
}

// approx: the fp32 decode of the centring reference (viterbi_ref_kernel)
// instead of the exact one; the generic family always decodes exactly
int run_viterbi(const float* w, int64_t B, int64_t L, const float* codebook, int n, int k,
                int32_t* states, float* w_hard, void* workspace, size_t ws_bytes,
                hipStream_t stream, bool approx = false, const int32_t* flags = nullptr) {
  if (!workspace || ((uintptr_t)workspace & 15u)) return BCJR_ERR_WORKSPACE;
  if (!supported(n, k))
    return run_gen_viterbi(w, B, L, codebook, n, k, states, w_hard, workspace, ws_bytes, stream);
  const Family f = family(n, k, false);
  VitFn fn = approx ? vit_ref_pick(n, k, f) : vit_pick(n, k, f);
  if (!fn) return BCJR_ERR_UNSUPPORTED;
  const size_t lds = vit_lds_bytes(f, n, k);
  const size_t slot = vit_slot_bytes(L, n, k);
  int herr = 0;
  const int64_t grid = grid_size((const void*)fn, f, lds, B, ws_bytes, slot, &herr);
  if (herr) return BCJR_ERR_HIP;
  if (grid < 1) return BCJR_ERR_WORKSPACE;
  VitArgs a = {};
  a.w = w; a.c = codebook; a.B = B; a.L = L; a.n = n; a.sgt = f.sgt;
  a.states = states; a.w_hard = w_hard;
  a.flags = approx ? flags : nullptr;
  a.bp = static_cast<uint8_t*>(workspace);
  hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(f.nt), lds, stream, a);
  return hipGetLastError() == hipSuccess ? BCJR_OK : BCJR_ERR_HIP;
}

// `ref` is the centring reference of the backward tangent ([B, L]); when it
// is null the minimum-distortion codewords are decoded into the front of the
// workspace first.
// With `repair_flags` only the blocks marked there are decoded and run:
// the repair pass of the linear-domain kernel below T = 0.04.
int run_fb_hp(const float* w, int64_t B, int64_t L, const float* codebook, int n, int k, float T,
              const float* g, const float* ref, float* w_soft, float* logZ, float* dW,
              float* dCodebook, void* workspace, size_t ws_bytes, hipStream_t stream,
              int32_t* repair_flags = nullptr, double* dc_add = nullptr) {
  const bool dc = dCodebook != nullptr || dc_add != nullptr;
  const Family f = fb_family(n, k, false);
  const HpLayout lay = hp_layout(L, n, k, dc);
  FbFn fn = hp_pick(n, k, f, dc);
  if (!fn) return BCJR_ERR_UNSUPPORTED;
  char* ws = static_cast<char*>(workspace);
  char* rest = ws;
  size_t rest_bytes = ws_bytes;
  if (!ref) {
    const size_t pre = hp_prefix_bytes(B, L);
    if (ws_bytes <= pre) return BCJR_ERR_WORKSPACE;
    float* w_hard = reinterpret_cast<float*>(ws);
    int32_t* states = reinterpret_cast<int32_t*>(ws + pre / 2);
    rest = ws + pre;
    rest_bytes = ws_bytes - pre;
    int st = run_viterbi(w, B, L, codebook, n, k, states, w_hard, rest, rest_bytes, stream, true,
                         repair_flags);
    if (st != BCJR_OK) return st;
    ref = w_hard;
  }
  const size_t lds = hp_lds_bytes(f, n, k);
  int herr = 0;
  const int64_t grid = grid_size((const void*)fn, f, lds, B, rest_bytes, lay.slot, &herr);
  if (herr) return BCJR_ERR_HIP;
  if (grid < 1) return BCJR_ERR_WORKSPACE;
  const int64_t slots = grid * f.bpw;
  char* p = rest;
  FbArgs a = {};
  a.w = w; a.g = g; a.c = codebook; a.B = B; a.L = L; a.n = n; a.sgt = f.sgt;
  const double Td = (double)T;
  a.k2 = (float)(1.4426950408889634074 / (2.0 * Td));
  a.k2d = 1.4426950408889634074 / (2.0 * Td);
  a.invT = (float)(1.0 / Td);
  a.w_soft = w_soft; a.logZ = logZ; a.dW = dW;
  a.bref = ref;
  a.flags = repair_flags;
  a.repair = repair_flags ? 1 : 0;
  a.histHB = reinterpret_cast<float*>(p);             p += slots * lay.hist;
  a.histGA = dc ? reinterpret_cast<float*>(p) : nullptr;  p += slots * lay.histGA;
  a.small = reinterpret_cast<float*>(p);              p += slots * lay.small;
  a.dc_part = dc ? reinterpret_cast<double*>(p) : nullptr;
  const int64_t S = (int64_t)1 << n;
  if (dc) {  // the (G, A, lo) entries of step 0 are zero for every block of a slot
    const int64_t hstep = hp_step_bytes(n, k) / 4;
    hipLaunchKernelGGL(fill_rows_kernel, dim3((unsigned)ceil_div(slots * hstep, 256)), dim3(256), 0,
                       stream, a.histGA, L * hstep, slots, hstep, 0.f);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  }
  if (dc_add) {  // a repair pass adds every slot's blocks into zeroed partials
    hipLaunchKernelGGL(fill_d_kernel, dim3((unsigned)ceil_div(slots * S, 256)), dim3(256), 0, stream,
                       a.dc_part, slots * S);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(f.nt), lds, stream, a);
  if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  if (dc) {
    const int64_t used = slots < B ? slots : B;
    if (dc_add)
      hipLaunchKernelGGL(dc_reduce_add_kernel, dim3((unsigned)ceil_div(S, 256)), dim3(256), 0, stream,
                         a.dc_part, used, S, dc_add);
    else
      hipLaunchKernelGGL(dc_reduce_kernel, dim3((unsigned)ceil_div(S, 256)), dim3(256), 0, stream,
                         a.dc_part, used, S, dCodebook);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  }
  return BCJR_OK;
}

// ------------------------------------------------------------ pruned VJP
// S = 65536, k = 2 at T <= 0.015: the sum-product and VJP over the states
// within kPrunedMargin nats of the block's best path (bcjr_pruned_kernels.h).
// Workspace: [block flags][fp64 dCodebook accumulator][slots: min-sum bytes,
// kept-state bits, step minima, best cost, kept-state entries].  Blocks are
// taken in chunks of one slot each; a block the pruned kernel cannot finish
// (more kept state-steps than its slot holds, or no finite logZ) is marked
// and recomputed afterwards by the double-float kernel in its repair mode,
// over the same slot memory, its dCodebook added into the accumulator.
constexpr double kPrunedMaxT = 0.015;
constexpr double kPrunedMargin = 30.0;   // nats below the best path
constexpr int64_t kPrunedMaxL = 2048;
constexpr int64_t kPrunedMaxSlots = 2048;
constexpr int64_t kPrunedEntriesPerStep = 1024;  // average kept states per step a slot holds
// from this temperature up the sum-product takes two kept states per lane and
// pass (a step keeps hundreds of states there; below, a few)
constexpr double kPrunedPairT = 0.01;

bool pruned_ok(int n, int k, float T, int64_t L) {
  return n == 16 && k == 2 && T <= (float)kPrunedMaxT && L <= kPrunedMaxL;  // (T as the caller rounded it)
}

struct PrLayout {
  size_t q, bm, hmin, best, ent, slot;
  int64_t ecap;
};

PrLayout pr_layout(int64_t L) {
  PrLayout l;
  l.ecap = kPrunedEntriesPerStep * L;
  l.q = align_up((size_t)L * pr::GS);
  l.bm = align_up((size_t)L * pr::WORDS * sizeof(uint64_t));
  l.hmin = align_up((size_t)L * sizeof(float));
  l.best = align_up(sizeof(float));
  l.ent = align_up((size_t)2 * l.ecap * sizeof(double));
  l.slot = l.q + l.bm + l.hmin + l.best + l.ent;
  return l;
}

int run_fb_pruned(const float* w, int64_t B, int64_t L, const float* codebook, int n, int k,
                  float T, const float* g, float* w_soft, float* logZ, float* dW, float* dCodebook,
                  void* workspace, size_t ws_bytes, hipStream_t stream) {
  const int64_t S = (int64_t)1 << n;
  const size_t fl = flag_bytes(B);
  const size_t dcb = dCodebook ? align_up((size_t)S * sizeof(double)) : 0;
  if (ws_bytes <= fl + dcb) return BCJR_ERR_WORKSPACE;
  const size_t region = ws_bytes - fl - dcb;
  const PrLayout lay = pr_layout(L);
  int64_t slots = std::min<int64_t>(std::min<int64_t>(B, kPrunedMaxSlots), (int64_t)(region / lay.slot));
  // the chunks must be large enough to fill the GPU, and the repair pass must fit
  if (slots < std::min<int64_t>(B, 64)) return BCJR_ERR_WORKSPACE;
  {  // a chunk of whole rounds of one min-sum workgroup per CU (a partial last
     // round costs as much as a full one)
    int dev = 0, cus = kDeviceCUs;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return BCJR_ERR_HIP;
    if (slots < B && slots > cus) slots -= slots % cus;
  }
  if (region < hp_prefix_bytes(B, L) + std::max(hp_layout(L, n, k, dCodebook != nullptr).slot,
                                                vit_slot_bytes(L, n, k)))
    return BCJR_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  int32_t* flags = reinterpret_cast<int32_t*>(ws);
  double* dcacc = dCodebook ? reinterpret_cast<double*>(ws + fl) : nullptr;
  char* base = ws + fl + dcb;
  static std::once_flag attr_once;
  static hipError_t attr_err = hipSuccess;
  std::call_once(attr_once, [] {
    if (hipFuncSetAttribute((const void*)mm_back_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)pr::kMinSumLds) != hipSuccess ||
        hipFuncSetAttribute((const void*)mm_fwd_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)pr::kMinSumLds) != hipSuccess ||
        hipFuncSetAttribute((const void*)pruned_sp_kernel<1>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)pr::kSpLds) != hipSuccess ||
        hipFuncSetAttribute((const void*)pruned_sp_kernel<2>, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)pr::kSpLds) != hipSuccess)
      attr_err = hipErrorInvalidValue;
  });
  if (attr_err != hipSuccess) return BCJR_ERR_HIP;
  hipLaunchKernelGGL(fill_kernel, dim3((unsigned)ceil_div(B, 256)), dim3(256), 0, stream,
                     reinterpret_cast<float*>(flags), B, 0.f);
  if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  if (dcacc) {
    hipLaunchKernelGGL(fill_d_kernel, dim3((unsigned)ceil_div(S, 256)), dim3(256), 0, stream, dcacc, S);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  }
  PrArgs a = {};
  a.w = w; a.g = g; a.c = codebook; a.B = B; a.L = L;
  a.T = (double)T;
  a.theta = (float)(2.0 * (double)T * kPrunedMargin);
  a.qscale = (float)(16.0 / (2.0 * (double)T * kPrunedMargin));
  char* p = base;
  a.q = reinterpret_cast<uint8_t*>(p);   p += (size_t)slots * lay.q;
  a.bm = reinterpret_cast<uint64_t*>(p); p += (size_t)slots * lay.bm;
  a.hmin = reinterpret_cast<float*>(p);  p += (size_t)slots * lay.hmin;
  a.best = reinterpret_cast<float*>(p);  p += (size_t)slots * lay.best;
  a.ent = reinterpret_cast<double*>(p);
  a.ecap = lay.ecap;
  a.dc = dcacc;
  a.w_soft = w_soft; a.logZ = logZ; a.dW = dW;
  a.flags = flags;
  // (the per-slot strides inside the kernels are L-based; hmin and best are
  // packed arrays of slots x L and slots floats)
  const bool pair = T >= (float)kPrunedPairT;
  for (int64_t b0 = 0; b0 < B; b0 += slots) {
    a.b0 = b0;
    a.nblk = std::min<int64_t>(slots, B - b0);
    hipLaunchKernelGGL(mm_back_kernel, dim3((unsigned)a.nblk), dim3(pr::NT), pr::kMinSumLds, stream, a);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
    hipLaunchKernelGGL(mm_fwd_kernel, dim3((unsigned)a.nblk), dim3(pr::NT), pr::kMinSumLds, stream, a);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
    hipLaunchKernelGGL(pair ? pruned_sp_kernel<2> : pruned_sp_kernel<1>,
                       dim3((unsigned)ceil_div(a.nblk, pr::SP_WAVES)), dim3(pr::SP_WAVES * 64), pr::kSpLds,
                       stream, a);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  }
  // marked blocks: the double-float kernel (it decodes their centring
  // reference first); every workgroup exits at once when none is marked
  int st = run_fb_hp(w, B, L, codebook, n, k, T, g, nullptr, w_soft, logZ, dW, nullptr, base, region,
                     stream, flags, dcacc);
  if (st != BCJR_OK) return st;
  if (dcacc) {
    hipLaunchKernelGGL(dc_store_kernel, dim3((unsigned)ceil_div(S, 256)), dim3(256), 0, stream, dcacc, S,
                       dCodebook);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  }
  return BCJR_OK;
}

// The linear-domain kernel (S = 65536, k = 2, T >= 0.0206; the soft
// codeword alone, or with dW): [scaled codebook][block flags][slots:
// lin_layout].  The blocks it marks are recomputed in a repair pass over the
// same slot memory once the first pass is complete: by the log-domain
// kernels (the soft codeword at any T, the VJP at T >= 0.04), or below
// T = 0.04 by the double-float VJP kernel centred on those blocks' decoded
// codewords.
int run_fb_lin(const float* w, int64_t B, int64_t L, const float* codebook, int n, int k, float T,
               const float* g, float* w_soft, float* logZ, float* dW, void* workspace,
               size_t ws_bytes, hipStream_t stream, bool vjp) {
  const Family f = fb_family(n, k, false);
  Family fl = f;
  fl.nt = fb_lin_threads();
  const FbLayout lay = lin_layout(L, n, k, vjp);
  const size_t lds = fb_lds_bytes(fl, n, k);
  const size_t front = cs_bytes(n) + flag_bytes(B);
  if (ws_bytes < front) return BCJR_ERR_WORKSPACE;
  const bool hp = vjp && use_high_precision(T);
  // the repair pass needs room for one slot of its own kernel (below T =
  // 0.04 after the decoded reference)
  if (hp && ws_bytes - front < hp_prefix_bytes(B, L) + std::max(hp_layout(L, n, k, false).slot,
                                                                 vit_slot_bytes(L, n, k)))
    return BCJR_ERR_WORKSPACE;
  int herr = 0;
  const int64_t grid = grid_size(fb_lin_kernel(vjp), fl, lds, B, ws_bytes - front, lay.slot, &herr);
  if (herr) return BCJR_ERR_HIP;
  if (grid < 1) return BCJR_ERR_WORKSPACE;
  const size_t lds_rep = fb_lds_bytes(f, n, k);
  FbFn soft_fn = vjp ? nullptr : fb_pick(n, k, f, false, false);
  if (!vjp && !soft_fn) return BCJR_ERR_UNSUPPORTED;
  const void* rep_kern = vjp ? fb_rot_kernel() : (const void*)soft_fn;
  if (!hp && hipFuncSetAttribute(rep_kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_rep) !=
                 hipSuccess)
    return BCJR_ERR_HIP;
  const int64_t slots = grid * f.bpw;
  const int64_t S = (int64_t)1 << n;
  float* cs = static_cast<float*>(workspace);
  int32_t* flags = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + cs_bytes(n));
  char* base = static_cast<char*>(workspace) + front;
  FbArgs a = {};
  a.w = w; a.g = g; a.c = codebook; a.cs = cs; a.B = B; a.L = L; a.n = n; a.sgt = f.sgt;
  const double Td = (double)T;
  a.k2 = (float)(1.4426950408889634074 / (2.0 * Td));
  a.invT = (float)(1.0 / Td);
  a.kap = (float)std::sqrt(1.4426950408889634074 / (2.0 * Td));
  a.inv_kap = (float)(1.0 / (double)a.kap);
  a.dws = (float)(1.0 / ((double)a.kap * (double)a.kap * Td));
  a.w_soft = w_soft; a.logZ = logZ; a.dW = dW;
  a.flags = flags;
  hipLaunchKernelGGL(scale_kernel, dim3((unsigned)ceil_div(S, 256)), dim3(256), 0, stream, codebook,
                     a.kap, cs, S);
  if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  a.histH = vjp ? nullptr : reinterpret_cast<float*>(base);
  a.histHB = vjp ? reinterpret_cast<float*>(base) : nullptr;
  a.small = reinterpret_cast<float*>(base + slots * lay.hist);
  if (fb_lin_launch(vjp, (unsigned)grid, lds, stream, a) != 0) return BCJR_ERR_HIP;
  // ---- repair pass over the marked blocks
  if (hp)
    return run_fb_hp(w, B, L, codebook, n, k, T, g, nullptr, w_soft, logZ, dW, nullptr, base,
                     ws_bytes - front, stream, flags);
  a.repair = 1;
  if (!vjp) {  // the log-domain soft-codeword kernel writes its own history
    hipLaunchKernelGGL(soft_fn, dim3((unsigned)grid), dim3(f.nt), lds_rep, stream, a);
    return hipGetLastError() == hipSuccess ? BCJR_OK : BCJR_ERR_HIP;
  }
  // log domain: its planar step L - 1 (H, B) entries are zero
  const int64_t hstep = 2 * ((int64_t)1 << (n - k));
  hipLaunchKernelGGL(fill_rows_kernel, dim3((unsigned)ceil_div(slots * hstep, 256)), dim3(256), 0,
                     stream, a.histHB + (L - 1) * hstep, L * hstep, slots, hstep, 0.f);
  if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  if (fb_rot_launch((unsigned)grid, lds_rep, stream, a) != 0) return BCJR_ERR_HIP;
  return BCJR_OK;
}

int run_fb(const float* w, int64_t B, int64_t L, const float* codebook, int n, int k, float T,
           const float* g, const float* ref, float* w_soft, float* logZ, float* dW,
           float* dCodebook, void* workspace, size_t ws_bytes, hipStream_t stream, bool vjp) {
  if (!workspace || ((uintptr_t)workspace & 15u)) return BCJR_ERR_WORKSPACE;
  if (!supported(n, k))
    return run_gen(w, B, L, codebook, n, k, T, g, w_soft, logZ, dW, dCodebook, workspace, ws_bytes,
                   stream, vjp);
  if (!dCodebook && linear_ok(n, k, T))
    return run_fb_lin(w, B, L, codebook, n, k, T, g, w_soft, logZ, dW, workspace, ws_bytes, stream,
                      vjp);
  if (vjp && pruned_ok(n, k, T, L)) {
    const int st = run_fb_pruned(w, B, L, codebook, n, k, T, g, w_soft, logZ, dW, dCodebook, workspace,
                                 ws_bytes, stream);
    if (st != BCJR_ERR_WORKSPACE) return st;  // (a workspace too small for it: the dense kernel)
  }
  if (vjp && use_high_precision(T))
    return run_fb_hp(w, B, L, codebook, n, k, T, g, ref, w_soft, logZ, dW, dCodebook, workspace,
                     ws_bytes, stream);
  const bool dc = vjp && dCodebook != nullptr;
  const Family f = fb_family(n, k, dc);
  const FbLayout lay = fb_layout(L, n, k, vjp, dc);
  FbFn fn = fb_pick(n, k, f, vjp, dc);
  if (!fn) return BCJR_ERR_UNSUPPORTED;
  const size_t lds = fb_lds_bytes(f, n, k);
  int herr = 0;
  if (ws_bytes < cs_bytes(n)) return BCJR_ERR_WORKSPACE;
  const int64_t grid = grid_size((const void*)fn, f, lds, B, ws_bytes - cs_bytes(n), lay.slot, &herr);
  if (herr) return BCJR_ERR_HIP;
  if (grid < 1) return BCJR_ERR_WORKSPACE;
  const int64_t slots = grid * f.bpw;
  const int64_t S = (int64_t)1 << n;
  // [scaled codebook][slots: histories][slots: shifts][slots: dCodebook partials]
  float* cs = static_cast<float*>(workspace);
  char* base = static_cast<char*>(workspace) + cs_bytes(n);
  FbArgs a = {};
  a.w = w; a.g = g; a.c = codebook; a.cs = cs; a.B = B; a.L = L; a.n = n; a.sgt = f.sgt;
  const double Td = (double)T;
  a.k2 = (float)(1.4426950408889634074 / (2.0 * Td));
  a.invT = (float)(1.0 / Td);
  a.kap = (float)std::sqrt(1.4426950408889634074 / (2.0 * Td));
  a.inv_kap = (float)(1.0 / (double)a.kap);
  a.dws = (float)(1.0 / ((double)a.kap * (double)a.kap * Td));
  a.w_soft = w_soft; a.logZ = logZ; a.dW = dW;
  hipLaunchKernelGGL(scale_kernel, dim3((unsigned)ceil_div(S, 256)), dim3(256), 0, stream, codebook,
                     a.kap, cs, S);
  if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  a.histH = vjp ? nullptr : reinterpret_cast<float*>(base);
  a.histHB = vjp ? reinterpret_cast<float*>(base) : nullptr;
  a.histGA = dc ? reinterpret_cast<float*>(base + slots * lay.hist) : nullptr;
  a.small = reinterpret_cast<float*>(base + slots * (lay.hist + lay.histGA));
  a.dc_part = dc ? reinterpret_cast<double*>(base + slots * (lay.hist + lay.histGA + lay.small))
                 : nullptr;
  if (vjp) {  // the (H, B) rows of step L - 1 are zero for every block of a slot
    const int64_t hstep = 2 * ((int64_t)1 << (n - k));
    hipLaunchKernelGGL(fill_rows_kernel, dim3((unsigned)ceil_div(slots * hstep, 256)), dim3(256), 0,
                       stream, a.histHB + (L - 1) * hstep, L * hstep, slots, hstep, 0.f);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
    if (dc) {  // and the (G, A) entries of step 0
      hipLaunchKernelGGL(fill_rows_kernel, dim3((unsigned)ceil_div(slots * hstep, 256)), dim3(256), 0,
                         stream, a.histGA, L * hstep, slots, hstep, 0.f);
      if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
    }
  }
  hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(f.nt), lds, stream, a);
  if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  if (dc) {
    const int64_t used = slots < B ? slots : B;
    hipLaunchKernelGGL(dc_reduce_kernel, dim3((unsigned)ceil_div(S, 256)), dim3(256), 0, stream,
                       a.dc_part, used, S, dCodebook);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  }
  return BCJR_OK;
}

int fwd_vjp(const float* w, int64_t B, int64_t L, const float* codebook, int state_bits, int k,
            float T, const float* grad_w_soft, const float* ref, float* w_soft, float* logZ,
            float* dW, float* dCodebook, void* workspace, size_t ws_bytes, hipStream_t stream) {
  int st = common_checks(w, B, L, codebook, state_bits, k, true);
  if (st != BCJR_OK) return st;
  if (!temperature_ok(T)) return BCJR_ERR_INVALID_ARG;
  if (B > 0 && !grad_w_soft) return BCJR_ERR_INVALID_ARG;
  if (grad_w_soft && ((uintptr_t)grad_w_soft & 3u)) return BCJR_ERR_INVALID_ARG;
  if (ref && ((uintptr_t)ref & 3u)) return BCJR_ERR_INVALID_ARG;
  if (B == 0) return fill_zero(dCodebook, (int64_t)1 << state_bits, stream);
  if (!w_soft && !logZ && !dW && !dCodebook) return BCJR_OK;
  return run_fb(w, B, L, codebook, state_bits, k, T, grad_w_soft, ref, w_soft, logZ, dW,
                dCodebook, workspace, ws_bytes, stream, true);
}

// ------------------------------------------------------------ vector emission
// k = 4 bits and V = 2 weights per step (16 predecessors per state).  One
// tile of 16 x 16 states per 16 lanes; 512 threads per workgroup, so that
// at S = 65536 two blocks (two workgroups, 66 KiB of LDS each) share a CU
// and one's barriers overlap the other's arithmetic.
bool vec_supported(int n, int k, int V) { return V == 2 && k == 4 && n >= 8 && n <= 16; }

struct VecFamily {
  int nt = 512, tpb = 0, sgt = 0, bpw = 0, occ_est = 2;
};

VecFamily vec_family(int n) {
  VecFamily f;
  const int lanes = 16 << (n - 8);
  f.tpb = std::min(lanes, f.nt);
  f.sgt = lanes / f.tpb;
  f.bpw = f.nt / f.tpb;
  return f;
}

size_t vec_vsz(int n) { return ((size_t)1 << (n - 4)) + ((n - 8) >= 4 ? 64 : 0); }

size_t fbv_lds_bytes(const VecFamily& f, int n) {
  return (size_t)f.bpw * 4 * vec_vsz(n) * sizeof(float) + (size_t)(f.nt / 64) * 2 * kRed * sizeof(float);
}

size_t vitv_lds_bytes(const VecFamily& f, int n) {
  return (size_t)f.bpw * 2 * vec_vsz(n) * sizeof(double) +
         (size_t)(f.nt / 64) * (sizeof(double) + sizeof(int));
}

// One workgroup's histories are addressed with 32-bit byte offsets: blocks
// per workgroup x N steps x S/16 groups x 16 bytes (4 for the soft codeword
// alone) below 2^31.
bool vec_length_ok(int64_t N, int n, bool vjp) {
  const VecFamily f = vec_family(n);
  // 16 bytes per group for the VJP (the low-temperature variant's entries)
  const int64_t per_step = (int64_t)f.bpw * (vjp ? 16 : 4) * ((int64_t)1 << (n - 4));
  return N >= 1 && N <= 0x7FFFFFFF / per_step;
}

// the scaled codebook and its transposed copy
size_t vec_cs_bytes(int n) { return 2 * align_up(((size_t)8) << n); }

FbLayout fbv_layout(int64_t N, int n, bool vjp, bool dc) {
  const size_t gs = (size_t)1 << (n - 4);
  FbLayout l;
  l.hist = align_up((size_t)N * (vjp ? 2 : 1) * gs * sizeof(float));
  l.histGA = dc ? align_up((size_t)N * 2 * gs * sizeof(float)) : 0;
  l.small = align_up((size_t)4 * N * sizeof(float));
  l.dc = dc ? align_up(((size_t)2 << n) * sizeof(double)) : 0;
  l.slot = l.hist + l.histGA + l.small + l.dc;
  return l;
}

size_t vitv_slot_bytes(int64_t N, int n) { return align_up((size_t)N * ((size_t)1 << (n - 4))); }

// Low-temperature V = 2 VJP: histories of (hi, lo, tangent, 0) entries, the
// lo-word exchange buffer, the per-step scalars (with lambda_t in fp64).
struct HpvLayout {
  size_t hist, histGA, xlo, small, dc, slot;
};

HpvLayout fbv_hp_layout(int64_t N, int n, bool dc) {
  const size_t gs = (size_t)1 << (n - 4);
  HpvLayout l;
  l.hist = align_up((size_t)N * gs * 16);
  l.histGA = dc ? align_up((size_t)N * gs * 16) : 0;
  l.xlo = align_up(2 * gs * sizeof(float));
  l.small = align_up((size_t)6 * N * sizeof(float));
  l.dc = dc ? align_up(((size_t)2 << n) * sizeof(double)) : 0;
  l.slot = l.hist + l.histGA + l.xlo + l.small + l.dc;
  return l;
}

// [w_hard B*L f32][states B*(L/2) i32]: the reference decode of the
// low-temperature VJP
size_t fbv_hp_prefix_bytes(int64_t B, int64_t L) {
  return align_up((size_t)B * L * 4) + align_up((size_t)B * (L / 2) * 4);
}

size_t fbv_hp_lds_bytes(const VecFamily& f, int n) {
  return fbv_lds_bytes(f, n) + (size_t)(f.nt / 64) * sizeof(double);
}

using FbvFn = void (*)(FbvArgs);
using VitvFn = void (*)(VitvArgs);

template <int NB, int SGM>
FbvFn fbv_variant(bool vjp, bool dc) {
  if (!vjp) return fbv_kernel<NB, SGM, 512, false, false>;
  if (!dc) return fbv_kernel<NB, SGM, 512, true, false>;
  return fbv_kernel<NB, SGM, 512, true, true>;
}

FbvFn fbv_pick(int n, bool vjp, bool dc) {
  if (n == 16) return fbv_variant<16, 8>(vjp, dc);
  return fbv_variant<0, 8>(vjp, dc);
}

FbvFn fbv_hp_pick(int n, bool dc) {
  if (n == 16) return dc ? fbv_kernel_hp<16, 8, 512, true> : fbv_kernel_hp<16, 8, 512, false>;
  return dc ? fbv_kernel_hp<0, 8, 512, true> : fbv_kernel_hp<0, 8, 512, false>;
}

VitvFn vitv_pick(int n) {
  if (n == 16) return vitv_kernel<16, 8, 512>;
  return vitv_kernel<0, 8, 512>;
}

int vec_checks(const float* w, int64_t B, int64_t L, const float* codebook, int n, int k, int V,
               bool vjp) {
  if (B < 0 || L < 1 || k < 1 || n < k || n > 16 || V < 1) return BCJR_ERR_INVALID_ARG;
  if (L % V) return BCJR_ERR_INVALID_ARG;
  if (B > 0 && (!w || !codebook)) return BCJR_ERR_INVALID_ARG;
  if (codebook && ((uintptr_t)codebook & 15u)) return BCJR_ERR_INVALID_ARG;
  if (w && ((uintptr_t)w & 3u)) return BCJR_ERR_INVALID_ARG;
  if (!vec_supported(n, k, V) || !vec_length_ok(L / V, n, vjp)) return BCJR_ERR_UNSUPPORTED;
  return BCJR_OK;
}

int run_vitv(const float* w, int64_t B, int64_t L, const float* codebook, int n, int32_t* states,
             float* w_hard, void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (!workspace || ((uintptr_t)workspace & 15u)) return BCJR_ERR_WORKSPACE;
  const VecFamily f = vec_family(n);
  const int64_t N = L / 2;
  VitvFn fn = vitv_pick(n);
  const size_t lds = vitv_lds_bytes(f, n);
  Family ff;
  ff.nt = f.nt; ff.bpw = f.bpw;
  int herr = 0;
  const int64_t grid = grid_size((const void*)fn, ff, lds, B, ws_bytes, vitv_slot_bytes(N, n), &herr);
  if (herr) return BCJR_ERR_HIP;
  if (grid < 1) return BCJR_ERR_WORKSPACE;
  VitvArgs a;
  a.w = w; a.c = codebook; a.B = B; a.N = N; a.n = n; a.sgt = f.sgt;
  a.states = states; a.w_hard = w_hard;
  a.bp = static_cast<uint8_t*>(workspace);
  hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(f.nt), lds, stream, a);
  return hipGetLastError() == hipSuccess ? BCJR_OK : BCJR_ERR_HIP;
}

// `ref` is the centring reference of the backward tangent ([B, L]); when it
// is null the minimum-distortion codewords are decoded into the workspace
// first.
int run_fbv_hp(const float* w, int64_t B, int64_t L, const float* codebook, int n, float T,
               const float* g, const float* ref, float* w_soft, float* logZ, float* dW,
               float* dCodebook, void* workspace, size_t ws_bytes, hipStream_t stream) {
  const bool dc = dCodebook != nullptr;
  const VecFamily f = vec_family(n);
  const int64_t N = L / 2;
  const HpvLayout lay = fbv_hp_layout(N, n, dc);
  FbvFn fn = fbv_hp_pick(n, dc);
  const size_t cb = vec_cs_bytes(n);
  if (ws_bytes <= cb) return BCJR_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  float* cs = reinterpret_cast<float*>(ws);
  const int64_t S2 = (int64_t)2 << n;
  char* rest = ws + cb;
  size_t rest_bytes = ws_bytes - cb;
  if (!ref) {
    const size_t pre = fbv_hp_prefix_bytes(B, L);
    if (rest_bytes <= pre) return BCJR_ERR_WORKSPACE;
    float* w_hard = reinterpret_cast<float*>(rest);
    int32_t* states = reinterpret_cast<int32_t*>(rest + align_up((size_t)B * L * 4));
    rest += pre;
    rest_bytes -= pre;
    int st = run_vitv(w, B, L, codebook, n, states, w_hard, rest, rest_bytes, stream);
    if (st != BCJR_OK) return st;
    ref = w_hard;
  }
  const size_t lds = fbv_hp_lds_bytes(f, n);
  Family ff;
  ff.nt = f.nt; ff.bpw = f.bpw;
  int herr = 0;
  const int64_t grid = grid_size((const void*)fn, ff, lds, B, rest_bytes, lay.slot, &herr);
  if (herr) return BCJR_ERR_HIP;
  if (grid < 1) return BCJR_ERR_WORKSPACE;
  const int64_t slots = grid * f.bpw;
  FbvArgs a = {};
  a.w = w; a.g = g; a.cs = cs; a.csT = cs + S2; a.B = B; a.N = N; a.n = n; a.sgt = f.sgt;
  const double Td = (double)T;
  a.k2d = 1.4426950408889634074 / (2.0 * Td);
  a.invT = (float)(1.0 / Td);
  a.w_soft = w_soft; a.logZ = logZ; a.dW = dW;
  a.bref = ref;
  // the unscaled codebook and its transposed copy
  hipLaunchKernelGGL(scale_vec_kernel, dim3((unsigned)ceil_div((int64_t)1 << n, 256)), dim3(256), 0,
                     stream, codebook, 1.0f, cs, const_cast<float*>(a.csT), n);
  if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  char* p = rest;
  a.hist = reinterpret_cast<float*>(p);                     p += slots * lay.hist;
  a.histGA = dc ? reinterpret_cast<float*>(p) : nullptr;    p += slots * lay.histGA;
  a.xlo = reinterpret_cast<float*>(p);                      p += slots * lay.xlo;
  a.small = reinterpret_cast<float*>(p);                    p += slots * lay.small;
  a.dc_part = dc ? reinterpret_cast<double*>(p) : nullptr;
  hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(f.nt), lds, stream, a);
  if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  if (dc) {
    const int64_t used = slots < B ? slots : B;
    hipLaunchKernelGGL(dc_reduce_kernel, dim3((unsigned)ceil_div(S2, 256)), dim3(256), 0, stream,
                       a.dc_part, used, S2, dCodebook);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  }
  return BCJR_OK;
}

int run_fbv(const float* w, int64_t B, int64_t L, const float* codebook, int n, float T,
            const float* g, float* w_soft, float* logZ, float* dW, float* dCodebook,
            void* workspace, size_t ws_bytes, hipStream_t stream, bool vjp) {
  if (!workspace || ((uintptr_t)workspace & 15u)) return BCJR_ERR_WORKSPACE;
  if (vjp && use_high_precision(T))
    return run_fbv_hp(w, B, L, codebook, n, T, g, nullptr, w_soft, logZ, dW, dCodebook, workspace,
                      ws_bytes, stream);
  const bool dc = vjp && dCodebook != nullptr;
  const VecFamily f = vec_family(n);
  const int64_t N = L / 2;
  const FbLayout lay = fbv_layout(N, n, vjp, dc);
  FbvFn fn = fbv_pick(n, vjp, dc);
  const size_t lds = fbv_lds_bytes(f, n);
  if (ws_bytes < vec_cs_bytes(n)) return BCJR_ERR_WORKSPACE;
  Family ff;
  ff.nt = f.nt; ff.bpw = f.bpw;
  int herr = 0;
  const int64_t grid = grid_size((const void*)fn, ff, lds, B, ws_bytes - vec_cs_bytes(n), lay.slot, &herr);
  if (herr) return BCJR_ERR_HIP;
  if (grid < 1) return BCJR_ERR_WORKSPACE;
  const int64_t slots = grid * f.bpw;
  const int64_t S2 = (int64_t)2 << n;  // codebook floats
  // [scaled codebook][slots: histories][slots: (G, A) histories][slots: scalars][slots: dCodebook]
  float* cs = static_cast<float*>(workspace);
  char* base = static_cast<char*>(workspace) + vec_cs_bytes(n);
  FbvArgs a = {};
  a.w = w; a.g = g; a.cs = cs; a.B = B; a.N = N; a.n = n; a.sgt = f.sgt;
  const double Td = (double)T;
  a.kap = (float)std::sqrt(1.4426950408889634074 / (2.0 * Td));
  a.inv_kap = (float)(1.0 / (double)a.kap);
  a.dws = (float)(1.0 / ((double)a.kap * (double)a.kap * Td));
  a.w_soft = w_soft; a.logZ = logZ; a.dW = dW;
  a.csT = cs + S2;
  hipLaunchKernelGGL(scale_vec_kernel, dim3((unsigned)ceil_div((int64_t)1 << n, 256)), dim3(256), 0,
                     stream, codebook, a.kap, cs, const_cast<float*>(a.csT), n);
  if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  a.hist = reinterpret_cast<float*>(base);
  a.histGA = dc ? reinterpret_cast<float*>(base + slots * lay.hist) : nullptr;
  a.small = reinterpret_cast<float*>(base + slots * (lay.hist + lay.histGA));
  a.dc_part = dc ? reinterpret_cast<double*>(base + slots * (lay.hist + lay.histGA + lay.small))
                 : nullptr;
  hipLaunchKernelGGL(fn, dim3((unsigned)grid), dim3(f.nt), lds, stream, a);
  if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  if (dc) {
    const int64_t used = slots < B ? slots : B;
    hipLaunchKernelGGL(dc_reduce_kernel, dim3((unsigned)ceil_div(S2, 256)), dim3(256), 0, stream,
                       a.dc_part, used, S2, dCodebook);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  }
  return BCJR_OK;
}

// ------------------------------------------------------------ BlockLDLQ
// [A: d x d fp64][Rinv: (d / b) blocks of b x b fp64][mean]
size_t ldl_ws_bytes(int64_t d, int64_t b) {
  return align_up((size_t)(d * d) * sizeof(double)) + align_up((size_t)(d * b) * sizeof(double)) + kAlign;
}

bool ldl_args_ok(int64_t d, int64_t b, double damp) {
  return d >= 1 && b >= 1 && d % b == 0 && d <= ((int64_t)1 << 20) && std::isfinite(damp) && damp >= 0.0;
}

unsigned blocks_for(int64_t count, int per) { return (unsigned)ceil_div(count, per); }

int run_block_ldl(const float* H, int64_t d, int64_t b, double damp, double* M, double* D, char* ws,
                  hipStream_t stream) {
  double* A = reinterpret_cast<double*>(ws);
  double* Rinv = reinterpret_cast<double*>(ws + align_up((size_t)(d * d) * sizeof(double)));
  double* mean = reinterpret_cast<double*>(ws + align_up((size_t)(d * d) * sizeof(double)) +
                                           align_up((size_t)(d * b) * sizeof(double)));
  hipLaunchKernelGGL(ldl::diag_mean_kernel, dim3(1), dim3(256), 0, stream, H, d, mean);
  hipLaunchKernelGGL(ldl::flip_damp_kernel, dim3(blocks_for(d * d, 256)), dim3(256), 0, stream, H, d,
                     damp, (const double*)mean, A);
  for (int64_t p = 0; p < d; p += ldl::kPanel) {
    const int w = (int)std::min<int64_t>(ldl::kPanel, d - p);
    hipLaunchKernelGGL(ldl::chol_diag_kernel, dim3(1), dim3(256), 0, stream, A, d, p, w);
    const int64_t rest = d - p - w;
    if (rest > 0) {
      hipLaunchKernelGGL(ldl::chol_trsm_kernel, dim3(blocks_for(rest, 256)), dim3(256), 0, stream, A, d,
                         p, w);
      const int64_t nt = ceil_div(rest, ldl::kPanel);
      hipLaunchKernelGGL(ldl::chol_update_kernel, dim3((unsigned)(nt * (nt + 1) / 2)), dim3(256), 0,
                         stream, A, d, p, w);
    }
  }
  hipLaunchKernelGGL(ldl::rinv_kernel, dim3((unsigned)(d / b)), dim3(256), 0, stream, (const double*)A, d,
                     b, Rinv);
  hipLaunchKernelGGL(ldl::m_kernel, dim3(blocks_for(d * d, 256)), dim3(256), 0, stream, (const double*)A, d,
                     b, (const double*)Rinv, M);
  if (D)
    hipLaunchKernelGGL(ldl::dblk_kernel, dim3(blocks_for(d * d, 256)), dim3(256), 0, stream,
                       (const double*)A, d, b, D);
  return hipGetLastError() == hipSuccess ? BCJR_OK : BCJR_ERR_HIP;
}

size_t ldlq_decode_ws(int64_t rows, int64_t b, int n, int k, int V) {
  return V == 1 ? bcjr_workspace_bytes(rows, b, n, k, BCJR_OP_VITERBI)
                : bcjr_vec_workspace_bytes(rows, b, n, k, V, BCJR_OP_VITERBI);
}

// [M: d x d fp64][block LDL workspace][target: rows x b f32][w_hat block: rows x b f32][decode]
size_t ldlq_ws_bytes(int64_t rows, int64_t cols, int64_t b, int n, int k, int V) {
  return align_up((size_t)(cols * cols) * sizeof(double)) + ldl_ws_bytes(cols, b) +
         2 * align_up((size_t)(rows * b) * sizeof(float)) + ldlq_decode_ws(rows, b, n, k, V);
}

// Device address of the current GPU's copy of `scratch`, looked up once per
// device (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

int scratch_address(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return BCJR_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return BCJR_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return BCJR_ERR_HIP;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return BCJR_OK;
}

}  // namespace
}  // namespace bcjr

using namespace bcjr;

extern "C" {

size_t bcjr_workspace_bytes(int64_t B, int64_t L, int state_bits, int k, int op) {
  if (B < 0 || L < 1 || k < 1 || state_bits < k || state_bits > 16) return 0;
  if (!length_ok(L, state_bits, k, op != BCJR_OP_FWD && op != BCJR_OP_VITERBI)) return 0;
  if (B == 0) return 0;
  if (op != BCJR_OP_FWD && op != BCJR_OP_VJP && op != BCJR_OP_FWD_VJP && op != BCJR_OP_VITERBI)
    return 0;
  if (!supported(state_bits, k)) {
    const int64_t grid = std::min<int64_t>(B, (int64_t)kDeviceCUs * kGenOccEst);
    if (op == BCJR_OP_VITERBI) return (size_t)(grid * gen_vit_slot_bytes(L, state_bits, k));
    return (size_t)(grid * gen_slot_doubles(L, state_bits, k, op != BCJR_OP_FWD)) * sizeof(double);
  }
  if (op == BCJR_OP_VITERBI) {
    const Family f = family(state_bits, k, false);
    const int64_t grid = std::min<int64_t>(ceil_div(B, f.bpw), (int64_t)kDeviceCUs * f.occ_est);
    return (size_t)(grid * f.bpw) * vit_slot_bytes(L, state_bits, k);
  }
  if (op != BCJR_OP_FWD && op != BCJR_OP_VJP && op != BCJR_OP_FWD_VJP) return 0;
  const bool vjp = op != BCJR_OP_FWD;
  // a VJP workspace is sized for the dCodebook family (never smaller)
  const Family f = family(state_bits, k, vjp);
  const Family f2 = family(state_bits, k, false);
  const int64_t g1 = std::min<int64_t>(ceil_div(B, f.bpw), (int64_t)kDeviceCUs * f.occ_est);
  const int64_t g2 = std::min<int64_t>(ceil_div(B, f2.bpw), (int64_t)kDeviceCUs * f2.occ_est);
  const int64_t slots = std::max<int64_t>(g1 * f.bpw, g2 * f2.bpw);
  size_t bytes = cs_bytes(state_bits) + flag_bytes(B) +
                 (size_t)slots * fb_layout(L, state_bits, k, vjp, vjp).slot;
  if (vjp) {  // the temperature decides the variant at call time: cover both
    const size_t vit = (size_t)(g2 * f2.bpw) * vit_slot_bytes(L, state_bits, k);
    const size_t hp = (size_t)(g2 * f2.bpw) * hp_layout(L, state_bits, k, true).slot;
    bytes = std::max(bytes, hp_prefix_bytes(B, L) + std::max(vit, hp));
    // the linear-domain path's repair pass: after its codebook and flags the
    // decoded reference and one double-float slot
    bytes = std::max(bytes, cs_bytes(state_bits) + flag_bytes(B) + hp_prefix_bytes(B, L) +
                                std::max(hp_layout(L, state_bits, k, false).slot,
                                         vit_slot_bytes(L, state_bits, k)));
    // the pruned path: flags, the fp64 dCodebook accumulator, then enough
    // slots for a chunk, or the repair pass's decoded reference and one slot
    if (state_bits == 16 && k == 2 && L <= kPrunedMaxL)
      bytes = std::max(bytes, flag_bytes(B) + align_up(((size_t)1 << state_bits) * sizeof(double)) +
                                  std::max((size_t)std::min<int64_t>(B, 64) * pr_layout(L).slot,
                                           hp_prefix_bytes(B, L) +
                                               std::max(hp_layout(L, state_bits, k, true).slot,
                                                        vit_slot_bytes(L, state_bits, k))));
  }
  return bytes;
}

int bcjr_soft_codeword(const float* w, int64_t B, int64_t L, const float* codebook, int state_bits,
                       int k, float T, float* w_soft, float* logZ, void* workspace,
                       size_t ws_bytes, hipStream_t stream) {
  int st = common_checks(w, B, L, codebook, state_bits, k, false);
  if (st != BCJR_OK) return st;
  if (!temperature_ok(T)) return BCJR_ERR_INVALID_ARG;
  if (B > 0 && !w_soft) return BCJR_ERR_INVALID_ARG;
  if (B == 0) return BCJR_OK;
  return run_fb(w, B, L, codebook, state_bits, k, T, nullptr, nullptr, w_soft, logZ, nullptr,
                nullptr, workspace, ws_bytes, stream, false);
}

int bcjr_soft_codeword_fwd_vjp(const float* w, int64_t B, int64_t L, const float* codebook,
                               int state_bits, int k, float T, const float* grad_w_soft,
                               float* w_soft, float* logZ, float* dW, float* dCodebook,
                               void* workspace, size_t ws_bytes, hipStream_t stream) {
  return fwd_vjp(w, B, L, codebook, state_bits, k, T, grad_w_soft, nullptr, w_soft, logZ, dW,
                 dCodebook, workspace, ws_bytes, stream);
}

int bcjr_soft_codeword_fwd_vjp_noalloc(const float* w, int64_t B, int64_t L, const float* codebook,
                                       int state_bits, int k, float T, const float* grad_w_soft,
                                       float* w_soft, float* logZ, float* dW, float* dCodebook,
                                       hipStream_t stream) {
  void* ws = nullptr;
  const int st = scratch_address(&ws);
  if (st != BCJR_OK) return st;
  return fwd_vjp(w, B, L, codebook, state_bits, k, T, grad_w_soft, nullptr, w_soft, logZ, dW,
                 dCodebook, ws, kScratchBytes, stream);
}

int bcjr_soft_codeword_vjp(const float* w, int64_t B, int64_t L, const float* codebook,
                           int state_bits, int k, float T, const float* grad_w_soft, float* dW,
                           float* dCodebook, void* workspace, size_t ws_bytes,
                           hipStream_t stream) {
  return bcjr_soft_codeword_fwd_vjp(w, B, L, codebook, state_bits, k, T, grad_w_soft, nullptr,
                                    nullptr, dW, dCodebook, workspace, ws_bytes, stream);
}

int bcjr_ste_vjp(const float* w, int64_t B, int64_t L, const float* codebook, int state_bits,
                 int k, float T, const float* w_hard, const float* grad_w_soft, float* dW,
                 float* dCodebook, void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (B > 0 && !w_hard) return BCJR_ERR_INVALID_ARG;
  return fwd_vjp(w, B, L, codebook, state_bits, k, T, grad_w_soft, w_hard, nullptr, nullptr, dW,
                 dCodebook, workspace, ws_bytes, stream);
}

int viterbi_decode(const float* w, int64_t B, int64_t L, const float* codebook, int state_bits,
                   int k, int32_t* states, float* w_hard, void* workspace, size_t ws_bytes,
                   hipStream_t stream) {
  int st = common_checks(w, B, L, codebook, state_bits, k, false);
  if (st != BCJR_OK) return st;
  if (B > 0 && !states) return BCJR_ERR_INVALID_ARG;
  if (B == 0) return BCJR_OK;
  return run_viterbi(w, B, L, codebook, state_bits, k, states, w_hard, workspace, ws_bytes, stream);
}

size_t bcjr_vec_workspace_bytes(int64_t B, int64_t L, int state_bits, int k, int V, int op) {
  if (V == 1) return bcjr_workspace_bytes(B, L, state_bits, k, op);
  const bool vjp = op == BCJR_OP_VJP || op == BCJR_OP_FWD_VJP;
  if (op != BCJR_OP_FWD && !vjp && op != BCJR_OP_VITERBI) return 0;
  if (B <= 0 || vec_checks(nullptr, 0, L, nullptr, state_bits, k, V, vjp) != BCJR_OK) return 0;
  const VecFamily f = vec_family(state_bits);
  const int64_t N = L / V;
  const int64_t slots = std::min<int64_t>(ceil_div(B, f.bpw), (int64_t)kDeviceCUs * f.occ_est) * f.bpw;
  if (op == BCJR_OP_VITERBI) return (size_t)slots * vitv_slot_bytes(N, state_bits);
  size_t bytes = vec_cs_bytes(state_bits) + (size_t)slots * fbv_layout(N, state_bits, vjp, vjp).slot;
  if (vjp) {  // the temperature decides the variant at call time: cover both
    const size_t vit = (size_t)slots * vitv_slot_bytes(N, state_bits);
    const size_t hp = (size_t)slots * fbv_hp_layout(N, state_bits, true).slot;
    bytes = std::max(bytes, vec_cs_bytes(state_bits) + fbv_hp_prefix_bytes(B, L) + std::max(vit, hp));
  }
  return bytes;
}

int bcjr_vec_soft_codeword(const float* w, int64_t B, int64_t L, const float* codebook,
                           int state_bits, int k, int V, float T, float* w_soft, float* logZ,
                           void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (V == 1)
    return bcjr_soft_codeword(w, B, L, codebook, state_bits, k, T, w_soft, logZ, workspace, ws_bytes,
                              stream);
  int st = vec_checks(w, B, L, codebook, state_bits, k, V, false);
  if (st != BCJR_OK) return st;
  if (!temperature_ok(T)) return BCJR_ERR_INVALID_ARG;
  if (B > 0 && !w_soft) return BCJR_ERR_INVALID_ARG;
  if (B == 0) return BCJR_OK;
  return run_fbv(w, B, L, codebook, state_bits, T, nullptr, w_soft, logZ, nullptr, nullptr, workspace,
                 ws_bytes, stream, false);
}

int bcjr_vec_soft_codeword_fwd_vjp(const float* w, int64_t B, int64_t L, const float* codebook,
                                   int state_bits, int k, int V, float T, const float* grad_w_soft,
                                   float* w_soft, float* logZ, float* dW, float* dCodebook,
                                   void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (V == 1)
    return bcjr_soft_codeword_fwd_vjp(w, B, L, codebook, state_bits, k, T, grad_w_soft, w_soft, logZ,
                                      dW, dCodebook, workspace, ws_bytes, stream);
  int st = vec_checks(w, B, L, codebook, state_bits, k, V, true);
  if (st != BCJR_OK) return st;
  if (!temperature_ok(T)) return BCJR_ERR_INVALID_ARG;
  if (B > 0 && !grad_w_soft) return BCJR_ERR_INVALID_ARG;
  if (grad_w_soft && ((uintptr_t)grad_w_soft & 3u)) return BCJR_ERR_INVALID_ARG;
  if (B == 0) return fill_zero(dCodebook, (int64_t)V << state_bits, stream);
  if (!w_soft && !logZ && !dW && !dCodebook) return BCJR_OK;
  return run_fbv(w, B, L, codebook, state_bits, T, grad_w_soft, w_soft, logZ, dW, dCodebook,
                 workspace, ws_bytes, stream, true);
}

int bcjr_vec_soft_codeword_vjp(const float* w, int64_t B, int64_t L, const float* codebook,
                               int state_bits, int k, int V, float T, const float* grad_w_soft,
                               float* dW, float* dCodebook, void* workspace, size_t ws_bytes,
                               hipStream_t stream) {
  return bcjr_vec_soft_codeword_fwd_vjp(w, B, L, codebook, state_bits, k, V, T, grad_w_soft, nullptr,
                                        nullptr, dW, dCodebook, workspace, ws_bytes, stream);
}

int bcjr_vec_viterbi_decode(const float* w, int64_t B, int64_t L, const float* codebook,
                            int state_bits, int k, int V, int32_t* states, float* w_hard,
                            void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (V == 1)
    return viterbi_decode(w, B, L, codebook, state_bits, k, states, w_hard, workspace, ws_bytes,
                          stream);
  int st = vec_checks(w, B, L, codebook, state_bits, k, V, false);
  if (st != BCJR_OK) return st;
  if (B > 0 && !states) return BCJR_ERR_INVALID_ARG;
  if (B == 0) return BCJR_OK;
  return run_vitv(w, B, L, codebook, state_bits, states, w_hard, workspace, ws_bytes, stream);
}

size_t bcjr_block_ldl_workspace_bytes(int64_t d, int64_t block) {
  if (!ldl_args_ok(d, block, 0.0)) return 0;
  return ldl_ws_bytes(d, block);
}

int bcjr_block_ldl(const float* H, int64_t d, int64_t block, double damp, double* M, double* D,
                   void* workspace, size_t ws_bytes, hipStream_t stream) {
  if (!ldl_args_ok(d, block, damp) || !H || !M) return BCJR_ERR_INVALID_ARG;
  if (((uintptr_t)H & 3u) || ((uintptr_t)M & 7u) || ((uintptr_t)D & 7u)) return BCJR_ERR_INVALID_ARG;
  if (!workspace || ((uintptr_t)workspace & 15u) || ws_bytes < ldl_ws_bytes(d, block))
    return BCJR_ERR_WORKSPACE;
  return run_block_ldl(H, d, block, damp, M, D, static_cast<char*>(workspace), stream);
}

size_t bcjr_ldlq_workspace_bytes(int64_t rows, int64_t cols, int64_t block, int state_bits, int k, int V) {
  if (rows < 1 || V < 1 || !ldl_args_ok(cols, block, 0.0) || block % V) return 0;
  if (ldlq_decode_ws(rows, block, state_bits, k, V) == 0) return 0;
  return ldlq_ws_bytes(rows, cols, block, state_bits, k, V);
}

int bcjr_ldlq_viterbi(const float* W, int64_t rows, int64_t cols, const float* codebook, int state_bits,
                      int k, int V, const float* H, int64_t block, double damp, float* W_hat,
                      int32_t* states, float* targets, void* workspace, size_t ws_bytes,
                      hipStream_t stream) {
  if (rows < 1 || V < 1 || !ldl_args_ok(cols, block, damp) || block % V) return BCJR_ERR_INVALID_ARG;
  if (!W || !codebook || !H || !W_hat || !states) return BCJR_ERR_INVALID_ARG;
  if (((uintptr_t)W & 3u) || ((uintptr_t)H & 3u) || ((uintptr_t)W_hat & 3u) || ((uintptr_t)states & 3u) ||
      ((uintptr_t)targets & 3u) || ((uintptr_t)codebook & 15u))
    return BCJR_ERR_INVALID_ARG;
  const int st0 = V == 1 ? common_checks(W, rows, block, codebook, state_bits, k, false)
                         : vec_checks(W, rows, block, codebook, state_bits, k, V, false);
  if (st0 != BCJR_OK) return st0;
  if (!workspace || ((uintptr_t)workspace & 15u) ||
      ws_bytes < ldlq_ws_bytes(rows, cols, block, state_bits, k, V))
    return BCJR_ERR_WORKSPACE;
  char* p = static_cast<char*>(workspace);
  double* M = reinterpret_cast<double*>(p);
  p += align_up((size_t)(cols * cols) * sizeof(double));
  char* lws = p;
  p += ldl_ws_bytes(cols, block);
  float* tgt = reinterpret_cast<float*>(p);
  p += align_up((size_t)(rows * block) * sizeof(float));
  float* wh = reinterpret_cast<float*>(p);
  p += align_up((size_t)(rows * block) * sizeof(float));
  const size_t dec_bytes = ws_bytes - (size_t)(p - static_cast<char*>(workspace));
  int st = run_block_ldl(H, cols, block, damp, M, nullptr, lws, stream);
  if (st != BCJR_OK) return st;
  const int64_t nb = cols / block;
  for (int64_t j = 0; j < nb; ++j) {
    float* t = targets ? targets + j * rows * block : tgt;
    hipLaunchKernelGGL(ldl::feedback_kernel, dim3(blocks_for(rows, ldl::kPanel), blocks_for(block, ldl::kPanel)),
                       dim3(256), 0, stream, W, (const float*)W_hat, (const double*)M, rows, cols, block,
                       j * block, t);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
    int32_t* sj = states + j * rows * (block / V);
    st = V == 1 ? run_viterbi(t, rows, block, codebook, state_bits, k, sj, wh, p, dec_bytes, stream)
                : run_vitv(t, rows, block, codebook, state_bits, sj, wh, p, dec_bytes, stream);
    if (st != BCJR_OK) return st;
    hipLaunchKernelGGL(ldl::scatter_kernel, dim3(blocks_for(rows * block, 256)), dim3(256), 0, stream,
                       (const float*)wh, rows, cols, block, j * block, W_hat);
    if (hipGetLastError() != hipSuccess) return BCJR_ERR_HIP;
  }
  return BCJR_OK;
}

int bcjr_gaussian_codebook(float* codebook, int state_bits, int V, uint64_t seed,
                           hipStream_t stream) {
  if (!codebook || state_bits < 1 || state_bits > 24 || V < 1 || V > kMaxV)
    return BCJR_ERR_INVALID_ARG;
  if ((uintptr_t)codebook & 3u) return BCJR_ERR_INVALID_ARG;
  const int64_t count = (int64_t)V << state_bits;
  hipLaunchKernelGGL(gauss_codebook_kernel, dim3((unsigned)ceil_div(count, 256)), dim3(256), 0, stream,
                     codebook, state_bits, V, perm_set(seed, V));
  return hipGetLastError() == hipSuccess ? BCJR_OK : BCJR_ERR_HIP;
}

int qat_adam_step(float* param, const float* grad, float* m, float* v, int64_t count, float lr,
                  float beta1, float beta2, float eps, int64_t step, float grad_clip,
                  hipStream_t stream) {
  if (count < 0 || step < 1 || !(lr >= 0.f) || !(beta1 >= 0.f && beta1 < 1.f) ||
      !(beta2 >= 0.f && beta2 < 1.f) || !(eps > 0.f) || !(grad_clip >= 0.f))
    return BCJR_ERR_INVALID_ARG;
  if (count == 0) return BCJR_OK;
  if (!param || !grad || !m || !v) return BCJR_ERR_INVALID_ARG;
  const float c1 = (float)(1.0 / (1.0 - std::pow((double)beta1, (double)step)));
  const float c2 = (float)(1.0 / (1.0 - std::pow((double)beta2, (double)step)));
  hipLaunchKernelGGL(adam_kernel, dim3((unsigned)ceil_div(count, 256)), dim3(256), 0, stream, param,
                     grad, m, v, count, lr, beta1, beta2, eps, c1, c2, grad_clip);
  return hipGetLastError() == hipSuccess ? BCJR_OK : BCJR_ERR_HIP;
}

int qat_sgd_step(float* param, const float* grad, int64_t count, float lr, float grad_clip,
                 hipStream_t stream) {
  if (count < 0 || !(lr >= 0.f) || !(grad_clip >= 0.f)) return BCJR_ERR_INVALID_ARG;
  if (count == 0) return BCJR_OK;
  if (!param || !grad) return BCJR_ERR_INVALID_ARG;
  hipLaunchKernelGGL(sgd_kernel, dim3((unsigned)ceil_div(count, 256)), dim3(256), 0, stream, param,
                     grad, count, lr, grad_clip);
  return hipGetLastError() == hipSuccess ? BCJR_OK : BCJR_ERR_HIP;
}

const char* bcjr_status_string(int status) {
  switch (status) {
    case BCJR_OK: return "ok";
    case BCJR_ERR_INVALID_ARG: return "invalid argument";
    case BCJR_ERR_UNSUPPORTED: return "unsupported (state_bits, k)";
    case BCJR_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case BCJR_ERR_HIP: return "HIP runtime or launch error";
    default: return "unknown status";
  }
}

}  // extern "C"
