// bcjr_rot.hip -- the rotating-exchange forward-backward kernels
// (bcjr_rot_kernels.h: log domain and linear domain) in their own translation unit, built with the AMDGPU
// max-ilp instruction scheduler; the rest of the library keeps the default
// one, under which the V = 2 kernel runs 8 % faster.  The dispatcher in
// bcjr_capi.hip reaches the kernels through these functions.
#include <hip/hip_runtime.h>

#include "bcjr_rot_kernels.h"

namespace bcjr {

const void* fb_rot_kernel() { return reinterpret_cast<const void*>(&fb_kernel_rot); }

// 0 on success, -1 when the launch reports a HIP error
int fb_rot_launch(unsigned grid, size_t lds, hipStream_t stream, const FbArgs& a) {
  hipLaunchKernelGGL(fb_kernel_rot, dim3(grid), dim3(512), lds, stream, a);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

// 512 threads (two waves per SIMD, the codebook rows resident in registers);
// the 1024-thread form (four waves per SIMD, 128 VGPRs) measured 221.7
// against 218.1 ms on one box
constexpr int kLinThreads = 512;

int fb_lin_threads() { return kLinThreads; }

const void* fb_lin_kernel(bool vjp) {
  return vjp ? reinterpret_cast<const void*>(&fb_kernel_lin<kLinThreads, true>)
             : reinterpret_cast<const void*>(&fb_kernel_lin<kLinThreads, false>);
}

int fb_lin_launch(bool vjp, unsigned grid, size_t lds, hipStream_t stream, const FbArgs& a) {
  if (vjp)
    hipLaunchKernelGGL((fb_kernel_lin<kLinThreads, true>), dim3(grid), dim3(kLinThreads), lds, stream, a);
  else
    hipLaunchKernelGGL((fb_kernel_lin<kLinThreads, false>), dim3(grid), dim3(kLinThreads), lds, stream, a);
  return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace bcjr
