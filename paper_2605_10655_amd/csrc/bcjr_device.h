// bcjr_device.h -- device helpers shared by the forward-backward kernels:
// fast exp2 / log2 / reciprocal, register pinning and scheduling fences, LDS
// vector moves, buffer-descriptor loads and stores, lane and scalar reads,
// and the block reductions (DPP within a wave, LDS across waves).  All of it
// has internal linkage, so each translation unit that includes it holds its
// own copy.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "bcjr_internal.h"

namespace bcjr {

namespace {

__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float lg2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Materialises a value in a register at this point.  Results that are held
// across a barrier are pinned so the compiler cannot sink the arithmetic that
// produces them below the barrier (which would keep its inputs live instead).
__device__ __forceinline__ void pin(float& x) { asm volatile("" : "+v"(x)); }

template <int K, class T>
__device__ __forceinline__ T max_of(const T (&x)[K]) {
  T m = x[0];
#pragma unroll
  for (int b = 1; b < K; ++b) m = fmax(m, x[b]);
  return m;
}

// Keeps the scheduler from hoisting the next super-group's loads above the
// current one: that hoisting multiplies the live registers by SGMAX.
__device__ __forceinline__ void sg_fence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

template <int N>
__device__ __forceinline__ void ld_vec(const float* p, float (&v)[N]) {
  static_assert(N == 1 || N == 2 || N % 4 == 0, "vector width");
  if constexpr (N == 1) {
    v[0] = p[0];
  } else if constexpr (N == 2) {
    const float2 t = *reinterpret_cast<const float2*>(p);
    v[0] = t.x; v[1] = t.y;
  } else {
#pragma unroll
    for (int q = 0; q < N / 4; ++q) {
      const float4 t = reinterpret_cast<const float4*>(p)[q];
      v[4 * q + 0] = t.x; v[4 * q + 1] = t.y; v[4 * q + 2] = t.z; v[4 * q + 3] = t.w;
    }
  }
}

template <int N>
__device__ __forceinline__ void st_vec(float* p, const float (&v)[N]) {
  if constexpr (N == 1) {
    p[0] = v[0];
  } else if constexpr (N == 2) {
    *reinterpret_cast<float2*>(p) = make_float2(v[0], v[1]);
  } else {
#pragma unroll
    for (int q = 0; q < N / 4; ++q)
      reinterpret_cast<float4*>(p)[q] =
          make_float4(v[4 * q + 0], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  }
}

// ---------------------------------------------------------------------------
// Buffer-resource access.  A descriptor (4 SGPRs) holds the array's base and
// size; every access gives a per-thread byte offset (one VGPR, fixed for the
// whole call) and a block-uniform byte offset (an SGPR).  This keeps the
// per-super-group addresses out of vector registers.
// ---------------------------------------------------------------------------
using rsrc_t = __amdgpu_buffer_rsrc_t;
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kRsrcFlags = 0x00020000;  // raw (unswizzled) buffer, 32-bit elements

__device__ __forceinline__ rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, kRsrcFlags);
}

// Vector elements are moved through plain scalars: a bit cast applied to an
// element expression (x.y) reads element 0 with this compiler.
__device__ __forceinline__ float as_f(unsigned u) { return __uint_as_float(u); }
__device__ __forceinline__ unsigned as_u(float f) { return __float_as_uint(f); }

// Cache policy of a buffer access: 0 = default, kStream = non-temporal (the
// line is inserted in L2 as the first to evict).  Write-once/read-once
// history rows go through kStream so that they do not push out of L2 the
// small vectors a block rewrites every step.
constexpr int kStream = 2;

template <int N, int CP = 0>
__device__ __forceinline__ void buf_ld(rsrc_t r, uint32_t voff, uint32_t soff, float (&v)[N]) {
  static_assert(N == 1 || N == 2 || N % 4 == 0, "vector width");
  if constexpr (N == 1) {
    v[0] = as_f(__builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, CP));
  } else if constexpr (N == 2) {
    const u32x2 x = __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, (int)soff, CP);
    const unsigned x0 = x.x, x1 = x.y;
    v[0] = as_f(x0);
    v[1] = as_f(x1);
  } else {
#pragma unroll
    for (int q = 0; q < N / 4; ++q) {
      const u32x4 x = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)(soff + 16u * q), CP);
      const unsigned x0 = x.x, x1 = x.y, x2 = x.z, x3 = x.w;
      v[4 * q + 0] = as_f(x0);
      v[4 * q + 1] = as_f(x1);
      v[4 * q + 2] = as_f(x2);
      v[4 * q + 3] = as_f(x3);
    }
  }
}

// Stores take the whole offset in the VGPR and a zero scalar offset.  With a
// register scalar offset the compiler assumes no wait state is needed between
// a wider-than-8-byte store and a VALU write of its data registers; on this
// GPU such a write corrupted the stored data.
template <int N, int CP = 0>
__device__ __forceinline__ void buf_st(rsrc_t r, uint32_t voff0, uint32_t soff0, const float (&v)[N]) {
  static_assert(N == 1 || N == 2 || N % 4 == 0, "vector width");
  const uint32_t voff = voff0 + soff0, soff = 0;
  if constexpr (N == 1) {
    __builtin_amdgcn_raw_buffer_store_b32(as_u(v[0]), r, (int)voff, (int)soff, CP);
  } else if constexpr (N == 2) {
    const u32x2 x = {as_u(v[0]), as_u(v[1])};
    __builtin_amdgcn_raw_buffer_store_b64(x, r, (int)voff, (int)soff, CP);
  } else {
#pragma unroll
    for (int q = 0; q < N / 4; ++q) {
      const u32x4 x = {as_u(v[4 * q + 0]), as_u(v[4 * q + 1]), as_u(v[4 * q + 2]), as_u(v[4 * q + 3])};
      __builtin_amdgcn_raw_buffer_store_b128(x, r, (int)voff, (int)(soff + 16u * q), CP);
    }
  }
}

// History row of one super-group: its K entries of H and, with the VJP, of
// B `plane` bytes after them; streamed (read once).
template <int K, bool VJP>
__device__ __forceinline__ void hist_row(rsrc_t h, uint32_t voff, uint32_t step_off, uint32_t sg_off,
                                         uint32_t plane, float (&H)[K], float (&B)[K]) {
  buf_ld<K, kStream>(h, voff, step_off + sg_off, H);
  if constexpr (VJP) buf_ld<K, kStream>(h, voff, step_off + sg_off + plane, B);
}

__device__ __forceinline__ void pin_u(uint32_t& x) { asm volatile("" : "+v"(x)); }

// Lane index from the hardware lane count, recomputed at each use so that
// nothing per-lane has to stay live (or be spilled) to recover it.
__device__ __forceinline__ int lane_id() {
  uint32_t lane;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane));
  return (int)lane;
}

// Load of a value that is the same for the whole wave (uniform pointer and
// index) through the scalar unit: it lands in an SGPR and its wait does not
// share the vector-memory counter with the history stores.
__device__ __forceinline__ float ld_uniform(const float* p, int64_t i) {
  typedef const __attribute__((address_space(4))) float cfloat;
  return ((cfloat*)p)[i];
}

__device__ __forceinline__ int ld_uniform_i(const int32_t* p, int64_t i) {
  typedef const __attribute__((address_space(4))) int32_t cint;
  return ((cint*)p)[i];
}

// Thread index rebuilt the same way from the wave index (a scalar).
__device__ __forceinline__ uint32_t lane_tid(uint32_t wave) { return (wave << 6) + (uint32_t)lane_id(); }

__device__ __forceinline__ float read_lane(float v, int lane) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

// One row of a block (w or g) is read 64 entries at a time: lane l of the
// wave holds row[base + l] (0 past the end); a step takes its entry with a
// lane read into a scalar register.
__device__ __forceinline__ float row_chunk(const float* row, int64_t base, int64_t L) {
  const int64_t i = base + (threadIdx.x & 63);
  return i < L ? row[i] : 0.f;
}

// ---------------------------------------------------------------------------
// Reductions over the TPB threads that own one block.  TPB is a power of two.
// Below 64 the threads are an aligned lane segment of one wave; above, whole
// waves, combined through a small LDS area after the caller's barrier.
// Within a wave the tree uses DPP lane permutations (quad xor 1, quad xor 2,
// half-row mirror, row mirror), then the four 16-lane rows are combined in a
// fixed order; every lane ends with bitwise-identical results.
// ---------------------------------------------------------------------------
constexpr int kRed = 8;  // floats per wave in the cross-wave reduction area

struct RedCtx {
  int width;     // lanes combined inside a wave: min(TPB, 64)
  int rw;        // waves per block (1 when TPB <= 64)
  int wave;      // wave index in the workgroup (uniform)
  float* red;    // [waves][kRed] floats
};

template <bool MAX>
__device__ __forceinline__ float red_op(float a, float b) { return MAX ? fmaxf(a, b) : a + b; }

template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// all-reduce over aligned segments of `width` lanes (a power of two <= 64)
template <bool MAX>
__device__ __forceinline__ float seg_reduce(float v, int width) {
  if (width >= 2) v = red_op<MAX>(v, dpp<0xB1>(v));   // quad_perm [1,0,3,2]
  if (width >= 4) v = red_op<MAX>(v, dpp<0x4E>(v));   // quad_perm [2,3,0,1]
  if (width >= 8) v = red_op<MAX>(v, dpp<0x141>(v));  // row_half_mirror
  if (width >= 16) v = red_op<MAX>(v, dpp<0x140>(v)); // row_mirror
  if (width == 32) v = red_op<MAX>(v, __shfl_xor(v, 16));
  if (width == 64)
    v = red_op<MAX>(red_op<MAX>(read_lane(v, 0), read_lane(v, 16)),
                    red_op<MAX>(read_lane(v, 32), read_lane(v, 48)));
  return v;
}

template <int NQ, unsigned MAXMASK>
__device__ __forceinline__ void red_pre(float (&v)[NQ], const RedCtx& r) {
#pragma unroll
  for (int q = 0; q < NQ; ++q)
    v[q] = ((MAXMASK >> q) & 1u) ? seg_reduce<true>(v[q], r.width) : seg_reduce<false>(v[q], r.width);
  if (r.rw > 1 && lane_id() == 0) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) r.red[r.wave * kRed + q] = v[q];
  }
}

// call after a barrier that follows red_pre: lane l reads the partial of
// wave (l mod rw) of its block, and the partials are reduced like a segment
template <int NQ, unsigned MAXMASK>
__device__ __forceinline__ void red_post(float (&v)[NQ], const RedCtx& r) {
  if (r.rw > 1) {
    const int src = (r.wave / r.rw) * r.rw + (lane_id() & (r.rw - 1));
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const float x = r.red[src * kRed + q];
      v[q] = ((MAXMASK >> q) & 1u) ? seg_reduce<true>(x, r.rw) : seg_reduce<false>(x, r.rw);
    }
  }
}

// (max, scaled sum) pairs: combine((m1,s1),(m2,s2)) = (M, s1 2^(m1-M) + s2 2^(m2-M))
__device__ __forceinline__ void lse_pair(float& m, float& s, float mo, float so) {
  const float M = fmaxf(m, mo);
  s = s * ex2(m - M) + so * ex2(mo - M);
  m = M;
}

__device__ __forceinline__ void lse_pre(float& m, float& s, const RedCtx& r) {
  for (int off = 1; off < r.width; off <<= 1) {
    const float mo = __shfl_xor(m, off);
    const float so = __shfl_xor(s, off);
    lse_pair(m, s, mo, so);
  }
  if (r.rw > 1 && lane_id() == 0) {
    r.red[r.wave * kRed + 0] = m;
    r.red[r.wave * kRed + 1] = s;
  }
}

__device__ __forceinline__ void lse_post(float& m, float& s, const RedCtx& r) {
  if (r.rw > 1) {
    const int first = (r.wave / r.rw) * r.rw;
    m = r.red[first * kRed + 0];
    s = r.red[first * kRed + 1];
    for (int i = 1; i < r.rw; ++i) lse_pair(m, s, r.red[(first + i) * kRed + 0], r.red[(first + i) * kRed + 1]);
  }
}

// (max, scaled sum, scaled weighted sum) triples, combined like lse_pair
__device__ __forceinline__ void lse3_pair(float& m, float& s, float& y, float mo, float so, float yo) {
  const float M = fmaxf(m, mo);
  const float f = ex2(m - M), fo = ex2(mo - M);
  s = s * f + so * fo;
  y = y * f + yo * fo;
  m = M;
}

__device__ __forceinline__ void lse3_pre(float& m, float& s, float& y, const RedCtx& r) {
  for (int off = 1; off < r.width; off <<= 1) {
    const float mo = __shfl_xor(m, off);
    const float so = __shfl_xor(s, off);
    const float yo = __shfl_xor(y, off);
    lse3_pair(m, s, y, mo, so, yo);
  }
  if (r.rw > 1 && lane_id() == 0) {
    r.red[r.wave * kRed + 0] = m;
    r.red[r.wave * kRed + 1] = s;
    r.red[r.wave * kRed + 2] = y;
  }
}

__device__ __forceinline__ void lse3_post(float& m, float& s, float& y, const RedCtx& r) {
  if (r.rw > 1) {
    const int first = (r.wave / r.rw) * r.rw;
    m = r.red[first * kRed + 0];
    s = r.red[first * kRed + 1];
    y = r.red[first * kRed + 2];
    for (int i = 1; i < r.rw; ++i)
      lse3_pair(m, s, y, r.red[(first + i) * kRed + 0], r.red[(first + i) * kRed + 1],
                r.red[(first + i) * kRed + 2]);
  }
}

}  // namespace

}  // namespace bcjr
