// Device-side helpers shared by the gfx950 kernels of the jagged HSTU
// attention library: MFMA operand types, bf16 packing, the relative-time
// bucket rule, SiLU and its derivative.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "internal.h"

namespace hstu {

// 64-bit fixed-point value of v (FIX_ONE per unit, rounded to nearest) for
// the deterministic table-gradient sums: integer additions give the same
// result in any order.  |v| < 2^31.
__device__ __forceinline__ unsigned long long to_fix(float v) {
  return (unsigned long long)(long long)__builtin_rint((double)v * FIX_ONE);
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

// 32x32x16 bf16 MFMA, fp32 accumulate.  Operand layout (wave64):
//   A [32 x 16]: lane l holds row l%32, k-slots 8*(l/32) .. +7
//   B [16 x 32]: lane l holds col l%32, k-slots 8*(l/32) .. +7
//   C [32 x 32]: lane l holds col l%32, rows 8*(r/4) + 4*(l/32) + r%4, r=0..15
__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Row index (within a 32x32 C block) of accumulator register r of lane group g.
__device__ __forceinline__ constexpr int c_row(int r, int g) {
  return 8 * (r >> 2) + 4 * g + (r & 3);
}

// bf16 bits -> float.
__device__ __forceinline__ float bf2f(u16 x) {
  return __uint_as_float(((uint32_t)x) << 16);
}

// Two floats -> packed bf16 pair (round to nearest even, hardware cvt).
__device__ __forceinline__ uint32_t pack2(float a, float b) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  bf16x2 r;
  r[0] = (__bf16)a;
  r[1] = (__bf16)b;
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 x) {
  return __builtin_bit_cast(bf16x8, x);
}

// Relative-time bucket: |x| < 4 -> |x|; otherwise four log-spaced buckets per
// octave, 4*(e-1) + (two bits below the leading one) with e = floor(log2|x|);
// clamped to nb-1.  Integer-only, so every device and the host agree.
__device__ __forceinline__ int time_bucket(int64_t delta, int nb) {
  uint64_t x = delta < 0 ? (uint64_t)0 - (uint64_t)delta : (uint64_t)delta;
  int b;
  if (x < 4) {
    b = (int)x;
  } else {
    int e = 63 - __clzll((long long)x);
    b = 4 * (e - 1) + (int)((x >> (e - 2)) & 3u);
  }
  return b < nb - 1 ? b : nb - 1;
}

// Work-group barrier that orders LDS only: it waits for this wave's
// outstanding LDS operations, not for its global loads, stores or atomics
// (__syncthreads waits for those too).  For kernels whose threads exchange
// data through LDS alone, so that fire-and-forget global atomics and
// prefetch loads stay in flight across the barrier.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Raw buffer loads: a resource over `bytes` bytes from `base` and a per-lane
// byte offset; loads at or past `bytes` return 0.  The offset is a plain
// 32-bit register, so a loop that moves the base keeps one register per load
// instead of a 64-bit address.  `base` and `bytes` must be the same in every
// lane of the wave: they are read from the first active lane, which puts the
// resource in scalar registers (the compiler cannot always prove a work-group
// item's base uniform and would otherwise loop over lanes around each load).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
  void *ub = (void *)(uintptr_t)(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, 0, (int)__builtin_amdgcn_readfirstlane(bytes),
                                           0x00020000);
}
__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  typedef unsigned u32x4b __attribute__((ext_vector_type(4)));
  const u32x4b v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// Cross-lane moves inside rows of 16 lanes (DPP on the vector ALU): lane l
// receives x from lane l + K (row_shl) or l - K (row_shr) of its own row,
// and 0 where that lane lies outside the row (the bound control reads 0
// there, so no register has to be cleared first).  Every lane of the row
// must be active.
template <int K>
__device__ __forceinline__ float row_shl(float x) {
  static_assert(K >= 1 && K <= 15, "row shift");
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
      0, __builtin_bit_cast(int, x), 0x100 + K, 0xF, 0xF, true));
}
template <int K>
__device__ __forceinline__ float row_shr(float x) {
  static_assert(K >= 1 && K <= 15, "row shift");
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(
      0, __builtin_bit_cast(int, x), 0x110 + K, 0xF, 0xF, true));
}

// sigma(x) = 1 / (1 + e^-x) = 1 / (1 + 2^(-x log2 e)) in fp32 on the
// hardware exp2 and reciprocal (v_exp_f32, v_rcp_f32).  Saturates cleanly:
// 2^(+large) = inf gives 0, 2^(-large) = 0 gives 1.
__device__ __forceinline__ float sigmoid_f(float x) {
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x * -1.44269504088896341f));
}

// silu(x) = x sigma(x) and its derivative silu'(x) = sigma(x) (1 + x (1 -
// sigma(x))).
__device__ __forceinline__ float silu_f(float x) { return x * sigmoid_f(x); }
__device__ __forceinline__ float dsilu_f(float x) {
  const float sg = sigmoid_f(x);
  return sg * __builtin_fmaf(x, 1.0f - sg, 1.0f);
}

}  // namespace hstu
