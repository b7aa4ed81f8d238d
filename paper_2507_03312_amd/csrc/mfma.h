// Shared device helpers of the MFMA kernels (GEMM, fused attention): vector
// types, compile-time loops, the 32x32x16 MFMA, LDS address helpers and the
// quad transpose of accumulator runs.  Internal; not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "common.h"

namespace mpx {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
// Clang vector types for 8- and 16-byte global accesses (a store through the
// HIP uint2 / float4 structs is split into 4-byte stores)
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

// Compile-time loop: f(std::integral_constant<int, I>) for I in [0, N).  The
// accumulator tiles are indexed only with such constants, so they stay in
// registers (a runtime index would force them into scratch memory).
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

template <int DT>
__device__ __forceinline__ f32x16 mfma32(uint4 a, uint4 b, f32x16 c) {
  if constexpr (DT == MPX_F16) {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a),
                                                  __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
}

__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint2 lds_tr_b64(uint32_t addr) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(uintptr_t)addr);
  return __builtin_bit_cast(uint2, v);
}

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 lds_b128(uint32_t addr) {
  const u32x4 v = *(const __attribute__((address_space(3))) u32x4*)(uintptr_t)addr;
  return __builtin_bit_cast(uint4, v);
}

// 4x4 transpose across each group of 4 lanes (two butterfly exchanges
// through DPP quad permutations: lane ^ 1 is quad_perm [1,0,3,2], lane ^ 2 is
// [2,3,0,1]): lane q of the group then holds row q of the 4 x 4 block.
__device__ __forceinline__ void quad_transpose(float (&v)[4], int q4) {
  auto xchg = [&](float& lo, float& hi_v, int st) {
    const bool hi = (q4 & st) != 0;
    const int send = __builtin_bit_cast(int, hi ? lo : hi_v);
    const int got = st == 1 ? __builtin_amdgcn_mov_dpp(send, 0xB1, 0xF, 0xF, false)
                            : __builtin_amdgcn_mov_dpp(send, 0x4E, 0xF, 0xF, false);
    if (hi) lo = __builtin_bit_cast(float, got);
    else hi_v = __builtin_bit_cast(float, got);
  };
  xchg(v[0], v[1], 1);
  xchg(v[2], v[3], 1);
  xchg(v[0], v[2], 2);
  xchg(v[1], v[3], 2);
}

// 16- and 8-byte global accesses through clang vector types
__device__ __forceinline__ uint4 ld_u4(const uint16_t* p) {
  return __builtin_bit_cast(uint4, *reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ u32x2 ld_u2(const uint16_t* p) { return *reinterpret_cast<const u32x2*>(p); }
__device__ __forceinline__ void st_u2(uint16_t* p, u32x2 v) { *reinterpret_cast<u32x2*>(p) = v; }

// Exchange the upper lane half (32..63) of x with the lower lane half of y
// (v_permlane32_swap on both dwords).
__device__ __forceinline__ void half_swap(u32x2& x, u32x2& y) {
  const auto r0 = __builtin_amdgcn_permlane32_swap(x.x, y.x, false, false);
  const auto r1 = __builtin_amdgcn_permlane32_swap(x.y, y.y, false, false);
  x = u32x2{r0[0], r1[0]};
  y = u32x2{r0[1], r1[1]};
}

}  // namespace mpx
