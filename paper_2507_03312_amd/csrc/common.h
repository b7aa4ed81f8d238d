// Internal helpers shared by the HIP sources of libmpx (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "mpx.h"

namespace mpx {

// ---------------------------------------------------------------- errors --

// Per-thread message of the last failing call (mpx_last_error).
void set_error(const std::string& msg);
void clear_error();

#define MPX_REQUIRE(cond, msg)                                  \
  do {                                                          \
    if (!(cond)) {                                              \
      ::mpx::set_error(std::string(__func__) + ": " + (msg));   \
      return MPX_ERR_INVALID;                                   \
    }                                                           \
  } while (0)

#define MPX_HIP(call)                                                              \
  do {                                                                             \
    hipError_t e_ = (call);                                                        \
    if (e_ != hipSuccess) {                                                        \
      ::mpx::set_error(std::string(__func__) + ": " #call ": " + hipGetErrorString(e_)); \
      return MPX_ERR_HIP;                                                          \
    }                                                                              \
  } while (0)

// Check the launch that was just enqueued.
#define MPX_LAUNCHED() MPX_HIP(hipGetLastError())

inline bool is_half(mpx_dtype d) { return d == MPX_F16 || d == MPX_BF16; }

// ------------------------------------------------------- 16-bit formats --

// Round-to-nearest-even float32 -> half bits, via the hardware conversions
// (v_cvt_f16_f32 in the default round-to-nearest-even mode; v_cvt_pk_bf16_f32,
// which rounds to nearest even and keeps NaN a NaN).
template <int DT> __device__ __forceinline__ uint16_t f2h(float x);
template <> __device__ __forceinline__ uint16_t f2h<MPX_F16>(float x) {
  return __builtin_bit_cast(uint16_t, (_Float16)x);
}
template <> __device__ __forceinline__ uint16_t f2h<MPX_BF16>(float x) {
  return __builtin_bit_cast(uint16_t, (__bf16)x);
}

// Exact widening half bits -> float32.
template <int DT> __device__ __forceinline__ float h2f(uint16_t h);
template <> __device__ __forceinline__ float h2f<MPX_F16>(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}
template <> __device__ __forceinline__ float h2f<MPX_BF16>(uint16_t h) {
  return __builtin_bit_cast(float, (uint32_t)h << 16);
}

// Exponent field all ones: +-inf or NaN.
template <int DT> __device__ __forceinline__ bool h_nonfinite(uint16_t h);
template <> __device__ __forceinline__ bool h_nonfinite<MPX_F16>(uint16_t h) {
  return (h & 0x7C00u) == 0x7C00u;
}
template <> __device__ __forceinline__ bool h_nonfinite<MPX_BF16>(uint16_t h) {
  return (h & 0x7F80u) == 0x7F80u;
}

// Number of +-inf / NaN values among the two halves packed in w, without
// branches: a half whose exponent field is all ones, plus one unit of that
// field, is exactly 0x8000 (bit 15 of its 16 bits); any other exponent stays
// below it, and neither sum carries into the next half.
template <int DT> __device__ __forceinline__ int nonfinite2(uint32_t w) {
  constexpr uint32_t EXP = DT == MPX_F16 ? 0x7C007C00u : 0x7F807F80u;
  constexpr uint32_t ONE = DT == MPX_F16 ? 0x04000400u : 0x00800080u;
  return __builtin_popcount(((w & EXP) + ONE) & 0x80008000u);
}

// Adds a lane's count of non-finite results to the device counter *cnt (the
// finite check fused into the kernels that write parameter gradients).  Only
// lanes with something to add issue the (vector) atomic, so a pass whose
// results are all finite leaves the counter untouched.
__device__ __forceinline__ void add_nonfinite(int32_t* cnt, int n) {
  if (n) atomicAdd(cnt, n);
}

// GELU, tanh form, and its derivative, in float32.  With
// sigma = (1 + tanh(u)) / 2 = 1 / (1 + exp(-2u)), u = c (x + a x^3):
//   gelu(x) = x sigma,  gelu'(x) = sigma + 2 x sigma (1 - sigma) c (1 + 3 a x^2).
// The sigmoid form avoids the cancellation of 1 + tanh(u) for negative x.
// sigma = 1 / (1 + exp(-2u)) = 1 / (1 + 2^(x (k1 + k2 x^2))) with
// k1 = -2 c log2(e), k2 = -2 c a log2(e), on the hardware exp2 and
// reciprocal (about 1e-6 relative error in float32, far inside one
// half-precision ulp; exp2 overflowing to +inf gives sigma = 0 as it should).
__device__ __forceinline__ float gelu_sigma(float x) {
  const float k1 = -2.302208198144325f, k2 = -0.1029432395800235f;
  return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x * __builtin_fmaf(k2, x * x, k1)));
}
__device__ __forceinline__ float gelu_tanh(float x) { return x * gelu_sigma(x); }
// gelu'(x) = s + s (1 - s) x (2c + 6ac x^2): four fused operations after sigma
// (s (1 - s) as s - s^2; the bracket as one fma on x^2).
__device__ __forceinline__ float gelu_tanh_grad(float x) {
  const float k2 = 1.5957691216057308f;   // 2c
  const float k6 = 0.21406444881780073f;  // 6ac
  const float s = gelu_sigma(x);
  const float u = __builtin_fmaf(-s, s, s);
  return __builtin_fmaf(u, x * __builtin_fmaf(k6, x * x, k2), s);
}

// ------------------------------------------------------------ reductions --

// Wave-wide reductions in a fixed order, on DPP lane permutations (no LDS
// round trips): pairs (lane ^ 1), then lane ^ 2 (quad permutes), then the
// mirror within 8 lanes and within 16 lanes give every lane its 16-lane row
// total; the four row totals are then read out of lanes 0, 16, 32, 48 and
// combined as (r0 + r1) + (r2 + r3).  The result is the same on every lane.
template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, Op op) {
  auto dpp = [](T x, int ctrl) {
    const int b = __builtin_bit_cast(int, x);
    int r;
    switch (ctrl) {  // the control word must be a constant
      case 0xB1: r = __builtin_amdgcn_mov_dpp(b, 0xB1, 0xF, 0xF, false); break;   // quad_perm [1,0,3,2]
      case 0x4E: r = __builtin_amdgcn_mov_dpp(b, 0x4E, 0xF, 0xF, false); break;   // quad_perm [2,3,0,1]
      case 0x141: r = __builtin_amdgcn_mov_dpp(b, 0x141, 0xF, 0xF, false); break; // row_half_mirror
      default: r = __builtin_amdgcn_mov_dpp(b, 0x140, 0xF, 0xF, false); break;   // row_mirror
    }
    return __builtin_bit_cast(T, r);
  };
  v = op(v, dpp(v, 0xB1));
  v = op(v, dpp(v, 0x4E));
  v = op(v, dpp(v, 0x141));
  v = op(v, dpp(v, 0x140));
  auto lane_val = [&](int l) {
    return __builtin_bit_cast(T, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), l));
  };
  return op(op(lane_val(0), lane_val(16)), op(lane_val(32), lane_val(48)));
}
__device__ __forceinline__ float wave_sum(float v) {
  return wave_reduce(v, [](float a, float b) { return a + b; });
}
__device__ __forceinline__ float wave_max(float v) {
  return wave_reduce(v, [](float a, float b) { return fmaxf(a, b); });
}
__device__ __forceinline__ int wave_sum_int(int v) {
  return wave_reduce(v, [](int a, int b) { return a + b; });
}

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace mpx
