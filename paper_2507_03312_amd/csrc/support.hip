// Support ops of the half-precision forward/backward passes: the
// full-precision islands MPX keeps in float32 (§3.2 force_full_precision:
// sums, means, softmax) — LayerNorm, softmax, the losses — plus the data
// movement of a ViT's token embedding.  Every op widens half inputs to
// float32, computes in float32 and rounds once to half at its output.
#include <hip/hip_runtime.h>

#include <initializer_list>

#include <algorithm>

#include "colsum.h"
#include "common.h"
#include "mfma.h"
#include "support_f32.h"

namespace mpx {

constexpr float kLnEps = 1e-5f;

// ------------------------------------------------------------- LayerNorm --
//
// One wave per row, R rows per wave with all their loads issued before any
// reduction (memory parallelism), VPL 8-element vectors per lane (a row of up
// to 512 * VPL columns).  Lane `lane` owns columns v*512 + lane*8 + j.

template <int VPL>
struct RowVec {
  float x[VPL][8];
};

template <int DT, int VPL>
__device__ __forceinline__ void load_row(const uint16_t* __restrict__ row, int64_t d, int lane,
                                         RowVec<VPL>& r) {
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    const int64_t c = (int64_t)v * 512 + lane * 8;
#pragma unroll
    for (int j = 0; j < 8; ++j) r.x[v][j] = 0.0f;
    if (c + 8 <= d && (reinterpret_cast<uintptr_t>(row + c) & 15u) == 0) {
      const uint4 u = *reinterpret_cast<const uint4*>(row + c);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        r.x[v][2 * j] = h2f<DT>((uint16_t)(w[j] & 0xFFFFu));
        r.x[v][2 * j + 1] = h2f<DT>((uint16_t)(w[j] >> 16));
      }
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (c + j < d) r.x[v][j] = h2f<DT>(row[c + j]);
    }
  }
}

template <int DT, int VPL>
__device__ __forceinline__ void store_row(uint16_t* __restrict__ row, int64_t d, int lane,
                                          const uint16_t (&h)[VPL][8]) {
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    const int64_t c = (int64_t)v * 512 + lane * 8;
    if (c + 8 <= d && (reinterpret_cast<uintptr_t>(row + c) & 15u) == 0) {
      *reinterpret_cast<uint4*>(row + c) =
          make_uint4(h[v][0] | ((uint32_t)h[v][1] << 16), h[v][2] | ((uint32_t)h[v][3] << 16),
                     h[v][4] | ((uint32_t)h[v][5] << 16), h[v][6] | ((uint32_t)h[v][7] << 16));
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (c + j < d) row[c + j] = h[v][j];
    }
  }
}

__device__ __forceinline__ bool col_ok(int64_t d, int lane, int v, int j) {
  return (int64_t)v * 512 + lane * 8 + j < d;
}

// LayerNorm output before rounding, (x - mean) rstd gamma + beta, with the
// last multiply-add fused explicitly and its float32 result kept as such (the
// empty asm): left alone, the compiler may turn the multiply-add and the
// rounding to half into one mixed-precision fma that rounds the exact value
// once, which differs from rounding the float32 value on half-way cases.
// Every kernel that normalises a row (the forward, its fused input-cast
// form, the classifier head) so rounds the same float32 value.
__device__ __forceinline__ float ln_affine(float x, float mean, float rstd, float g, float b) {
  float y = __builtin_fmaf((x - mean) * rstd, g, b);
  asm volatile("" : "+v"(y));
  return y;
}

// The LayerNorm backward's per-element arithmetic with every multiply-add
// written out and every rounded product kept as such (the empty asm), so
// each kernel that evaluates it (one wave per row, rows of 16 or 32 lanes,
// the classifier head) rounds identically whatever the compiler would
// otherwise contract:
//   dxh = dy g (rounded), s1 += dxh, s2 = fma(dxh, xhat, s2),
//   dx = rstd fma(-xhat, m2, fma(dy, g, -m1)) (rounded before the cast),
//   dgamma partial = fma(dy, xhat, p), dbeta partial += dy.
__device__ __forceinline__ float ln_dxh(float dy, float g) {
  float t = dy * g;
  asm volatile("" : "+v"(t));
  return t;
}
__device__ __forceinline__ float ln_dx(float dy, float g, float xh, float m1, float m2, float rstd) {
  float t = rstd * __builtin_fmaf(-xh, m2, __builtin_fmaf(dy, g, -m1));
  asm volatile("" : "+v"(t));
  return t;
}

// mean and 1/sqrt(var + eps) of one row held by a wave (two-pass)
template <int VPL>
__device__ __forceinline__ void row_stats(const RowVec<VPL>& r, int64_t d, int lane, float& mean,
                                          float& rstd) {
  float s = 0.0f;
#pragma unroll
  for (int v = 0; v < VPL; ++v)
#pragma unroll
    for (int j = 0; j < 8; ++j) s += r.x[v][j];
  mean = wave_sum(s) / (float)d;
  float q = 0.0f;
#pragma unroll
  for (int v = 0; v < VPL; ++v)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float c = col_ok(d, lane, v, j) ? r.x[v][j] - mean : 0.0f;
      q = __builtin_fmaf(c, c, q);
    }
  rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + kLnEps);
}

// rows per wave: one row per wave measured faster than two (12608 x 768:
// 10.6 vs 12.9 us; 8320 x 384: 5.9 vs 6.25) and four (17.0, 7.3)
constexpr int kLnRows = 1;

template <int DT, int VPL>
__global__ __launch_bounds__(256) void layernorm_fwd_kernel(const uint16_t* __restrict__ X, int64_t ldx,
                                                            const uint16_t* __restrict__ gamma,
                                                            const uint16_t* __restrict__ beta,
                                                            uint16_t* __restrict__ Y,
                                                            float* __restrict__ mr, int64_t rows,
                                                            int64_t d) {
  const int lane = threadIdx.x & 63;
  const int64_t r0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * kLnRows;
  RowVec<VPL> x[kLnRows];
#pragma unroll
  for (int i = 0; i < kLnRows; ++i)
    if (r0 + i < rows) load_row<DT, VPL>(X + (r0 + i) * ldx, d, lane, x[i]);
  RowVec<VPL> g, b;
  load_row<DT, VPL>(gamma, d, lane, g);
  load_row<DT, VPL>(beta, d, lane, b);
#pragma unroll
  for (int i = 0; i < kLnRows; ++i) {
    if (r0 + i >= rows) break;
    float mean, rstd;
    row_stats<VPL>(x[i], d, lane, mean, rstd);
    uint16_t h[VPL][8];
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) h[v][j] = f2h<DT>(ln_affine(x[i].x[v][j], mean, rstd, g.x[v][j], b.x[v][j]));
    store_row<DT, VPL>(Y + (r0 + i) * d, d, lane, h);
    if (mr && lane == 0) {
      mr[2 * (r0 + i)] = mean;
      mr[2 * (r0 + i) + 1] = rstd;
    }
  }
}

// The input cast (§3.4) fused with the first LayerNorm: each float32 value
// is rounded to half, the half row is written out (the residual stream needs
// it) and normalised exactly as layernorm_fwd_kernel normalises that half
// row, so both outputs are the bits of the cast followed by the LayerNorm.
template <int DT, int VPL>
__global__ __launch_bounds__(256) void layernorm_fwd_cast_kernel(
    const float* __restrict__ X, int64_t ldx, const uint16_t* __restrict__ gamma,
    const uint16_t* __restrict__ beta, uint16_t* __restrict__ Xh, uint16_t* __restrict__ Y,
    float* __restrict__ mr, int64_t rows, int64_t d) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const float* xr = X + r * ldx;
  RowVec<VPL> x;
  uint16_t xh[VPL][8];
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    const int64_t c = (int64_t)v * 512 + lane * 8;
    float f[8];
    if (c + 8 <= d && (reinterpret_cast<uintptr_t>(xr + c) & 15u) == 0) {
      const f32x4 a = *reinterpret_cast<const f32x4*>(xr + c);
      const f32x4 b = *reinterpret_cast<const f32x4*>(xr + c + 4);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        f[j] = a[j];
        f[4 + j] = b[j];
      }
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) f[j] = c + j < d ? xr[c + j] : 0.0f;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      xh[v][j] = f2h<DT>(f[j]);
      x.x[v][j] = col_ok(d, lane, v, j) ? h2f<DT>(xh[v][j]) : 0.0f;
    }
  }
  store_row<DT, VPL>(Xh + r * d, d, lane, xh);
  RowVec<VPL> g, b;
  load_row<DT, VPL>(gamma, d, lane, g);
  load_row<DT, VPL>(beta, d, lane, b);
  float mean, rstd;
  row_stats<VPL>(x, d, lane, mean, rstd);
  uint16_t h[VPL][8];
#pragma unroll
  for (int v = 0; v < VPL; ++v)
#pragma unroll
    for (int j = 0; j < 8; ++j) h[v][j] = f2h<DT>(ln_affine(x.x[v][j], mean, rstd, g.x[v][j], b.x[v][j]));
  store_row<DT, VPL>(Y + r * d, d, lane, h);
  if (mr && lane == 0) {
    mr[2 * r] = mean;
    mr[2 * r + 1] = rstd;
  }
}

// Backward: dX for each row (optionally plus a residual cotangent), and
// per-workgroup column partials of dgamma (sum dy*xhat) and dbeta (sum dy)
// into part[blockIdx][0:d] and part[blockIdx][d:2d].  One wave per row.  The rows stay in registers as packed halves
// (widened to float32 as they are used) and each wave loads its next row while
// it computes the current one; the grid is capped at 512 workgroups of 4
// waves that stride over the rows, which also bounds the gamma / beta
// partials (one pair of float32 rows per workgroup).  Holding four float32
// rows per wave instead left room for one wave per SIMD at d = 768 and ran
// 2.4x slower (79 vs 32 us at 12608 x 768).  A call without gamma / beta
// writes no partials and takes up to 2048 workgroups: more waves in flight
// hide the row loads (25.3 -> 21.4 us at 12608 x 768, 22.6 -> 16.4 at
// 16640 x 384, 11.4 -> 8.8 at 8320 x 384); more partials (1024 or 2048
// workgroups) made the gamma / beta calls slower.
constexpr int kLnBwdWaves = 4;
constexpr int kLnBwdMaxBlocks = 512;
constexpr int kLnBwdDxMaxBlocks = 2048;

template <int VPL>
struct RowH {
  u32x4 w[VPL];  // lane's 8 halves of chunk v (zeros past d)
};

template <int VPL>
__device__ __forceinline__ void load_row_h(const uint16_t* __restrict__ row, int64_t d, int lane,
                                           RowH<VPL>& r) {
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    const int64_t c = (int64_t)v * 512 + lane * 8;
    if (c + 8 <= d && (reinterpret_cast<uintptr_t>(row + c) & 15u) == 0) {
      r.w[v] = *reinterpret_cast<const u32x4*>(row + c);
    } else {
      uint32_t h[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) h[j] = c + j < d ? row[c + j] : 0u;
      r.w[v] = u32x4{h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16)};
    }
  }
}

// element j of a packed chunk, widened
template <int DT>
__device__ __forceinline__ float hx(const u32x4& w, int j) {
  const uint32_t u = w[j >> 1];
  return h2f<DT>((uint16_t)((j & 1) ? (u >> 16) : (u & 0xFFFFu)));
}

// DX: compute dX; PART: write the gamma / beta column partials (either or both).
template <int DT, int VPL, bool DX, bool PART>
__global__ __launch_bounds__(64 * kLnBwdWaves) void layernorm_bwd_kernel(
    const uint16_t* __restrict__ X, int64_t ldx, const uint16_t* __restrict__ gamma,
    const uint16_t* __restrict__ dY, const uint16_t* __restrict__ Rg, uint16_t* __restrict__ dX,
    int64_t ldo, int64_t rows, int64_t d, float* __restrict__ part) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  RowVec<VPL> g;
  load_row<DT, VPL>(gamma, d, lane, g);
  float pg[VPL][8], pb[VPL][8];
#pragma unroll
  for (int v = 0; v < VPL; ++v)
#pragma unroll
    for (int j = 0; j < 8; ++j) pg[v][j] = pb[v][j] = 0.0f;

  const int64_t step = (int64_t)gridDim.x * kLnBwdWaves;
  int64_t r = (int64_t)blockIdx.x * kLnBwdWaves + wave;
  RowH<VPL> x, dy, rg;
  auto load = [&](int64_t i, RowH<VPL>& a, RowH<VPL>& b, RowH<VPL>& c) {
    load_row_h<VPL>(X + i * ldx, d, lane, a);
    load_row_h<VPL>(dY + i * d, d, lane, b);
    if (DX && Rg) load_row_h<VPL>(Rg + i * ldo, d, lane, c);
  };
  // Calls with gamma / beta stride over several rows per wave and load the
  // next row during the current one; a dX-only call has one or two rows per
  // wave and no prefetch, which cuts its registers (108 -> 85) so that more
  // waves are in flight (12608 x 768: 21.2 -> 18.4 us alone, and a faster
  // step, where the call is on the critical path).
  constexpr bool kPrefetch = PART;
  if (kPrefetch && r < rows) load(r, x, dy, rg);
  for (; r < rows; r += step) {
    RowH<VPL> nx, ndy, nrg;
    if (!kPrefetch) load(r, x, dy, rg);
    else if (r + step < rows) load(r + step, nx, ndy, nrg);  // in flight during this row
    RowVec<VPL> xf;
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) xf.x[v][j] = hx<DT>(x.w[v], j);
    float mean, rstd;
    row_stats<VPL>(xf, d, lane, mean, rstd);
    float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float xh = col_ok(d, lane, v, j) ? (xf.x[v][j] - mean) * rstd : 0.0f;
        xf.x[v][j] = xh;
        const float dyv = hx<DT>(dy.w[v], j);
        const float dxh = ln_dxh(dyv, g.x[v][j]);
        s1 += dxh;
        s2 = __builtin_fmaf(dxh, xh, s2);
        if (PART) {
          pg[v][j] = __builtin_fmaf(dyv, xh, pg[v][j]);
          pb[v][j] += dyv;
        }
      }
    if (DX) {
      s1 = wave_sum(s1) / (float)d;
      s2 = wave_sum(s2) / (float)d;
      uint16_t h[VPL][8];
#pragma unroll
      for (int v = 0; v < VPL; ++v)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float dx = ln_dx(hx<DT>(dy.w[v], j), g.x[v][j], xf.x[v][j], s1, s2, rstd);
          uint16_t o = f2h<DT>(dx);
          if (Rg) o = f2h<DT>(hx<DT>(rg.w[v], j) + h2f<DT>(o));
          h[v][j] = o;
        }
      store_row<DT, VPL>(dX + r * ldo, d, lane, h);
    }
    if (kPrefetch) {
      x = nx;
      dy = ndy;
      rg = nrg;
    }
  }
  if (!PART) return;
  // the waves' column partials, combined in wave order through LDS
  __shared__ float red[kLnBwdWaves][2][512];
  float* out = part + (int64_t)blockIdx.x * 2 * d;
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      red[wave][0][lane * 8 + j] = pg[v][j];
      red[wave][1][lane * 8 + j] = pb[v][j];
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 1024; i += 64 * kLnBwdWaves) {
      const int which = i >> 9, c = i & 511;
      const int64_t col = (int64_t)v * 512 + c;
      if (col < d) {
        float t = red[0][which][c];
#pragma unroll
        for (int w = 1; w < kLnBwdWaves; ++w) t += red[w][which][c];
        out[which * d + col] = t;
      }
    }
  }
}

// --------------------------------------- LayerNorm rows of 16 or 32 lanes --
//
// At the ViT widths (d = 384 and 768: 48 and 96 chunks of 8 halves) a
// 64-lane wave per row leaves a quarter of its lane slots empty and the
// grid needs more waves than the chip holds at once.  These kernels give a
// row LPR lanes instead (16 or 32, so 4 or 2 rows per wave, 3 chunks per
// lane) and keep the bits of the one-wave-per-row kernels: there lane l sums
// its chunks l, l + 64, ... in order, each 16-lane row is reduced by the DPP
// tree of wave_reduce and the four row totals are combined as
// (R0 + R1) + (R2 + R3).  Here lane li of a group stands for the wave lanes
// li + LPR k (k < 64 / LPR): it keeps one running sum per such lane in the
// same order (absent chunks add the same zeros), reduces each with the same
// tree over its own 16-lane row, and combines the four results in the same
// order (the two 16-lane halves of a 32-lane group exchanged by a shuffle;
// the sum of two floats does not depend on their order).  Mean, rstd and the
// backward's two row sums therefore carry the same bits, and so does every
// output.  Forward alone: 12608 x 768 rows 11.3 -> 8.0 us, 16640 x 384 8.9 -> 5.8;
// dX alone: 17.7 -> 13.7 and 14.0 -> 9.8.
template <int LPR, int VPL, int NCH>
struct LnGroup {
  static constexpr int K = 64 / LPR;     // wave lanes per lane, rows per wave
  static constexpr int D = 8 * NCH;      // row width
  static_assert(NCH % LPR == 0 && NCH <= 64 * VPL && NCH > 64 * (VPL - 1), "layout");
  // chunk slot (k, v) of lane li holds chunk li + LPR (k + K v) when that is < NCH
  static constexpr bool valid(int k, int v) { return (k + K * v) * LPR < NCH; }
  static __device__ __forceinline__ int chunk(int li, int k, int v) { return li + LPR * (k + K * v); }
};

// one sum over a 16-lane row with the DPP steps of wave_reduce (every lane of
// the row gets the same total)
__device__ __forceinline__ float row16_sum(float v) {
  auto dpp = [](float x, int ctrl) {
    const int b = __builtin_bit_cast(int, x);
    int r;
    switch (ctrl) {
      case 0xB1: r = __builtin_amdgcn_mov_dpp(b, 0xB1, 0xF, 0xF, false); break;
      case 0x4E: r = __builtin_amdgcn_mov_dpp(b, 0x4E, 0xF, 0xF, false); break;
      case 0x141: r = __builtin_amdgcn_mov_dpp(b, 0x141, 0xF, 0xF, false); break;
      default: r = __builtin_amdgcn_mov_dpp(b, 0x140, 0xF, 0xF, false); break;
    }
    return __builtin_bit_cast(float, r);
  };
  v = v + dpp(v, 0xB1);
  v = v + dpp(v, 0x4E);
  v = v + dpp(v, 0x141);
  v = v + dpp(v, 0x140);
  return v;
}

// the whole-row total from the per-wave-lane sums s[k], as wave_sum combines them
template <int LPR>
__device__ __forceinline__ float group_total(const float (&s)[64 / LPR]) {
  if constexpr (LPR == 16) {
    const float r0 = row16_sum(s[0]), r1 = row16_sum(s[1]), r2 = row16_sum(s[2]), r3 = row16_sum(s[3]);
    return (r0 + r1) + (r2 + r3);
  } else {
    static_assert(LPR == 32, "16 or 32 lanes per row");
    const float a = row16_sum(s[0]), b = row16_sum(s[1]);  // R0 | R1 and R2 | R3 by 16-lane half
    return (a + __shfl_xor(a, 16)) + (b + __shfl_xor(b, 16));
  }
}

// a group's row: raw chunks (zeros in absent slots) and their float values
template <int DT, int LPR, int VPL, int NCH>
struct GroupRow {
  using G = LnGroup<LPR, VPL, NCH>;
  u32x4 w[G::K][VPL];
  __device__ __forceinline__ void load(const uint16_t* __restrict__ row, int li) {
#pragma unroll
    for (int k = 0; k < G::K; ++k)
#pragma unroll
      for (int v = 0; v < VPL; ++v)
        w[k][v] = G::valid(k, v) ? *reinterpret_cast<const u32x4*>(row + 8 * G::chunk(li, k, v))
                                 : u32x4{0u, 0u, 0u, 0u};
  }
  __device__ __forceinline__ float f(int k, int v, int j) const {
    return G::valid(k, v) ? hx<DT>(w[k][v], j) : 0.0f;
  }
};

// mean and rstd of a group's row: the arithmetic of row_stats, per wave lane
template <int DT, int LPR, int VPL, int NCH>
__device__ __forceinline__ void group_row_stats(const GroupRow<DT, LPR, VPL, NCH>& x, float& mean,
                                                float& rstd) {
  using G = LnGroup<LPR, VPL, NCH>;
  float s[G::K];
#pragma unroll
  for (int k = 0; k < G::K; ++k) {
    s[k] = 0.0f;
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) s[k] += x.f(k, v, j);
  }
  mean = group_total<LPR>(s) / (float)G::D;
#pragma unroll
  for (int k = 0; k < G::K; ++k) {
    s[k] = 0.0f;
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float c = G::valid(k, v) ? x.f(k, v, j) - mean : 0.0f;
        s[k] = __builtin_fmaf(c, c, s[k]);
      }
  }
  rstd = 1.0f / sqrtf(group_total<LPR>(s) / (float)G::D + kLnEps);
}

template <int DT, int LPR, int VPL, int NCH>
__global__ __launch_bounds__(256) void layernorm_fwd_group_kernel(
    const uint16_t* __restrict__ X, int64_t ldx, const uint16_t* __restrict__ gamma,
    const uint16_t* __restrict__ beta, uint16_t* __restrict__ Y, float* __restrict__ mr, int64_t rows) {
  using G = LnGroup<LPR, VPL, NCH>;
  const int lane = threadIdx.x & 63, li = lane % LPR;
  const int64_t r = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * G::K + lane / LPR;
  const int64_t rc = r < rows ? r : rows - 1;  // the last group of the grid may run past the rows
  GroupRow<DT, LPR, VPL, NCH> x, g, b;
  x.load(X + rc * ldx, li);
  g.load(gamma, li);
  b.load(beta, li);
  float mean, rstd;
  group_row_stats(x, mean, rstd);
  if (r >= rows) return;
#pragma unroll
  for (int k = 0; k < G::K; ++k)
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      if (!G::valid(k, v)) continue;
      uint32_t o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint16_t lo = f2h<DT>(ln_affine(x.f(k, v, 2 * j), mean, rstd, g.f(k, v, 2 * j), b.f(k, v, 2 * j)));
        const uint16_t hi =
            f2h<DT>(ln_affine(x.f(k, v, 2 * j + 1), mean, rstd, g.f(k, v, 2 * j + 1), b.f(k, v, 2 * j + 1)));
        o[j] = lo | ((uint32_t)hi << 16);
      }
      *reinterpret_cast<u32x4*>(Y + r * G::D + 8 * G::chunk(li, k, v)) = u32x4{o[0], o[1], o[2], o[3]};
    }
  if (mr && li == 0) {
    mr[2 * r] = mean;
    mr[2 * r + 1] = rstd;
  }
}

// The input cast fused with the first LayerNorm, in row groups: each float32
// chunk is rounded to half, written out, and normalised as the grouped
// forward normalises that half row (the bits of the cast followed by the
// LayerNorm, as layernorm_fwd_cast_kernel).
template <int DT, int LPR, int VPL, int NCH>
__global__ __launch_bounds__(256) void layernorm_fwd_cast_group_kernel(
    const float* __restrict__ X, int64_t ldx, const uint16_t* __restrict__ gamma,
    const uint16_t* __restrict__ beta, uint16_t* __restrict__ Xh, uint16_t* __restrict__ Y,
    float* __restrict__ mr, int64_t rows) {
  using G = LnGroup<LPR, VPL, NCH>;
  const int lane = threadIdx.x & 63, li = lane % LPR;
  const int64_t r = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * G::K + lane / LPR;
  const int64_t rc = r < rows ? r : rows - 1;
  GroupRow<DT, LPR, VPL, NCH> x, g, b;
#pragma unroll
  for (int k = 0; k < G::K; ++k)
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      if (!G::valid(k, v)) {
        x.w[k][v] = u32x4{0u, 0u, 0u, 0u};
        continue;
      }
      const float* src = X + rc * ldx + 8 * G::chunk(li, k, v);
      const f32x4 lo = *reinterpret_cast<const f32x4*>(src);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(src + 4);
      x.w[k][v] = u32x4{(uint32_t)f2h<DT>(lo[0]) | ((uint32_t)f2h<DT>(lo[1]) << 16),
                        (uint32_t)f2h<DT>(lo[2]) | ((uint32_t)f2h<DT>(lo[3]) << 16),
                        (uint32_t)f2h<DT>(hi[0]) | ((uint32_t)f2h<DT>(hi[1]) << 16),
                        (uint32_t)f2h<DT>(hi[2]) | ((uint32_t)f2h<DT>(hi[3]) << 16)};
    }
  g.load(gamma, li);
  b.load(beta, li);
  float mean, rstd;
  group_row_stats(x, mean, rstd);
  if (r >= rows) return;
#pragma unroll
  for (int k = 0; k < G::K; ++k)
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      if (!G::valid(k, v)) continue;
      const int64_t off = r * G::D + 8 * G::chunk(li, k, v);
      *reinterpret_cast<u32x4*>(Xh + off) = x.w[k][v];
      uint32_t o[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint16_t lo = f2h<DT>(ln_affine(x.f(k, v, 2 * j), mean, rstd, g.f(k, v, 2 * j), b.f(k, v, 2 * j)));
        const uint16_t hi =
            f2h<DT>(ln_affine(x.f(k, v, 2 * j + 1), mean, rstd, g.f(k, v, 2 * j + 1), b.f(k, v, 2 * j + 1)));
        o[j] = lo | ((uint32_t)hi << 16);
      }
      *reinterpret_cast<u32x4*>(Y + off) = u32x4{o[0], o[1], o[2], o[3]};
    }
  if (mr && li == 0) {
    mr[2 * r] = mean;
    mr[2 * r + 1] = rstd;
  }
}

// dX of one group row from its loaded x, dY, gamma (and residual
// cotangent): the arithmetic of layernorm_bwd_kernel's dX, shared by the
// grouped kernels with and without gamma / beta (the same bits either way).
// Returns mean and rstd for the caller's gamma / beta terms.
template <int DT, int LPR, int VPL, int NCH>
__device__ __forceinline__ void group_dx_row(const GroupRow<DT, LPR, VPL, NCH>& x,
                                             const GroupRow<DT, LPR, VPL, NCH>& dy,
                                             const GroupRow<DT, LPR, VPL, NCH>& g,
                                             const GroupRow<DT, LPR, VPL, NCH>& rg, bool has_rg,
                                             uint16_t* __restrict__ out, bool store, int li, float& mean,
                                             float& rstd) {
  using G = LnGroup<LPR, VPL, NCH>;
  group_row_stats(x, mean, rstd);
  float s1[G::K], s2[G::K];
#pragma unroll
  for (int k = 0; k < G::K; ++k) {
    s1[k] = 0.0f;
    s2[k] = 0.0f;
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float xh = G::valid(k, v) ? (x.f(k, v, j) - mean) * rstd : 0.0f;
        const float dxh = ln_dxh(dy.f(k, v, j), g.f(k, v, j));
        s1[k] += dxh;
        s2[k] = __builtin_fmaf(dxh, xh, s2[k]);
      }
  }
  const float m1 = group_total<LPR>(s1) / (float)G::D;
  const float m2 = group_total<LPR>(s2) / (float)G::D;
  if (!store) return;
#pragma unroll
  for (int k = 0; k < G::K; ++k)
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      if (!G::valid(k, v)) continue;
      uint16_t h[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float xh = (x.f(k, v, j) - mean) * rstd;
        const float dx = ln_dx(dy.f(k, v, j), g.f(k, v, j), xh, m1, m2, rstd);
        uint16_t o = f2h<DT>(dx);
        if (has_rg) o = f2h<DT>(rg.f(k, v, j) + h2f<DT>(o));
        h[j] = o;
      }
      *reinterpret_cast<u32x4*>(out + 8 * G::chunk(li, k, v)) =
          u32x4{h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16), h[4] | ((uint32_t)h[5] << 16),
                h[6] | ((uint32_t)h[7] << 16)};
    }
}

// dX alone (the call without gamma / beta), optionally plus a residual
// cotangent: one group row per group, no partials.
template <int DT, int LPR, int VPL, int NCH>
__global__ __launch_bounds__(256) void layernorm_bwd_dx_group_kernel(
    const uint16_t* __restrict__ X, int64_t ldx, const uint16_t* __restrict__ gamma,
    const uint16_t* __restrict__ dY, const uint16_t* __restrict__ Rg, uint16_t* __restrict__ dX,
    int64_t ldo, int64_t rows) {
  using G = LnGroup<LPR, VPL, NCH>;
  const int lane = threadIdx.x & 63, li = lane % LPR;
  const int64_t r = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * G::K + lane / LPR;
  const int64_t rc = r < rows ? r : rows - 1;
  GroupRow<DT, LPR, VPL, NCH> x, dy, g, rg;
  x.load(X + rc * ldx, li);
  dy.load(dY + rc * G::D, li);
  if (Rg) rg.load(Rg + rc * ldo, li);
  g.load(gamma, li);
  float mean, rstd;
  group_dx_row(x, dy, g, rg, Rg != nullptr, dX + rc * ldo, r < rows, li, mean, rstd);
}

// gamma / beta column partials (and dX when DX), grouped: the workgroups
// (at most kLnGroupMaxBlocks) stride over tiles of 4 K rows, each group of a
// wave taking one row of the tile; each lane accumulates its columns' terms
// dy xhat and dy over its group's rows in order, and the 4 K group sums of
// a workgroup are added in group order through LDS into one partial row.
// The gamma / beta call and the full call share this kernel and so give
// the same gamma / beta bits; their dX equals the dX-only kernel's.
// Workgroup cap of the grouped gamma / beta kernel: 256, half the partial
// rows of the one-wave kernel's 512 (one-block step +0.45%, ViT-S and ViT-B
// unchanged).
constexpr int kLnGroupMaxBlocks = 256;
static_assert(kLnGroupMaxBlocks <= kLnBwdMaxBlocks, "the workspace holds kLnBwdMaxBlocks partial rows");

template <int DT, int LPR, int VPL, int NCH, bool DX>
__global__ __launch_bounds__(256) void layernorm_bwd_part_group_kernel(
    const uint16_t* __restrict__ X, int64_t ldx, const uint16_t* __restrict__ gamma,
    const uint16_t* __restrict__ dY, const uint16_t* __restrict__ Rg, uint16_t* __restrict__ dX,
    int64_t ldo, int64_t rows, float* __restrict__ part) {
  using G = LnGroup<LPR, VPL, NCH>;
  constexpr int K = G::K, D = G::D;
  const int lane = threadIdx.x & 63, li = lane % LPR, gi = lane / LPR, w = threadIdx.x >> 6;
  GroupRow<DT, LPR, VPL, NCH> g;
  g.load(gamma, li);
  float pg[K][VPL][8], pb[K][VPL][8];
#pragma unroll
  for (int k = 0; k < K; ++k)
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) pg[k][v][j] = pb[k][v][j] = 0.0f;
  const int64_t stride = (int64_t)gridDim.x * 4 * K;
  for (int64_t base = ((int64_t)blockIdx.x * 4 + w) * K; base < rows; base += stride) {  // uniform
    const int64_t r = base + gi;
    const bool ok = r < rows;
    const int64_t rc = ok ? r : rows - 1;
    GroupRow<DT, LPR, VPL, NCH> x, dy, rg;
    x.load(X + rc * ldx, li);
    dy.load(dY + rc * D, li);
    if (DX && Rg) rg.load(Rg + rc * ldo, li);
    float mean, rstd;
    if (DX) {
      group_dx_row(x, dy, g, rg, Rg != nullptr, dX + rc * ldo, ok, li, mean, rstd);
    } else {
      group_row_stats(x, mean, rstd);
    }
    if (ok) {
#pragma unroll
      for (int k = 0; k < K; ++k)
#pragma unroll
        for (int v = 0; v < VPL; ++v)
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            if (!G::valid(k, v)) continue;
            const float xh = (x.f(k, v, j) - mean) * rstd;
            const float dyv = dy.f(k, v, j);
            pg[k][v][j] = __builtin_fmaf(dyv, xh, pg[k][v][j]);
            pb[k][v][j] += dyv;
          }
    }
  }
  // the 4 K group sums of the workgroup, added in group order
  __shared__ float red[4 * K][2][D];
#pragma unroll
  for (int k = 0; k < K; ++k)
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      if (!G::valid(k, v)) continue;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int col = 8 * G::chunk(li, k, v) + j;
        red[w * K + gi][0][col] = pg[k][v][j];
        red[w * K + gi][1][col] = pb[k][v][j];
      }
    }
  __syncthreads();
  float* out = part + (int64_t)blockIdx.x * 2 * D;
  for (int i = threadIdx.x; i < 2 * D; i += 256) {
    const int which = i / D, col = i - which * D;
    float t = red[0][which][col];
#pragma unroll
    for (int q = 1; q < 4 * K; ++q) t += red[q][which][col];
    out[i] = t;
  }
}

// Whether a call takes the grouped kernels: d of 384 or 768 and every row
// of every operand 16-byte aligned.
static bool ln_grouped(int64_t d, std::initializer_list<const void*> ptrs,
                       std::initializer_list<int64_t> lds) {
  if (d != 384 && d != 768) return false;
  for (const void* p : ptrs)
    if (p && (reinterpret_cast<uintptr_t>(p) & 15u) != 0) return false;
  for (int64_t ld : lds)
    if (ld % 8 != 0) return false;
  return true;
}

static int ln_bwd_blocks(int64_t rows, bool partials = true) {
  const int64_t nb = (rows + kLnBwdWaves - 1) / kLnBwdWaves;
  return (int)std::max<int64_t>(1, std::min<int64_t>(nb, partials ? kLnBwdMaxBlocks : kLnBwdDxMaxBlocks));
}

// --------------------------------------------------------------- softmax --
//
// One wave per row, SM_ROWS rows per wave loaded before any reduction; a row
// of up to 64 * SM_VPL values is held in registers (lane owns c = lane + 64 i).

constexpr int kSmRows = 4;

template <int DT, int VPL>
__global__ __launch_bounds__(256) void softmax_fwd_kernel(const uint16_t* __restrict__ S,
                                                          uint16_t* __restrict__ P, int64_t rows,
                                                          int64_t n, int64_t ld, float scale) {
  const int lane = threadIdx.x & 63;
  const int64_t r0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * kSmRows;
  float z[kSmRows][VPL];
#pragma unroll
  for (int i = 0; i < kSmRows; ++i)
#pragma unroll
    for (int k = 0; k < VPL; ++k) {
      const int64_t c = lane + 64 * k;
      z[i][k] = (r0 + i < rows && c < n) ? scale * h2f<DT>(S[(r0 + i) * ld + c]) : -INFINITY;
    }
#pragma unroll
  for (int i = 0; i < kSmRows; ++i) {
    if (r0 + i >= rows) break;
    float mx = z[i][0];
#pragma unroll
    for (int k = 1; k < VPL; ++k) mx = fmaxf(mx, z[i][k]);
    mx = wave_max(mx);
    float e[VPL], sum = 0.0f;
#pragma unroll
    for (int k = 0; k < VPL; ++k) {
      e[k] = lane + 64 * k < n ? expf(z[i][k] - mx) : 0.0f;
      sum += e[k];
    }
    const float inv = 1.0f / wave_sum(sum);
    uint16_t* p = P + (r0 + i) * ld;
#pragma unroll
    for (int k = 0; k < VPL; ++k) {
      const int64_t c = lane + 64 * k;
      if (c < ld) p[c] = c < n ? f2h<DT>(e[k] * inv) : (uint16_t)0;
    }
    for (int64_t c = lane + 64 * VPL; c < ld; c += 64) p[c] = 0;
  }
}

template <int DT, int VPL>
__global__ __launch_bounds__(256) void softmax_bwd_kernel(const uint16_t* __restrict__ P,
                                                          const uint16_t* __restrict__ dP,
                                                          uint16_t* __restrict__ dS, int64_t rows,
                                                          int64_t n, int64_t ld, float scale) {
  const int lane = threadIdx.x & 63;
  const int64_t r0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * kSmRows;
  float pv[kSmRows][VPL], dv[kSmRows][VPL];
#pragma unroll
  for (int i = 0; i < kSmRows; ++i)
#pragma unroll
    for (int k = 0; k < VPL; ++k) {
      const int64_t c = lane + 64 * k;
      const bool ok = r0 + i < rows && c < n;
      pv[i][k] = ok ? h2f<DT>(P[(r0 + i) * ld + c]) : 0.0f;
      dv[i][k] = ok ? h2f<DT>(dP[(r0 + i) * ld + c]) : 0.0f;
    }
#pragma unroll
  for (int i = 0; i < kSmRows; ++i) {
    if (r0 + i >= rows) break;
    float dot = 0.0f;
#pragma unroll
    for (int k = 0; k < VPL; ++k) dot += dv[i][k] * pv[i][k];
    dot = wave_sum(dot);
    uint16_t* ds = dS + (r0 + i) * ld;
#pragma unroll
    for (int k = 0; k < VPL; ++k) {
      const int64_t c = lane + 64 * k;
      if (c < ld) ds[c] = c < n ? f2h<DT>(scale * pv[i][k] * (dv[i][k] - dot)) : (uint16_t)0;
    }
    for (int64_t c = lane + 64 * VPL; c < ld; c += 64) ds[c] = 0;
  }
}

// ----------------------------------------------------------------- losses --

// One wave per row: the row's loss goes to rowloss[b]; dZ is seeded with the
// loss scale.  A second one-workgroup kernel adds the row losses in order.
template <int DT>
__global__ __launch_bounds__(256) void cross_entropy_kernel(const uint16_t* __restrict__ Z, int64_t ldz,
                                                            const int32_t* __restrict__ labels,
                                                            int64_t B, int64_t C,
                                                            const mpx_scale_state* __restrict__ st,
                                                            float* __restrict__ rowloss,
                                                            uint16_t* __restrict__ dZ) {
  const int lane = threadIdx.x & 63;
  const int64_t b = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;
  const float scale = st->scale;
  const uint16_t* z = Z + b * ldz;
  const int32_t y = labels[b];
  float mx = -INFINITY;
  for (int64_t c = lane; c < C; c += 64) mx = fmaxf(mx, h2f<DT>(z[c]));
  mx = wave_max(mx);
  float se = 0.0f;
  for (int64_t c = lane; c < C; c += 64) se += expf(h2f<DT>(z[c]) - mx);
  se = wave_sum(se);
  const float k = scale / (float)B;
  for (int64_t c = lane; c < C; c += 64) {
    const float pr = expf(h2f<DT>(z[c]) - mx) / se;
    dZ[b * C + c] = f2h<DT>(k * (pr - (c == y ? 1.0f : 0.0f)));
  }
  if (lane == 0) {
    const bool ok = y >= 0 && y < C;  // an out-of-range label gives a NaN loss, never a read
    rowloss[b] = ok ? logf(se) - (h2f<DT>(z[y]) - mx) : NAN;
  }
}

// *loss = (sum of vals[0..n)) / n, summed in a fixed order by one workgroup.
__global__ __launch_bounds__(256) void mean_kernel(const float* __restrict__ vals, int64_t n,
                                                   float* __restrict__ loss) {
  __shared__ float red[256];
  float s = 0.0f;
  for (int64_t i = threadIdx.x; i < n; i += 256) s += vals[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *loss = red[0] / (float)n;
}

// The classifier head of a ViT step in one pass per row: the final LayerNorm
// on the CLS rows, the linear layer to C <= 32 classes, the mean
// cross-entropy with the backward seeded by the loss scale (§3.3, §3.4),
// and the backward through the linear layer and the LayerNorm.  One wave per
// row; every piece repeats the arithmetic, summation order and rounding
// points of the separate kernels, so the results are the same bits:
//   Z = half(LN(x)) as the LayerNorm kernel;
//   logit = half(Z w_c + b_c) as the skinny product kernel (lane l sums
//     k = l, l + 64, ..., then a fixed xor butterfly; Z read back from LDS);
//   dlogit = half(scale / B (softmax - onehot)) as the cross-entropy kernel
//     (lane c holds class c);
//   dZ = half(sum_c dlogit_c W_c) with the classes in order, as the skinny
//     product kernel for a reduction of <= 32;
//   dX = half(LN backward of dZ) as the LayerNorm backward kernel, and the
//     gamma / beta column partials of the same 4-row workgroups.
constexpr int kHeadWaves = 4;
constexpr int kHeadMaxW = 16384;  // C * d halves of W staged in LDS (32 KiB)

template <int DT, int VPL>
__global__ __launch_bounds__(64 * kHeadWaves) void classifier_head_kernel(
    const uint16_t* __restrict__ X, int64_t ldx, const uint16_t* __restrict__ gamma,
    const uint16_t* __restrict__ beta, const uint16_t* __restrict__ W, const uint16_t* __restrict__ bias,
    const int32_t* __restrict__ labels, int64_t B, int64_t d, int C,
    const mpx_scale_state* __restrict__ st, uint16_t* __restrict__ Z, uint16_t* __restrict__ dlogits,
    uint16_t* __restrict__ dX, int64_t ldo, float* __restrict__ rowloss, float* __restrict__ part) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t r = (int64_t)blockIdx.x * kHeadWaves + wave;
  __shared__ uint16_t zrow[kHeadWaves][2048];  // the wave's Z row, read back lane-strided
  __shared__ __attribute__((aligned(16))) uint16_t sW[kHeadMaxW];  // W [C, d], staged once
  {
    // the workgroup's copy of W: 16-byte chunks, every load in flight before
    // the LDS writes (single halves when W is not 16-byte aligned)
    const int n = C * (int)d;
    if ((reinterpret_cast<uintptr_t>(W) & 15u) == 0 && n % 8 == 0) {
      constexpr int PER = kHeadMaxW / 8 / (64 * kHeadWaves);
      u32x4 wv[PER];
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int e = 8 * ((int)threadIdx.x + i * 64 * kHeadWaves);
        wv[i] = e < n ? *reinterpret_cast<const u32x4*>(W + e) : u32x4{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int e = 8 * ((int)threadIdx.x + i * 64 * kHeadWaves);
        if (e < n) *reinterpret_cast<u32x4*>(sW + e) = wv[i];
      }
    } else {
      for (int e = threadIdx.x; e < n; e += 64 * kHeadWaves) sW[e] = W[e];
    }
    __syncthreads();
  }
  RowVec<VPL> g, be;
  load_row<DT, VPL>(gamma, d, lane, g);
  load_row<DT, VPL>(beta, d, lane, be);
  float pg[VPL][8], pb[VPL][8];
#pragma unroll
  for (int v = 0; v < VPL; ++v)
#pragma unroll
    for (int j = 0; j < 8; ++j) pg[v][j] = pb[v][j] = 0.0f;
  if (r < B) {  // uniform over the wave
    RowVec<VPL> x;
    load_row<DT, VPL>(X + r * ldx, d, lane, x);
    float mean, rstd;
    row_stats<VPL>(x, d, lane, mean, rstd);
    uint16_t zh[VPL][8];
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) zh[v][j] = f2h<DT>(ln_affine(x.x[v][j], mean, rstd, g.x[v][j], be.x[v][j]));
    store_row<DT, VPL>(Z + r * d, d, lane, zh);
    uint16_t* zs = zrow[wave];
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (col_ok(d, lane, v, j)) zs[v * 512 + lane * 8 + j] = zh[v][j];
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");

    // logits two classes at a time (two independent chains, each in the
    // skinny product kernel's order: k = lane, lane + 64, ..., then the xor
    // butterfly and lane 0's value)
    float logit = -INFINITY;  // lane c < C: class c
    for (int c = 0; c < C; c += 2) {
      const bool two = c + 1 < C;
      const uint16_t* w0 = sW + c * d;
      const uint16_t* w1 = sW + (two ? c + 1 : c) * d;
      float a0 = 0.0f, a1 = 0.0f;
      for (int k = lane; k < (int)d; k += 64) {
        const float zk = h2f<DT>(zs[k]);
        a0 += zk * h2f<DT>(w0[k]);
        a1 += zk * h2f<DT>(w1[k]);
      }
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) {
        a0 += __shfl_xor(a0, o);
        a1 += __shfl_xor(a1, o);
      }
      const float l0 = h2f<DT>(f2h<DT>(__shfl(a0, 0) + h2f<DT>(bias[c])));
      if (lane == c) logit = l0;
      if (two) {
        const float l1 = h2f<DT>(f2h<DT>(__shfl(a1, 0) + h2f<DT>(bias[c + 1])));
        if (lane == c + 1) logit = l1;
      }
    }
    const float scale = st->scale;
    const int32_t y = labels[r];
    const float mx = wave_max(lane < C ? logit : -INFINITY);
    const float se = wave_sum(lane < C ? expf(logit - mx) : 0.0f);
    const float k = scale / (float)B;
    float dl = 0.0f;
    if (lane < C) {
      const float pr = expf(logit - mx) / se;
      const uint16_t h = f2h<DT>(k * (pr - (lane == y ? 1.0f : 0.0f)));
      dlogits[r * C + lane] = h;
      dl = h2f<DT>(h);
    }
    const bool ok = y >= 0 && y < C;  // an out-of-range label gives a NaN loss, never a read
    const float ly = __shfl(logit, ok ? y : 0);
    if (lane == 0) rowloss[r] = ok ? logf(se) - (ly - mx) : NAN;

    float dz[VPL][8];
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) dz[v][j] = 0.0f;
    const bool wvec = d % 8 == 0;  // W rows 16-byte aligned in LDS: a lane's 8 halves in one read
    for (int c = 0; c < C; ++c) {
      const float dlc = __shfl(dl, c);
      const uint16_t* wr = sW + c * d;
#pragma unroll
      for (int v = 0; v < VPL; ++v) {
        const int64_t c0 = (int64_t)v * 512 + lane * 8;
        if (wvec && c0 + 8 <= d) {
          const u32x4 w8 = *reinterpret_cast<const u32x4*>(wr + c0);
#pragma unroll
          for (int j = 0; j < 8; ++j) dz[v][j] += dlc * hx<DT>(w8, j);
        } else {
#pragma unroll
          for (int j = 0; j < 8; ++j)
            if (col_ok(d, lane, v, j)) dz[v][j] += dlc * h2f<DT>(wr[c0 + j]);
        }
      }
    }
    float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float dyv = h2f<DT>(f2h<DT>(dz[v][j] + 0.0f));  // + 0 as the linear layer's (absent) bias
        dz[v][j] = dyv;
        const float xh = col_ok(d, lane, v, j) ? (x.x[v][j] - mean) * rstd : 0.0f;
        x.x[v][j] = xh;
        const float dxh = ln_dxh(dyv, g.x[v][j]);
        s1 += dxh;
        s2 = __builtin_fmaf(dxh, xh, s2);
        pg[v][j] = __builtin_fmaf(dyv, xh, pg[v][j]);
        pb[v][j] += dyv;
      }
    s1 = wave_sum(s1) / (float)d;
    s2 = wave_sum(s2) / (float)d;
    uint16_t h[VPL][8];
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) h[v][j] = f2h<DT>(ln_dx(dz[v][j], g.x[v][j], x.x[v][j], s1, s2, rstd));
    store_row<DT, VPL>(dX + r * ldo, d, lane, h);
  }
  // the waves' column partials, combined in wave order through LDS
  __shared__ float red[kHeadWaves][2][512];
  float* out = part + (int64_t)blockIdx.x * 2 * d;
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      red[wave][0][lane * 8 + j] = pg[v][j];
      red[wave][1][lane * 8 + j] = pb[v][j];
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 1024; i += 64 * kHeadWaves) {
      const int which = i >> 9, c = i & 511;
      const int64_t col = (int64_t)v * 512 + c;
      if (col < d) {
        float t = red[0][which][c];
#pragma unroll
        for (int w = 1; w < kHeadWaves; ++w) t += red[w][which][c];
        out[which * d + col] = t;
      }
    }
  }
}

// Squared errors of 2048-element blocks into part[block]; dY seeded with the scale.
constexpr int kMseBlock = 2048;

template <int DT>
__global__ __launch_bounds__(256) void mse_kernel(const uint16_t* __restrict__ Y, const uint16_t* __restrict__ T,
                                                  int64_t n, const mpx_scale_state* __restrict__ st,
                                                  float* __restrict__ part, uint16_t* __restrict__ dY) {
  const float k = 2.0f * st->scale / (float)n;
  float acc = 0.0f;
  const int64_t base = (int64_t)blockIdx.x * kMseBlock;
#pragma unroll
  for (int u = 0; u < kMseBlock / 256; ++u) {
    const int64_t i = base + u * 256 + threadIdx.x;
    if (i < n) {
      const float df = h2f<DT>(Y[i]) - h2f<DT>(T[i]);
      acc += df * df;
      dY[i] = f2h<DT>(k * df);
    }
  }
  __shared__ float red[4];
  acc = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

// Float32 form of mse_kernel (full-precision training): same blocks and sums.
__global__ __launch_bounds__(256) void mse_f32_kernel(const float* __restrict__ Y, const float* __restrict__ T,
                                                      int64_t n, const mpx_scale_state* __restrict__ st,
                                                      float* __restrict__ part, float* __restrict__ dY) {
  const float k = 2.0f * st->scale / (float)n;
  float acc = 0.0f;
  const int64_t base = (int64_t)blockIdx.x * kMseBlock;
#pragma unroll
  for (int u = 0; u < kMseBlock / 256; ++u) {
    const int64_t i = base + u * 256 + threadIdx.x;
    if (i < n) {
      const float df = Y[i] - T[i];
      acc += df * df;
      dY[i] = k * df;
    }
  }
  __shared__ float red[4];
  acc = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

// sum of squared errors over blocks, divided by n
__global__ __launch_bounds__(256) void mse_final_kernel(const float* __restrict__ part, int64_t nb,
                                                        int64_t n, float* __restrict__ loss) {
  __shared__ float red[256];
  float s = 0.0f;
  for (int64_t i = threadIdx.x; i < nb; i += 256) s += part[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *loss = red[0] / (float)n;
}

// ------------------------------------------------------------ embeddings --

// Patch vectors: workgroups over (patch, 256 elements of its vector); a
// vector element e = i * (p C) + r is pixel row i of the patch, offset r in
// that row's p C contiguous floats.  32-bit index math (the host checks the
// sizes); patches stride over gridDim.y.
template <int DT>
__global__ __launch_bounds__(256) void patchify_cast_kernel(const float* __restrict__ img,
                                                            uint16_t* __restrict__ out, int B, int H,
                                                            int W, int C, int p) {
  const int pc = p * C, pd = p * pc;
  const int gw = W / p, G = (H / p) * gw;
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= pd) return;
  const int i = e / pc, r = e - i * pc;
  for (int row = blockIdx.y; row < B * G; row += gridDim.y) {
    const int b = row / G, g = row - b * G;
    const int gy = g / gw, gx = g - gy * gw;
    const int64_t src = (((int64_t)b * H + gy * p + i) * W + (int64_t)gx * p) * C + r;
    out[(int64_t)row * pd + e] = f2h<DT>(img[src]);
  }
}

// Token rows: workgroups over (256 columns, row); rows stride over gridDim.y.
template <int DT>
__global__ __launch_bounds__(256) void embed_assemble_kernel(const uint16_t* __restrict__ E,
                                                             const uint16_t* __restrict__ cls,
                                                             const uint16_t* __restrict__ pos,
                                                             uint16_t* __restrict__ X, int B, int T,
                                                             int64_t d) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= d) return;
  for (int row = blockIdx.y; row < B * T; row += gridDim.y) {
    const int b = row / T, t = row - b * T;
    const float base = t == 0 ? h2f<DT>(cls[c]) : h2f<DT>(E[((int64_t)b * (T - 1) + t - 1) * d + c]);
    X[(int64_t)row * d + c] = f2h<DT>(base + h2f<DT>(pos[(int64_t)t * d + c]));
  }
}

// Backward: dE rows are copies of the dX rows t > 0; dpos (and dcls, its
// t = 0 row) are column sums over the batch.  A wave owns 64 consecutive
// (t, c) outputs and the workgroup's four waves split the batch (b = w mod
// 4), so every access is 128 contiguous bytes; the four partial sums are
// added in a fixed order.
template <int DT>
__global__ __launch_bounds__(256) void embed_assemble_bwd_kernel(const uint16_t* __restrict__ dX,
                                                                 uint16_t* __restrict__ dE,
                                                                 uint16_t* __restrict__ dcls,
                                                                 uint16_t* __restrict__ dpos,
                                                                 int64_t B, int64_t T, int64_t d,
                                                                 int32_t* __restrict__ nonfinite) {
  __shared__ float red[4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t total = T * d;
  const int64_t o = (int64_t)blockIdx.x * 64 + lane;
  float s = 0.0f;
  if (o < total) {
    const bool body = o >= d;  // t > 0: a patch token, copied to dE
#pragma unroll 4
    for (int64_t b = w; b < B; b += 4) {
      const uint16_t v = dX[b * total + o];
      s += h2f<DT>(v);
      if (body) dE[b * (total - d) + (o - d)] = v;
    }
  }
  red[w][lane] = s;
  __syncthreads();
  if (w == 0 && o < total) {
    const uint16_t h = f2h<DT>((red[0][lane] + red[1][lane]) + (red[2][lane] + red[3][lane]));
    dpos[o] = h;
    if (o < d) dcls[o] = h;
    // dpos and, for the CLS position, dcls: one or two parameter elements
    if (nonfinite) add_nonfinite(nonfinite, h_nonfinite<DT>(h) ? (o < d ? 2 : 1) : 0);
  }
}

// Vector forms of the three kernels above for the usual shapes (rows of
// 8-element multiples, 16-byte aligned operands): each thread moves 8
// consecutive values (4 in the backward) with 16-byte (8-byte) accesses and
// does the same arithmetic per value, in the same order, as the scalar form.
// ViT-B shapes alone: patchify 35.5 -> 10.2 us, assembly 21.2 -> 7.1, its
// backward 13.9 -> 8.8.  The backward takes the vector form only from 65536
// outputs (T d) on: with ViT-S's 24960 its 98 workgroups ran 13.5 -> 17.2.
template <int DT>
__global__ __launch_bounds__(256) void patchify_cast_vec_kernel(const float* __restrict__ img,
                                                                uint16_t* __restrict__ out, int B, int H,
                                                                int W, int C, int p) {
  const int pc = p * C, pd = p * pc, pd8 = pd / 8;
  const int gw = W / p, G = (H / p) * gw;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)B * G * pd8) return;
  const int row = (int)(t / pd8), e = (int)(t - (int64_t)row * pd8) * 8;
  const int i = e / pc, r = e - i * pc;
  const int b = row / G, g = row - b * G;
  const int gy = g / gw, gx = g - gy * gw;
  const float* src = img + (((int64_t)b * H + gy * p + i) * W + (int64_t)gx * p) * C + r;
  const f32x4 a = *reinterpret_cast<const f32x4*>(src);
  const f32x4 c = *reinterpret_cast<const f32x4*>(src + 4);
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    o[j] = (uint32_t)f2h<DT>(a[2 * j]) | ((uint32_t)f2h<DT>(a[2 * j + 1]) << 16);
    o[2 + j] = (uint32_t)f2h<DT>(c[2 * j]) | ((uint32_t)f2h<DT>(c[2 * j + 1]) << 16);
  }
  *reinterpret_cast<u32x4*>(out + (int64_t)row * pd + e) = u32x4{o[0], o[1], o[2], o[3]};
}

template <int DT>
__global__ __launch_bounds__(256) void embed_assemble_vec_kernel(const uint16_t* __restrict__ E,
                                                                 const uint16_t* __restrict__ cls,
                                                                 const uint16_t* __restrict__ pos,
                                                                 uint16_t* __restrict__ X, int B, int T,
                                                                 int64_t d) {
  const int64_t d8 = d / 8;
  const int64_t t8 = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t8 >= (int64_t)B * T * d8) return;
  const int64_t row = t8 / d8, c = (t8 - row * d8) * 8;
  const int b = (int)(row / T), t = (int)(row - (int64_t)b * T);
  const uint16_t* bsrc = t == 0 ? cls + c : E + ((int64_t)b * (T - 1) + t - 1) * d + c;
  const u32x4 bv = *reinterpret_cast<const u32x4*>(bsrc);
  const u32x4 pv = *reinterpret_cast<const u32x4*>(pos + (int64_t)t * d + c);
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint16_t lo = f2h<DT>(h2f<DT>((uint16_t)(bv[j] & 0xFFFFu)) + h2f<DT>((uint16_t)(pv[j] & 0xFFFFu)));
    const uint16_t hi = f2h<DT>(h2f<DT>((uint16_t)(bv[j] >> 16)) + h2f<DT>((uint16_t)(pv[j] >> 16)));
    o[j] = (uint32_t)lo | ((uint32_t)hi << 16);
  }
  *reinterpret_cast<u32x4*>(X + row * d + c) = u32x4{o[0], o[1], o[2], o[3]};
}

// the backward with 4 consecutive outputs per lane (a wave owns 256)
template <int DT>
__global__ __launch_bounds__(256) void embed_assemble_bwd_vec_kernel(const uint16_t* __restrict__ dX,
                                                                     uint16_t* __restrict__ dE,
                                                                     uint16_t* __restrict__ dcls,
                                                                     uint16_t* __restrict__ dpos,
                                                                     int64_t B, int64_t T, int64_t d,
                                                                     int32_t* __restrict__ nonfinite) {
  __shared__ float red[4][4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t total = T * d;
  const int64_t o = ((int64_t)blockIdx.x * 64 + lane) * 4;
  float s[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (o < total) {
    const bool body = o >= d;  // d % 4 == 0: the 4 outputs are all CLS or all patch tokens
#pragma unroll 4
    for (int64_t b = w; b < B; b += 4) {
      const uint2 v = *reinterpret_cast<const uint2*>(dX + b * total + o);
      s[0] += h2f<DT>((uint16_t)(v.x & 0xFFFFu));
      s[1] += h2f<DT>((uint16_t)(v.x >> 16));
      s[2] += h2f<DT>((uint16_t)(v.y & 0xFFFFu));
      s[3] += h2f<DT>((uint16_t)(v.y >> 16));
      if (body) *reinterpret_cast<uint2*>(dE + b * (total - d) + (o - d)) = v;
    }
  }
#pragma unroll
  for (int e = 0; e < 4; ++e) red[e][w][lane] = s[e];
  __syncthreads();
  if (w == 0 && o < total) {
    uint16_t h[4];
    int bad = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      h[e] = f2h<DT>((red[e][0][lane] + red[e][1][lane]) + (red[e][2][lane] + red[e][3][lane]));
      bad += h_nonfinite<DT>(h[e]) ? (o < d ? 2 : 1) : 0;
    }
    const uint2 hv = make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
    *reinterpret_cast<uint2*>(dpos + o) = hv;
    if (o < d) *reinterpret_cast<uint2*>(dcls + o) = hv;
    // dpos and, for the CLS position, dcls: one or two parameter elements each
    if (nonfinite) add_nonfinite(nonfinite, bad);
  }
}

__global__ __launch_bounds__(256) void gather_rows_kernel(const uint16_t* __restrict__ src, int64_t stride,
                                                          uint16_t* __restrict__ dst, int64_t rows,
                                                          int64_t d) {
  const int64_t total = rows * d;
  for (int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x; o < total; o += (int64_t)gridDim.x * 256) {
    const int64_t r = o / d, c = o % d;
    dst[o] = src[r * stride * d + c];
  }
}

static unsigned grid_for(int64_t total) {
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, 65536));
}

}  // namespace mpx

using namespace mpx;

#define MPX_DT_DISPATCH(dt, KERNEL, grid, block, stream, ...)                         \
  do {                                                                                \
    if ((dt) == MPX_F16)                                                              \
      KERNEL<MPX_F16><<<(grid), (block), 0, (hipStream_t)(stream)>>>(__VA_ARGS__);    \
    else                                                                              \
      KERNEL<MPX_BF16><<<(grid), (block), 0, (hipStream_t)(stream)>>>(__VA_ARGS__);   \
    MPX_LAUNCHED();                                                                   \
  } while (0)

static int vpl_for(int64_t d) { return d <= 512 ? 1 : d <= 1024 ? 2 : 4; }

template <int DT>
static void ln_fwd_launch(int vpl, unsigned grid, hipStream_t s, const uint16_t* X, int64_t ldx,
                          const uint16_t* g, const uint16_t* b, uint16_t* Y, float* mr, int64_t rows,
                          int64_t d) {
  if (vpl == 1) layernorm_fwd_kernel<DT, 1><<<grid, 256, 0, s>>>(X, ldx, g, b, Y, mr, rows, d);
  else if (vpl == 2) layernorm_fwd_kernel<DT, 2><<<grid, 256, 0, s>>>(X, ldx, g, b, Y, mr, rows, d);
  else layernorm_fwd_kernel<DT, 4><<<grid, 256, 0, s>>>(X, ldx, g, b, Y, mr, rows, d);
}

template <int DT>
static void ln_bwd_launch(int vpl, unsigned grid, hipStream_t s, const uint16_t* X, int64_t ldx,
                          const uint16_t* g, const uint16_t* dY, const uint16_t* Rg, uint16_t* dX,
                          int64_t ldo, int64_t rows, int64_t d, float* part) {
  constexpr int NT = 64 * kLnBwdWaves;
#define MPX_LNB(V, DXv, PARTv) \
  layernorm_bwd_kernel<DT, V, DXv, PARTv><<<grid, NT, 0, s>>>(X, ldx, g, dY, Rg, dX, ldo, rows, d, part)
#define MPX_LNB_V(V)                        \
  do {                                      \
    if (dX && part) MPX_LNB(V, true, true); \
    else if (dX) MPX_LNB(V, true, false);   \
    else MPX_LNB(V, false, true);           \
  } while (0)
  if (vpl == 1) MPX_LNB_V(1);
  else if (vpl == 2) MPX_LNB_V(2);
  else MPX_LNB_V(4);
#undef MPX_LNB_V
#undef MPX_LNB
}

extern "C" int mpx_layernorm_fwd(const void* X, int64_t ldx, const void* gamma, const void* beta,
                                 void* Y, float* mean_rstd, int64_t rows, int64_t d, mpx_dtype dt,
                                 void* stream) {
  clear_error();
  MPX_REQUIRE(X && gamma && beta && Y, "NULL argument");
  MPX_REQUIRE(rows >= 1 && d >= 1 && d <= 2048 && ldx >= d, "bad sizes (1 <= d <= 2048, ldx >= d)");
  MPX_REQUIRE(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  if (dt == MPX_F32) {
    MPX_HIP(launch_layernorm_fwd_f32((const float*)X, ldx, (const float*)gamma, (const float*)beta,
                                     (float*)Y, mean_rstd, rows, d, (hipStream_t)stream));
    return MPX_OK;
  }
  hipStream_t s = (hipStream_t)stream;
  if (ln_grouped(d, {X, gamma, beta, Y}, {ldx})) {
    const int rows_per_block = d == 768 ? 8 : 16;  // 4 waves of 2 (32 lanes) or 4 (16 lanes) rows
    const unsigned g2 = (unsigned)((rows + rows_per_block - 1) / rows_per_block);
#define MPX_LNG(DTv, LPR, VPL, NCH)                                                                  \
  layernorm_fwd_group_kernel<DTv, LPR, VPL, NCH><<<g2, 256, 0, s>>>(                                 \
      (const uint16_t*)X, ldx, (const uint16_t*)gamma, (const uint16_t*)beta, (uint16_t*)Y, mean_rstd, rows)
    if (dt == MPX_F16) {
      if (d == 768) MPX_LNG(MPX_F16, 32, 2, 96);
      else MPX_LNG(MPX_F16, 16, 1, 48);
    } else {
      if (d == 768) MPX_LNG(MPX_BF16, 32, 2, 96);
      else MPX_LNG(MPX_BF16, 16, 1, 48);
    }
#undef MPX_LNG
    MPX_LAUNCHED();
    return MPX_OK;
  }
  const unsigned grid = (unsigned)((rows + 4 * kLnRows - 1) / (4 * kLnRows));
  if (dt == MPX_F16)
    ln_fwd_launch<MPX_F16>(vpl_for(d), grid, s, (const uint16_t*)X, ldx, (const uint16_t*)gamma,
                           (const uint16_t*)beta, (uint16_t*)Y, mean_rstd, rows, d);
  else
    ln_fwd_launch<MPX_BF16>(vpl_for(d), grid, s, (const uint16_t*)X, ldx, (const uint16_t*)gamma,
                            (const uint16_t*)beta, (uint16_t*)Y, mean_rstd, rows, d);
  MPX_LAUNCHED();
  return MPX_OK;
}

extern "C" int mpx_layernorm_fwd_cast(const float* X, int64_t ldx, const void* gamma,
                                      const void* beta, void* Xh, void* Y, float* mean_rstd,
                                      int64_t rows, int64_t d, mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(X && gamma && beta && Xh && Y, "NULL argument");
  MPX_REQUIRE(rows >= 1 && d >= 1 && d <= 2048 && ldx >= d, "bad sizes (1 <= d <= 2048, ldx >= d)");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  hipStream_t s = (hipStream_t)stream;
  if (ldx % 4 == 0 && ln_grouped(d, {X, gamma, beta, Xh, Y}, {})) {
    const int rows_per_block = d == 768 ? 8 : 16;
    const unsigned g2 = (unsigned)((rows + rows_per_block - 1) / rows_per_block);
#define MPX_LNGC(DTv, LPR, VPL, NCH)                                                              \
  layernorm_fwd_cast_group_kernel<DTv, LPR, VPL, NCH><<<g2, 256, 0, s>>>(                         \
      X, ldx, (const uint16_t*)gamma, (const uint16_t*)beta, (uint16_t*)Xh, (uint16_t*)Y, mean_rstd, rows)
    if (dt == MPX_F16) {
      if (d == 768) MPX_LNGC(MPX_F16, 32, 2, 96);
      else MPX_LNGC(MPX_F16, 16, 1, 48);
    } else {
      if (d == 768) MPX_LNGC(MPX_BF16, 32, 2, 96);
      else MPX_LNGC(MPX_BF16, 16, 1, 48);
    }
#undef MPX_LNGC
    MPX_LAUNCHED();
    return MPX_OK;
  }
  const unsigned grid = (unsigned)((rows + 3) / 4);
  const int vpl = vpl_for(d);
#define MPX_LNC(DTv, V)                                                                          \
  layernorm_fwd_cast_kernel<DTv, V><<<grid, 256, 0, s>>>(X, ldx, (const uint16_t*)gamma,        \
                                                         (const uint16_t*)beta, (uint16_t*)Xh,  \
                                                         (uint16_t*)Y, mean_rstd, rows, d)
  if (dt == MPX_F16) {
    if (vpl == 1) MPX_LNC(MPX_F16, 1);
    else if (vpl == 2) MPX_LNC(MPX_F16, 2);
    else MPX_LNC(MPX_F16, 4);
  } else {
    if (vpl == 1) MPX_LNC(MPX_BF16, 1);
    else if (vpl == 2) MPX_LNC(MPX_BF16, 2);
    else MPX_LNC(MPX_BF16, 4);
  }
#undef MPX_LNC
  MPX_LAUNCHED();
  return MPX_OK;
}

extern "C" size_t mpx_layernorm_bwd_workspace(int64_t rows, int64_t d) {
  if (rows < 1 || d < 1) return 0;
  return (size_t)ln_bwd_blocks(rows) * 2 * d * sizeof(float);
}

extern "C" int mpx_layernorm_bwd(const void* X, int64_t ldx, const void* gamma, const void* dY,
                                 const void* Rgrad, void* dX, int64_t ldo, void* dgamma, void* dbeta,
                                 int64_t rows, int64_t d, mpx_dtype dt, void* workspace,
                                 size_t ws_bytes, int32_t* d_nonfinite, void* stream) {
  clear_error();
  MPX_REQUIRE(X && gamma && dY, "NULL X, gamma or dY");
  MPX_REQUIRE((dgamma == nullptr) == (dbeta == nullptr), "dgamma and dbeta go together");
  MPX_REQUIRE(dX || dgamma, "nothing to compute: dX, dgamma and dbeta are all NULL");
  MPX_REQUIRE(rows >= 1 && d >= 1 && d <= 2048 && ldx >= d && ldo >= d, "bad sizes");
  MPX_REQUIRE(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  MPX_REQUIRE(dt != MPX_F32 || !d_nonfinite, "d_nonfinite is counted for half gradients only");
  float* part = nullptr;
  if (dgamma) {  // only the gamma / beta gradients use the workspace
    const size_t need = mpx_layernorm_bwd_workspace(rows, d);
    if (!workspace || ws_bytes < need) {
      set_error("mpx_layernorm_bwd: workspace of " + std::to_string(need) + " bytes required");
      return MPX_ERR_WORKSPACE;
    }
    part = (float*)workspace;
  }
  if (dt == MPX_F32) {  // its block count equals ln_bwd_blocks: the same workspace
    MPX_HIP(launch_layernorm_bwd_f32((const float*)X, ldx, (const float*)gamma, (const float*)dY,
                                     (const float*)Rgrad, (float*)dX, ldo, (float*)dgamma,
                                     (float*)dbeta, rows, d, part, (hipStream_t)stream));
    return MPX_OK;
  }
  hipStream_t s = (hipStream_t)stream;
  if (part && ln_grouped(d, {X, gamma, dY, Rgrad, dX}, {ldx, ldo})) {
    const int rows_per_tile = d == 768 ? 8 : 16;
    const int nbg = (int)std::min<int64_t>((rows + rows_per_tile - 1) / rows_per_tile, kLnGroupMaxBlocks);
#define MPX_LNGP(DTv, LPR, VPL, NCH, DXv)                                                                \
  layernorm_bwd_part_group_kernel<DTv, LPR, VPL, NCH, DXv><<<nbg, 256, 0, s>>>(                         \
      (const uint16_t*)X, ldx, (const uint16_t*)gamma, (const uint16_t*)dY, (const uint16_t*)Rgrad,     \
      (uint16_t*)dX, ldo, rows, part)
#define MPX_LNGP_D(DTv, DXv)                        \
  do {                                              \
    if (d == 768) MPX_LNGP(DTv, 32, 2, 96, DXv);    \
    else MPX_LNGP(DTv, 16, 1, 48, DXv);             \
  } while (0)
    const unsigned fin2 = colsum_final_blocks(2 * d);
    if (dt == MPX_F16) {
      if (dX) MPX_LNGP_D(MPX_F16, true);
      else MPX_LNGP_D(MPX_F16, false);
      colsum_final_kernel<MPX_F16><<<fin2, 256, 0, s>>>(part, nbg, 2 * d, (uint16_t*)dgamma, (uint16_t*)dbeta,
                                                        d, d_nonfinite);
    } else {
      if (dX) MPX_LNGP_D(MPX_BF16, true);
      else MPX_LNGP_D(MPX_BF16, false);
      colsum_final_kernel<MPX_BF16><<<fin2, 256, 0, s>>>(part, nbg, 2 * d, (uint16_t*)dgamma, (uint16_t*)dbeta,
                                                         d, d_nonfinite);
    }
#undef MPX_LNGP_D
#undef MPX_LNGP
    MPX_LAUNCHED();
    return MPX_OK;
  }
  if (dX && !part && ln_grouped(d, {X, gamma, dY, Rgrad, dX}, {ldx, ldo})) {
    const int rows_per_block = d == 768 ? 8 : 16;
    const unsigned g2 = (unsigned)((rows + rows_per_block - 1) / rows_per_block);
#define MPX_LNGB(DTv, LPR, VPL, NCH)                                                            \
  layernorm_bwd_dx_group_kernel<DTv, LPR, VPL, NCH><<<g2, 256, 0, s>>>(                         \
      (const uint16_t*)X, ldx, (const uint16_t*)gamma, (const uint16_t*)dY, (const uint16_t*)Rgrad, \
      (uint16_t*)dX, ldo, rows)
    if (dt == MPX_F16) {
      if (d == 768) MPX_LNGB(MPX_F16, 32, 2, 96);
      else MPX_LNGB(MPX_F16, 16, 1, 48);
    } else {
      if (d == 768) MPX_LNGB(MPX_BF16, 32, 2, 96);
      else MPX_LNGB(MPX_BF16, 16, 1, 48);
    }
#undef MPX_LNGB
    MPX_LAUNCHED();
    return MPX_OK;
  }
  const int nb = ln_bwd_blocks(rows, part != nullptr);
  const unsigned fin = colsum_final_blocks(2 * d);
  if (dt == MPX_F16) {
    ln_bwd_launch<MPX_F16>(vpl_for(d), (unsigned)nb, s, (const uint16_t*)X, ldx, (const uint16_t*)gamma,
                           (const uint16_t*)dY, (const uint16_t*)Rgrad, (uint16_t*)dX, ldo, rows, d, part);
    if (part)
      colsum_final_kernel<MPX_F16><<<fin, 256, 0, s>>>(part, nb, 2 * d, (uint16_t*)dgamma, (uint16_t*)dbeta, d,
                                                       d_nonfinite);
  } else {
    ln_bwd_launch<MPX_BF16>(vpl_for(d), (unsigned)nb, s, (const uint16_t*)X, ldx, (const uint16_t*)gamma,
                            (const uint16_t*)dY, (const uint16_t*)Rgrad, (uint16_t*)dX, ldo, rows, d, part);
    if (part)
      colsum_final_kernel<MPX_BF16><<<fin, 256, 0, s>>>(part, nb, 2 * d, (uint16_t*)dgamma, (uint16_t*)dbeta, d,
                                                        d_nonfinite);
  }
  MPX_LAUNCHED();
  return MPX_OK;
}

template <int DT>
static void softmax_launch(bool bwd, int vpl, unsigned grid, hipStream_t s, const uint16_t* A,
                           const uint16_t* Bp, uint16_t* O, int64_t rows, int64_t n, int64_t ld,
                           float scale) {
  if (!bwd) {
    if (vpl == 1) softmax_fwd_kernel<DT, 1><<<grid, 256, 0, s>>>(A, O, rows, n, ld, scale);
    else if (vpl == 2) softmax_fwd_kernel<DT, 2><<<grid, 256, 0, s>>>(A, O, rows, n, ld, scale);
    else if (vpl == 4) softmax_fwd_kernel<DT, 4><<<grid, 256, 0, s>>>(A, O, rows, n, ld, scale);
    else softmax_fwd_kernel<DT, 16><<<grid, 256, 0, s>>>(A, O, rows, n, ld, scale);
  } else {
    if (vpl == 1) softmax_bwd_kernel<DT, 1><<<grid, 256, 0, s>>>(A, Bp, O, rows, n, ld, scale);
    else if (vpl == 2) softmax_bwd_kernel<DT, 2><<<grid, 256, 0, s>>>(A, Bp, O, rows, n, ld, scale);
    else if (vpl == 4) softmax_bwd_kernel<DT, 4><<<grid, 256, 0, s>>>(A, Bp, O, rows, n, ld, scale);
    else softmax_bwd_kernel<DT, 16><<<grid, 256, 0, s>>>(A, Bp, O, rows, n, ld, scale);
  }
}

static int sm_vpl(int64_t n) { return n <= 64 ? 1 : n <= 128 ? 2 : n <= 256 ? 4 : 16; }

extern "C" int mpx_softmax_fwd(const void* S, void* P, int64_t rows, int64_t n, int64_t ld, float scale,
                               mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(S && P, "NULL argument");
  MPX_REQUIRE(rows >= 1 && n >= 1 && n <= 1024 && ld >= n, "bad sizes (1 <= n <= 1024, ld >= n)");
  MPX_REQUIRE(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  if (dt == MPX_F32) {
    MPX_HIP(launch_softmax_f32(false, (const float*)S, nullptr, (float*)P, rows, n, ld, scale,
                               (hipStream_t)stream));
    return MPX_OK;
  }
  const unsigned grid = (unsigned)((rows + 4 * kSmRows - 1) / (4 * kSmRows));
  if (dt == MPX_F16)
    softmax_launch<MPX_F16>(false, sm_vpl(n), grid, (hipStream_t)stream, (const uint16_t*)S, nullptr,
                            (uint16_t*)P, rows, n, ld, scale);
  else
    softmax_launch<MPX_BF16>(false, sm_vpl(n), grid, (hipStream_t)stream, (const uint16_t*)S, nullptr,
                             (uint16_t*)P, rows, n, ld, scale);
  MPX_LAUNCHED();
  return MPX_OK;
}

extern "C" int mpx_softmax_bwd(const void* P, const void* dP, void* dS, int64_t rows, int64_t n,
                               int64_t ld, float scale, mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(P && dP && dS, "NULL argument");
  MPX_REQUIRE(rows >= 1 && n >= 1 && n <= 1024 && ld >= n, "bad sizes (1 <= n <= 1024, ld >= n)");
  MPX_REQUIRE(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  if (dt == MPX_F32) {
    MPX_HIP(launch_softmax_f32(true, (const float*)P, (const float*)dP, (float*)dS, rows, n, ld, scale,
                               (hipStream_t)stream));
    return MPX_OK;
  }
  const unsigned grid = (unsigned)((rows + 4 * kSmRows - 1) / (4 * kSmRows));
  if (dt == MPX_F16)
    softmax_launch<MPX_F16>(true, sm_vpl(n), grid, (hipStream_t)stream, (const uint16_t*)P,
                            (const uint16_t*)dP, (uint16_t*)dS, rows, n, ld, scale);
  else
    softmax_launch<MPX_BF16>(true, sm_vpl(n), grid, (hipStream_t)stream, (const uint16_t*)P,
                             (const uint16_t*)dP, (uint16_t*)dS, rows, n, ld, scale);
  MPX_LAUNCHED();
  return MPX_OK;
}

extern "C" size_t mpx_loss_workspace(int64_t n) {
  if (n < 1) return 0;
  return (size_t)std::max<int64_t>(n, (n + kMseBlock - 1) / kMseBlock) * sizeof(float);
}

extern "C" int mpx_cross_entropy(const void* Z, int64_t ldz, const int32_t* labels, int64_t B,
                                 int64_t C, const mpx_scale_state* d_state, float* d_loss, void* dZ,
                                 mpx_dtype dt, void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  MPX_REQUIRE(Z && labels && d_state && d_loss && dZ, "NULL argument");
  MPX_REQUIRE(B >= 1 && C >= 1 && ldz >= C, "bad sizes");
  MPX_REQUIRE(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  if (!workspace || ws_bytes < mpx_loss_workspace(B)) {
    set_error("mpx_cross_entropy: workspace of " + std::to_string(mpx_loss_workspace(B)) + " bytes required");
    return MPX_ERR_WORKSPACE;
  }
  if (dt == MPX_F32) {
    MPX_HIP(launch_cross_entropy_f32((const float*)Z, ldz, labels, B, C, d_state, (float*)workspace,
                                     (float*)dZ, (hipStream_t)stream));
    mean_kernel<<<1, 256, 0, (hipStream_t)stream>>>((const float*)workspace, B, d_loss);
    MPX_LAUNCHED();
    return MPX_OK;
  }
  MPX_DT_DISPATCH(dt, cross_entropy_kernel, (unsigned)((B + 3) / 4), 256, stream, (const uint16_t*)Z, ldz,
                  labels, B, C, d_state, (float*)workspace, (uint16_t*)dZ);
  mean_kernel<<<1, 256, 0, (hipStream_t)stream>>>((const float*)workspace, B, d_loss);
  MPX_LAUNCHED();
  return MPX_OK;
}

static int64_t head_blocks(int64_t B) { return (B + kHeadWaves - 1) / kHeadWaves; }

extern "C" size_t mpx_classifier_head_workspace(int64_t B, int64_t d) {
  if (B < 1 || d < 1) return 0;
  const int64_t loss = (B + 63) / 64 * 64;  // row losses, then the gamma / beta partials
  return (size_t)(loss + head_blocks(B) * 2 * d) * sizeof(float);
}

extern "C" int mpx_classifier_head(const void* X, int64_t ldx, const void* gamma, const void* beta,
                                   const void* W, const void* b, const int32_t* labels, int64_t B,
                                   int64_t d, int64_t C, const mpx_scale_state* d_state, void* Z,
                                   float* d_loss, void* dlogits, void* dX, int64_t ldo, void* dgamma,
                                   void* dbeta, mpx_dtype dt, void* workspace, size_t ws_bytes,
                                   int32_t* d_nonfinite, void* stream) {
  clear_error();
  MPX_REQUIRE(X && gamma && beta && W && b && labels && d_state && Z && d_loss && dlogits && dX &&
                  dgamma && dbeta,
              "NULL argument");
  MPX_REQUIRE(B >= 1 && d >= 1 && d <= 2048 && ldx >= d && ldo >= d, "bad sizes (1 <= d <= 2048)");
  MPX_REQUIRE(C >= 1 && C <= 32, "C must be in [1, 32]");
  MPX_REQUIRE(B <= 2048, "B must be <= 2048");
  MPX_REQUIRE(C * d <= kHeadMaxW, "C * d must be <= 16384 (W is staged in 32 KiB of LDS)");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  const size_t need = mpx_classifier_head_workspace(B, d);
  if (!workspace || ws_bytes < need) {
    set_error("mpx_classifier_head: workspace of " + std::to_string(need) + " bytes required");
    return MPX_ERR_WORKSPACE;
  }
  float* rowloss = (float*)workspace;
  float* part = rowloss + (B + 63) / 64 * 64;
  const int64_t nb = head_blocks(B);
  hipStream_t s = (hipStream_t)stream;
#define MPX_HEAD(DTv, V)                                                                              \
  classifier_head_kernel<DTv, V><<<(unsigned)nb, 64 * kHeadWaves, 0, s>>>(                           \
      (const uint16_t*)X, ldx, (const uint16_t*)gamma, (const uint16_t*)beta, (const uint16_t*)W,   \
      (const uint16_t*)b, labels, B, d, (int)C, d_state, (uint16_t*)Z, (uint16_t*)dlogits,          \
      (uint16_t*)dX, ldo, rowloss, part)
  const int vpl = vpl_for(d);
  const unsigned fin = colsum_final_blocks(2 * d);
  if (dt == MPX_F16) {
    if (vpl == 1) MPX_HEAD(MPX_F16, 1);
    else if (vpl == 2) MPX_HEAD(MPX_F16, 2);
    else MPX_HEAD(MPX_F16, 4);
    colsum_final_kernel<MPX_F16><<<fin, 256, 0, s>>>(part, (int)nb, 2 * d, (uint16_t*)dgamma, (uint16_t*)dbeta, d,
                                                     d_nonfinite);
  } else {
    if (vpl == 1) MPX_HEAD(MPX_BF16, 1);
    else if (vpl == 2) MPX_HEAD(MPX_BF16, 2);
    else MPX_HEAD(MPX_BF16, 4);
    colsum_final_kernel<MPX_BF16><<<fin, 256, 0, s>>>(part, (int)nb, 2 * d, (uint16_t*)dgamma, (uint16_t*)dbeta, d,
                                                      d_nonfinite);
  }
#undef MPX_HEAD
  mean_kernel<<<1, 256, 0, s>>>(rowloss, B, d_loss);
  MPX_LAUNCHED();
  return MPX_OK;
}

extern "C" int mpx_mse(const void* Y, const void* T, int64_t n, const mpx_scale_state* d_state,
                       float* d_loss, void* dY, mpx_dtype dt, void* workspace, size_t ws_bytes,
                       void* stream) {
  clear_error();
  MPX_REQUIRE(Y && T && d_state && d_loss && dY, "NULL argument");
  MPX_REQUIRE(n >= 1, "n must be >= 1");
  MPX_REQUIRE(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  if (!workspace || ws_bytes < mpx_loss_workspace(n)) {
    set_error("mpx_mse: workspace of " + std::to_string(mpx_loss_workspace(n)) + " bytes required");
    return MPX_ERR_WORKSPACE;
  }
  const int64_t nb = (n + kMseBlock - 1) / kMseBlock;
  if (dt == MPX_F32) {
    mse_f32_kernel<<<(unsigned)nb, 256, 0, (hipStream_t)stream>>>((const float*)Y, (const float*)T, n,
                                                                  d_state, (float*)workspace, (float*)dY);
    mse_final_kernel<<<1, 256, 0, (hipStream_t)stream>>>((const float*)workspace, nb, n, d_loss);
    MPX_LAUNCHED();
    return MPX_OK;
  }
  MPX_DT_DISPATCH(dt, mse_kernel, (unsigned)nb, 256, stream, (const uint16_t*)Y, (const uint16_t*)T, n,
                  d_state, (float*)workspace, (uint16_t*)dY);
  mse_final_kernel<<<1, 256, 0, (hipStream_t)stream>>>((const float*)workspace, nb, n, d_loss);
  MPX_LAUNCHED();
  return MPX_OK;
}

extern "C" int mpx_patchify_cast(const float* images, void* patches, int64_t B, int64_t H, int64_t W,
                                 int64_t C, int64_t p, mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(images && patches, "NULL argument");
  MPX_REQUIRE(B >= 1 && C >= 1 && p >= 1 && H >= p && W >= p && H % p == 0 && W % p == 0,
              "bad sizes (H and W must be multiples of p)");
  MPX_REQUIRE(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  if (dt == MPX_F32) {
    MPX_HIP(launch_patchify_f32(images, (float*)patches, B, H, W, C, p, (hipStream_t)stream));
    return MPX_OK;
  }
  MPX_REQUIRE(B * H * W * C < ((int64_t)1 << 31), "at most 2^31 - 1 image values");
  if ((p * C) % 8 == 0 && (W * C) % 4 == 0 && (reinterpret_cast<uintptr_t>(images) & 15u) == 0 &&
      (reinterpret_cast<uintptr_t>(patches) & 15u) == 0) {
    const int64_t n8 = B * H * W * C / 8;  // one thread per 8 patch values
    MPX_DT_DISPATCH(dt, patchify_cast_vec_kernel, (unsigned)((n8 + 255) / 256), 256, stream, images,
                    (uint16_t*)patches, (int)B, (int)H, (int)W, (int)C, (int)p);
    return MPX_OK;
  }
  {
    const int64_t pd = p * p * C, rows = B * (H / p) * (W / p);
    const dim3 grid((unsigned)((pd + 255) / 256), (unsigned)std::min<int64_t>(rows, 65535));
    MPX_DT_DISPATCH(dt, patchify_cast_kernel, grid, 256, stream, images, (uint16_t*)patches, (int)B,
                    (int)H, (int)W, (int)C, (int)p);
  }
  return MPX_OK;
}

extern "C" int mpx_embed_assemble(const void* E, const void* cls, const void* pos, void* X, int64_t B,
                                  int64_t T, int64_t d, mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(E && cls && pos && X, "NULL argument");
  MPX_REQUIRE(B >= 1 && T >= 2 && d >= 1, "bad sizes");
  MPX_REQUIRE(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  if (dt == MPX_F32) {
    MPX_HIP(launch_embed_assemble_f32((const float*)E, (const float*)cls, (const float*)pos, (float*)X,
                                      B, T, d, (hipStream_t)stream));
    return MPX_OK;
  }
  MPX_REQUIRE(B * T < ((int64_t)1 << 31), "at most 2^31 - 1 token rows");
  auto al16 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 15u) == 0; };
  if (d % 8 == 0 && al16(E) && al16(cls) && al16(pos) && al16(X)) {
    const int64_t n8 = B * T * (d / 8);
    MPX_DT_DISPATCH(dt, embed_assemble_vec_kernel, (unsigned)((n8 + 255) / 256), 256, stream,
                    (const uint16_t*)E, (const uint16_t*)cls, (const uint16_t*)pos, (uint16_t*)X, (int)B,
                    (int)T, d);
    return MPX_OK;
  }
  {
    const dim3 grid((unsigned)((d + 255) / 256), (unsigned)std::min<int64_t>(B * T, 65535));
    MPX_DT_DISPATCH(dt, embed_assemble_kernel, grid, 256, stream, (const uint16_t*)E,
                    (const uint16_t*)cls, (const uint16_t*)pos, (uint16_t*)X, (int)B, (int)T, d);
  }
  return MPX_OK;
}

extern "C" int mpx_embed_assemble_bwd(const void* dX, void* dE, void* dcls, void* dpos, int64_t B,
                                      int64_t T, int64_t d, mpx_dtype dt, int32_t* d_nonfinite,
                                      void* stream) {
  clear_error();
  MPX_REQUIRE(dX && dE && dcls && dpos, "NULL argument");
  MPX_REQUIRE(B >= 1 && T >= 2 && d >= 1, "bad sizes");
  MPX_REQUIRE(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  if (dt == MPX_F32) {
    MPX_REQUIRE(!d_nonfinite, "d_nonfinite is counted for half gradients only");
    MPX_HIP(launch_embed_assemble_bwd_f32((const float*)dX, (float*)dE, (float*)dcls, (float*)dpos, B,
                                          T, d, (hipStream_t)stream));
    return MPX_OK;
  }
  auto al8 = [](const void* q) { return (reinterpret_cast<uintptr_t>(q) & 7u) == 0; };
  if (d % 4 == 0 && T * d >= 65536 && al8(dX) && al8(dE) && al8(dcls) && al8(dpos)) {
    MPX_DT_DISPATCH(dt, embed_assemble_bwd_vec_kernel, (unsigned)((T * d + 255) / 256), 256, stream,
                    (const uint16_t*)dX, (uint16_t*)dE, (uint16_t*)dcls, (uint16_t*)dpos, B, T, d,
                    d_nonfinite);
    return MPX_OK;
  }
  MPX_DT_DISPATCH(dt, embed_assemble_bwd_kernel, (unsigned)((T * d + 63) / 64), 256, stream,
                  (const uint16_t*)dX, (uint16_t*)dE, (uint16_t*)dcls, (uint16_t*)dpos, B, T, d,
                  d_nonfinite);
  return MPX_OK;
}

extern "C" int mpx_gather_rows(const void* src, int64_t stride_rows, void* dst, int64_t rows, int64_t d,
                               mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(src && dst, "NULL argument");
  MPX_REQUIRE(rows >= 1 && d >= 1 && stride_rows >= 1, "bad sizes");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  gather_rows_kernel<<<grid_for(rows * d), 256, 0, (hipStream_t)stream>>>(
      (const uint16_t*)src, stride_rows, (uint16_t*)dst, rows, d);
  MPX_LAUNCHED();
  return MPX_OK;
}
