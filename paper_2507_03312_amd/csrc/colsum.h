// Deterministic column sums of row-major matrices (bias gradients, the
// LayerNorm parameter gradients): float32 partial sums over fixed row slices,
// then a second pass that adds the slices in slice order and rounds once.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.h"

namespace mpx {

// Phase 1 over a half matrix X [rows, cols] (dense): part[s][col] = sum of the
// rows of slice s.  Workgroup: 32 column groups of 8 x 8 row lanes; grid
// (ceil(cols / 256), slices).  VEC requires cols % 8 == 0 and a 16-byte
// aligned X; otherwise each lane owns single columns.
template <int DT, bool VEC>
__global__ __launch_bounds__(256) void colsum_partial_kernel(const uint16_t* __restrict__ X, int64_t rows,
                                                             int64_t cols, int64_t rows_per,
                                                             float* __restrict__ part) {
  __shared__ float red[8][256];
  const int cg = threadIdx.x & 31, rl = threadIdx.x >> 5;
  const int64_t c0 = (int64_t)blockIdx.x * 256 + cg * 8;
  const int64_t r0 = (int64_t)blockIdx.y * rows_per;
  const int64_t r1 = min(rows, r0 + rows_per);
  float s[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) s[j] = 0.0f;
  if (VEC) {
    if (c0 < cols) {
#pragma unroll 4
      for (int64_t r = r0 + rl; r < r1; r += 8) {
        const uint4 u = *reinterpret_cast<const uint4*>(X + r * cols + c0);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          s[2 * j] += h2f<DT>((uint16_t)(w[j] & 0xFFFFu));
          s[2 * j + 1] += h2f<DT>((uint16_t)(w[j] >> 16));
        }
      }
    }
  } else {
    for (int64_t r = r0 + rl; r < r1; r += 8)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (c0 + j < cols) s[j] += h2f<DT>(X[r * cols + c0 + j]);
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) red[rl][cg * 8 + j] = s[j];
  __syncthreads();
  const int c = threadIdx.x;  // 256 columns of this block
  const int64_t col = (int64_t)blockIdx.x * 256 + c;
  if (col < cols) {
    float t = 0.0f;
#pragma unroll
    for (int k = 0; k < 8; ++k) t += red[k][c];
    part[(int64_t)blockIdx.y * cols + col] = t;
  }
}

// Phase 2: out[col] = half(sum_s part[s][col]) over nparts slices, in slice
// order within each of 4 interleaved lanes, lanes combined in lane order.
// Non-finite results are added to *nonfinite when it is set.
template <int DT>
__global__ __launch_bounds__(256) void colsum_final_kernel(const float* __restrict__ part, int nparts,
                                                           int64_t cols, uint16_t* __restrict__ out0,
                                                           uint16_t* __restrict__ out1, int64_t split,
                                                           int32_t* __restrict__ nonfinite) {
  // 32 columns per workgroup, 8 lanes per column: lane group q sums partials
  // q, q + 8, ... in order, then the 8 group sums are added pairwise in a
  // fixed tree
  __shared__ float red[8][32];
  const int c = threadIdx.x & 31, q = threadIdx.x >> 5;
  const int64_t col = (int64_t)blockIdx.x * 32 + c;
  float s = 0.0f;
  if (col < cols) {
#pragma unroll 8
    for (int p = q; p < nparts; p += 8) s += part[(int64_t)p * cols + col];
  }
  red[q][c] = s;
  __syncthreads();
  if (q == 0 && col < cols) {
    const float t = ((red[0][c] + red[1][c]) + (red[2][c] + red[3][c])) +
                    ((red[4][c] + red[5][c]) + (red[6][c] + red[7][c]));
    // columns [0, split) go to out0, [split, cols) to out1 (two results of one pass)
    const uint16_t h = f2h<DT>(t);
    if (col < split) out0[col] = h;
    else out1[col - split] = h;
    if (nonfinite) add_nonfinite(nonfinite, h_nonfinite<DT>(h) ? 1 : 0);
  }
}

// launch shape of colsum_final_kernel for `cols` columns
inline unsigned colsum_final_blocks(int64_t cols) { return (unsigned)((cols + 31) / 32); }

inline int64_t colsum_slices(int64_t rows, int64_t cols) {
  const int64_t gx = (cols + 255) / 256;
  int64_t s = std::max<int64_t>(1, std::min<int64_t>(rows / 64, 1024 / gx));
  return std::min<int64_t>(s, 512);
}

inline size_t colsum_workspace(int64_t rows, int64_t cols) {
  return (size_t)colsum_slices(rows, cols) * cols * sizeof(float);
}

// out[col] = half(sum_r X[r, col]) for a dense half matrix; non-finite
// results are added to *nonfinite when it is set.
template <int DT>
inline hipError_t colsum_run(const uint16_t* X, int64_t rows, int64_t cols, float* ws, uint16_t* out,
                             int32_t* nonfinite, hipStream_t s) {
  const int64_t sl = colsum_slices(rows, cols);
  const int64_t per = (rows + sl - 1) / sl;
  dim3 g1((unsigned)((cols + 255) / 256), (unsigned)sl);
  const bool vec = cols % 8 == 0 && (reinterpret_cast<uintptr_t>(X) & 15u) == 0;
  if (vec)
    colsum_partial_kernel<DT, true><<<g1, 256, 0, s>>>(X, rows, cols, per, ws);
  else
    colsum_partial_kernel<DT, false><<<g1, 256, 0, s>>>(X, rows, cols, per, ws);
  colsum_final_kernel<DT><<<colsum_final_blocks(cols), 256, 0, s>>>(ws, (int)sl, cols, out, nullptr,
                                                                       cols, nonfinite);
  return hipGetLastError();
}

}  // namespace mpx
