// Float32 GEMMs on the float32 MFMA (v_mfma_f32_32x32x2_f32) for full-precision
// training, the baseline MPX's mixed precision is measured against (§4: full
// precision vs mixed precision).  The structure follows the half kernels in a
// simpler form: 128 x 128 output tiles, four waves of 64 x 64 (2 x 2 blocks
// of 32 x 32), k tiles of 16 staged through registers into double-buffered
// LDS (one barrier per k tile), the same epilogue operations in float32.
#include "gemm_f32.h"

#include <algorithm>

#include "colsum.h"
#include "common.h"
#include "mfma.h"

namespace mpx {

namespace {

constexpr int kBM = 128, kBN = 128, kBK = 16;
// LDS rows of 128 floats padded to 160: the two half-waves of an operand read
// (k and k + 1) fall 32 banks apart
constexpr int kPitch = 160;

// One operand tile (128 rows of the output dimension x 16 k) into registers
// and then into LDS as [k][row].  KMAJ: element (r, k) at P[r*ld + k]
// (a lane loads 4 consecutive k of one row), otherwise at P[k*ld + r] (4
// consecutive rows of one k).  Out-of-range elements read as zero.
template <bool KMAJ>
struct TileF32 {
  float v[8];
  __device__ __forceinline__ void load(const float* P, int64_t ld, int64_t r0, int64_t rows,
                                       int64_t k0, int64_t kend, bool vec, int tid) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      int64_t r, k;
      if constexpr (KMAJ) {
        r = r0 + (tid >> 2) + 64 * i;
        k = k0 + 4 * (tid & 3);
      } else {
        k = k0 + (tid >> 5) + 8 * i;
        r = r0 + 4 * (tid & 31);
      }
      if (vec && (KMAJ ? (r < rows && k + 4 <= kend) : (k < kend && r + 4 <= rows))) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(P + (KMAJ ? r * ld + k : k * ld + r));
#pragma unroll
        for (int c = 0; c < 4; ++c) v[4 * i + c] = x[c];
      } else {
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const int64_t rr = KMAJ ? r : r + c, kk = KMAJ ? k + c : k;
          v[4 * i + c] = (rr < rows && kk < kend) ? P[KMAJ ? rr * ld + kk : kk * ld + rr] : 0.0f;
        }
      }
    }
  }
  __device__ __forceinline__ void store(float (*S)[kPitch], int tid) const {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      if constexpr (KMAJ) {
        const int r = (tid >> 2) + 64 * i, k = 4 * (tid & 3);
#pragma unroll
        for (int c = 0; c < 4; ++c) S[k + c][r] = v[4 * i + c];
      } else {
        const int k = (tid >> 5) + 8 * i, r = 4 * (tid & 31);
        *reinterpret_cast<f32x4*>(&S[k][r]) = f32x4{v[4 * i], v[4 * i + 1], v[4 * i + 2], v[4 * i + 3]};
      }
    }
  }
};

template <bool AK, bool BKM>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmF32Args g) {
  __shared__ __attribute__((aligned(16))) float sA[2][kBK][kPitch];
  __shared__ __attribute__((aligned(16))) float sB[2][kBK][kPitch];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave >> 1) * 64, wn0 = (wave & 1) * 64;
  const int64_t tiles_n = (g.N + kBN - 1) / kBN;
  const int64_t m0 = (int64_t)(blockIdx.x / tiles_n) * kBM;
  const int64_t n0 = (int64_t)(blockIdx.x % tiles_n) * kBN;
  int split = 0;
  const float* Ap = g.A;
  const float* Bp = g.B;
  int64_t offC = 0;
  if (g.splits > 1) {
    split = (int)blockIdx.y;
  } else {  // batch entry
    const int64_t i0 = blockIdx.y / g.nb1, i1 = blockIdx.y % g.nb1;
    Ap += i0 * g.sA0 + i1 * g.sA1;
    Bp += i0 * g.sB0 + i1 * g.sB1;
    offC = i0 * g.sC0 + i1 * g.sC1;
  }
  const int64_t kbeg = (int64_t)split * g.k_split;
  const int64_t kend = min(g.K, kbeg + g.k_split);
  const int nk = (int)((kend - kbeg + kBK - 1) / kBK);
  const bool va = (reinterpret_cast<uintptr_t>(Ap) & 15u) == 0 && g.lda % 4 == 0;
  const bool vb = (reinterpret_cast<uintptr_t>(Bp) & 15u) == 0 && g.ldb % 4 == 0;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  TileF32<AK> ta;
  TileF32<BKM> tb;
  if (nk > 0) {
    ta.load(Ap, g.lda, m0, g.M, kbeg, kend, va, tid);
    tb.load(Bp, g.ldb, n0, g.N, kbeg, kend, vb, tid);
    ta.store(sA[0], tid);
    tb.store(sB[0], tid);
  }
  __syncthreads();
  const int hk = lane >> 5, l32 = lane & 31;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {  // next k tile into registers while this one is multiplied
      ta.load(Ap, g.lda, m0, g.M, kbeg + (int64_t)(kt + 1) * kBK, kend, va, tid);
      tb.load(Bp, g.ldb, n0, g.N, kbeg + (int64_t)(kt + 1) * kBK, kend, vb, tid);
    }
#pragma unroll
    for (int kk = 0; kk < kBK; kk += 2) {
      // lane l supplies row / column l % 32 at k = kk + l / 32
      const float a0 = sA[buf][kk + hk][wm0 + l32], a1 = sA[buf][kk + hk][wm0 + 32 + l32];
      const float b0 = sB[buf][kk + hk][wn0 + l32], b1 = sB[buf][kk + hk][wn0 + 32 + l32];
      acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, b1, acc[1][1], 0, 0, 0);
    }
    if (more) {  // the other buffer was released by the previous barrier
      ta.store(sA[buf ^ 1], tid);
      tb.store(sB[buf ^ 1], tid);
    }
    __syncthreads();
  }

  // accumulator layout of a 32 x 32 block: lane l holds column l % 32, value r
  // is row 8 (r / 4) + 4 (l / 32) + r % 4
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int64_t n = n0 + wn0 + 32 * j + l32;
      if (n >= g.N) continue;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t m = m0 + wm0 + 32 * i + 8 * (r >> 2) + 4 * hk + (r & 3);
        if (m >= g.M) continue;
        float v = acc[i][j][r];
        if (g.splits > 1) {
          g.ws[((int64_t)split * g.M + m) * g.N + n] = v;
          continue;
        }
        const int64_t o = offC + m * g.ldc + n;
        if (g.bias) v += g.bias[n];
        if (g.pre) g.pre[o] = v;
        if (g.act == MPX_ACT_GELU_TANH) v = gelu_tanh(v);
        if (g.dact) v *= gelu_tanh_grad(g.dact[o]);
        if (g.resid) v += g.resid[o];
        g.C[o] = v;
      }
    }
  }
}

__global__ __launch_bounds__(256) void splitk_reduce_f32_kernel(const float* __restrict__ ws, int splits,
                                                                int64_t MN, float* __restrict__ C) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= MN) return;
  float s = ws[i];
  for (int k = 1; k < splits; ++k) s += ws[(int64_t)k * MN + i];
  C[i] = s;
}

// Column sums of a dense float32 matrix: partial sums over row slices (a
// lane per column, rows of the slice in order), then the slices in order.
__global__ __launch_bounds__(256) void colsum_f32_partial_kernel(const float* __restrict__ X, int64_t rows,
                                                                 int64_t cols, int64_t rows_per,
                                                                 float* __restrict__ part) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (col >= cols) return;
  const int64_t r0 = (int64_t)blockIdx.y * rows_per, r1 = min(rows, r0 + rows_per);
  float s = 0.0f;
  for (int64_t r = r0; r < r1; ++r) s += X[r * cols + col];
  part[(int64_t)blockIdx.y * cols + col] = s;
}

__global__ __launch_bounds__(256) void colsum_f32_final_kernel(const float* __restrict__ part, int64_t nparts,
                                                               int64_t cols, float* __restrict__ out) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (col >= cols) return;
  float s = 0.0f;
  for (int64_t p = 0; p < nparts; ++p) s += part[p * cols + col];
  out[col] = s;
}

}  // namespace

hipError_t launch_gemm_f32(const GemmF32Args& g, bool ak, bool bk, int64_t nbatch, hipStream_t s) {
  const int64_t tiles = ((g.M + kBM - 1) / kBM) * ((g.N + kBN - 1) / kBN);
  const int64_t gy = g.splits > 1 ? g.splits : nbatch;
  if (tiles > 0x7FFFFFFF || g.splits < 1 || gy < 1 || gy > 65535 || g.nb1 < 1 ||
      (g.splits > 1 && nbatch != 1))
    return hipErrorInvalidValue;
  const dim3 grid((unsigned)tiles, (unsigned)gy);
  if (ak && bk) gemm_f32_kernel<true, true><<<grid, 256, 0, s>>>(g);
  else if (ak) gemm_f32_kernel<true, false><<<grid, 256, 0, s>>>(g);
  else if (bk) gemm_f32_kernel<false, true><<<grid, 256, 0, s>>>(g);
  else gemm_f32_kernel<false, false><<<grid, 256, 0, s>>>(g);
  return hipGetLastError();
}

hipError_t launch_splitk_reduce_f32(const float* ws, int splits, int64_t MN, float* C, hipStream_t s) {
  splitk_reduce_f32_kernel<<<(unsigned)((MN + 255) / 256), 256, 0, s>>>(ws, splits, MN, C);
  return hipGetLastError();
}

hipError_t launch_colsum_f32(const float* X, int64_t rows, int64_t cols, float* ws, float* out,
                             hipStream_t s) {
  // the slice count of the half column sum, so the same workspace size serves
  const int64_t sl = colsum_slices(rows, cols);
  const int64_t per = (rows + sl - 1) / sl;
  const unsigned gx = (unsigned)((cols + 255) / 256);
  colsum_f32_partial_kernel<<<dim3(gx, (unsigned)sl), 256, 0, s>>>(X, rows, cols, per, ws);
  colsum_f32_final_kernel<<<gx, 256, 0, s>>>(ws, sl, cols, out);
  return hipGetLastError();
}

}  // namespace mpx
