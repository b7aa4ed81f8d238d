// Float32 products of the full-precision (mixed precision switched off)
// linear layers: the kernels live in gemm_f32.hip, the C ABI entry points
// (mpx_linear_fwd / mpx_linear_bwd with MPX_F32) in gemm.hip.  Internal.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mpx {

// C[M,N] = opA(m,k) opB(k,n) summed over k in float32, with the epilogue of
// the half products applied in float32:
//   v = acc + bias[n];  pre[m,n] = v;  v = gelu(v) (act);  v *= gelu'(dact[m,n]);
//   v += resid[m,n];  C[m,n] = v        (pre, dact, resid share the row stride ldc)
// opA(m,k) = A[m*lda + k] when ak (k-major), else A[k*lda + m];
// opB(k,n) = B[n*ldb + k] when bk (k-major), else B[k*ldb + n].
// splits > 1: split s sums k in [s*k_split, (s+1)*k_split) into ws[s][M][N]
// (no epilogue); reduce_f32 then adds the splits in order.  Batched (splits
// == 1): entry z = i0 * nb1 + i1 of nbatch offsets A, B, C by i0*s?0 + i1*s?1.
struct GemmF32Args {
  const float* A;
  const float* B;
  float* C;
  float* ws;
  int64_t M, N, K, lda, ldb, ldc;
  int32_t splits;
  int64_t k_split;
  const float* bias;
  const float* resid;
  float* pre;
  const float* dact;
  int32_t act;
  int64_t sA0, sA1, sB0, sB1, sC0, sC1, nb1;
};

hipError_t launch_gemm_f32(const GemmF32Args& g, bool ak, bool bk, int64_t nbatch, hipStream_t s);
// C[i] = sum over s < splits of ws[s*MN + i], in split order
hipError_t launch_splitk_reduce_f32(const float* ws, int splits, int64_t MN, float* C, hipStream_t s);
// out[col] = sum over rows of X[r, col] (dense float32 X), float32 partials
// over row slices in `ws` (colsum_workspace bytes), added in slice order
hipError_t launch_colsum_f32(const float* X, int64_t rows, int64_t cols, float* ws, float* out,
                             hipStream_t s);

}  // namespace mpx
