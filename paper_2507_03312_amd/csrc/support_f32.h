// Float32 forms of the support ops for full-precision training (MPX's mixed
// precision switched off): the kernels live in support_f32.hip, the C ABI
// entry points (the same calls with MPX_F32) in support.hip.  Internal.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mpx.h"

namespace mpx {

// LayerNorm limit of the float32 backward (the half one's): the gamma / beta
// partials of a workgroup's four waves are combined in LDS
constexpr int64_t kLnF32MaxD = 2048;

hipError_t launch_layernorm_fwd_f32(const float* X, int64_t ldx, const float* gamma,
                                    const float* beta, float* Y, float* mean_rstd, int64_t rows,
                                    int64_t d, hipStream_t s);
// part: nblocks x 2d floats (nblocks = ln_bwd_f32_blocks(rows)); dgamma / dbeta
// (both or neither) from the partials in block order
int64_t ln_bwd_f32_blocks(int64_t rows);
hipError_t launch_layernorm_bwd_f32(const float* X, int64_t ldx, const float* gamma,
                                    const float* dY, const float* Rgrad, float* dX, int64_t ldo,
                                    float* dgamma, float* dbeta, int64_t rows, int64_t d,
                                    float* part, hipStream_t s);
hipError_t launch_softmax_f32(bool bwd, const float* A, const float* Bp, float* O, int64_t rows,
                              int64_t n, int64_t ld, float scale, hipStream_t s);
// row losses into rowloss[B]; dZ seeded with the loss scale
hipError_t launch_cross_entropy_f32(const float* Z, int64_t ldz, const int32_t* labels, int64_t B,
                                    int64_t C, const mpx_scale_state* st, float* rowloss, float* dZ,
                                    hipStream_t s);
hipError_t launch_patchify_f32(const float* img, float* out, int64_t B, int64_t H, int64_t W,
                               int64_t C, int64_t p, hipStream_t s);
hipError_t launch_embed_assemble_f32(const float* E, const float* cls, const float* pos, float* X,
                                     int64_t B, int64_t T, int64_t d, hipStream_t s);
hipError_t launch_embed_assemble_bwd_f32(const float* dX, float* dE, float* dcls, float* dpos,
                                         int64_t B, int64_t T, int64_t d, hipStream_t s);

}  // namespace mpx
