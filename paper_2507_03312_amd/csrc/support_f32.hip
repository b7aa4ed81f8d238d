// Float32 support ops of full-precision training, the baseline MPX's mixed
// precision is measured against (§4).  Same definitions as the half kernels
// of support.hip (LayerNorm with eps 1e-5, softmax, cross-entropy seeded
// with the loss scale, patch gather, token assembly), every value float32,
// in a plain one-wave-per-row form: these kernels are a baseline, not tuned.
#include "support_f32.h"

#include <math.h>

#include <algorithm>

#include "common.h"

namespace mpx {

namespace {

constexpr float kEps = 1e-5f;

// mean and 1/std of one row (lane owns columns lane + 64 j), two passes
__device__ __forceinline__ void row_stats_f32(const float* __restrict__ x, int64_t d, int lane,
                                              float& mean, float& rstd) {
  float s = 0.0f;
  for (int64_t c = lane; c < d; c += 64) s += x[c];
  mean = wave_sum(s) / (float)d;
  float q = 0.0f;
  for (int64_t c = lane; c < d; c += 64) {
    const float v = x[c] - mean;
    q += v * v;
  }
  rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + kEps);
}

__global__ __launch_bounds__(256) void layernorm_fwd_f32_kernel(const float* __restrict__ X, int64_t ldx,
                                                                const float* __restrict__ gamma,
                                                                const float* __restrict__ beta,
                                                                float* __restrict__ Y,
                                                                float* __restrict__ mr, int64_t rows,
                                                                int64_t d) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const float* x = X + r * ldx;
  float mean, rstd;
  row_stats_f32(x, d, lane, mean, rstd);
  for (int64_t c = lane; c < d; c += 64) Y[r * d + c] = (x[c] - mean) * rstd * gamma[c] + beta[c];
  if (mr && lane == 0) {
    mr[2 * r] = mean;
    mr[2 * r + 1] = rstd;
  }
}

// dX = rstd (g - mean(g) - xhat mean(g xhat)) [+ Rgrad] with g = dY gamma;
// the gamma / beta column sums (dY xhat, dY) of the rows a workgroup's four
// waves visit go to part[block][0:d] and part[block][d:2d], the waves'
// register sums combined in LDS in wave order.

// CPL columns per lane (16 up to d = 1024, 32 up to 2048), one running
// gamma / beta sum per column
template <int CPL>
__global__ __launch_bounds__(256) void layernorm_bwd_f32_kernel(
    const float* __restrict__ X, int64_t ldx, const float* __restrict__ gamma,
    const float* __restrict__ dY, const float* __restrict__ Rg, float* __restrict__ dX, int64_t ldo,
    int64_t rows, int64_t d, float* __restrict__ part) {
  constexpr int kCpl = CPL;
  __shared__ float red[4][2 * 64 * CPL];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float pg[kCpl], pb[kCpl];
#pragma unroll
  for (int j = 0; j < kCpl; ++j) pg[j] = pb[j] = 0.0f;
  for (int64_t r = (int64_t)blockIdx.x * 4 + wave; r < rows; r += (int64_t)gridDim.x * 4) {
    const float* x = X + r * ldx;
    const float* dy = dY + r * d;
    float mean, rstd;
    row_stats_f32(x, d, lane, mean, rstd);
    float sg = 0.0f, sgx = 0.0f;
#pragma unroll
    for (int j = 0; j < kCpl; ++j) {
      const int64_t c = lane + 64 * j;
      if (c < d) {
        const float xh = (x[c] - mean) * rstd, g = dy[c] * gamma[c];
        sg += g;
        sgx += g * xh;
        pg[j] += dy[c] * xh;
        pb[j] += dy[c];
      }
    }
    const float mg = wave_sum(sg) / (float)d, mgx = wave_sum(sgx) / (float)d;
    if (dX) {
      for (int64_t c = lane; c < d; c += 64) {
        const float xh = (x[c] - mean) * rstd;
        float v = rstd * (dy[c] * gamma[c] - mg - xh * mgx);
        if (Rg) v += Rg[r * ldo + c];
        dX[r * ldo + c] = v;
      }
    }
  }
  if (!part) return;
#pragma unroll
  for (int j = 0; j < kCpl; ++j) {
    const int64_t c = lane + 64 * j;
    if (c < d) {
      red[wave][c] = pg[j];
      red[wave][d + c] = pb[j];
    }
  }
  __syncthreads();
  for (int64_t c = threadIdx.x; c < 2 * d; c += 256)
    part[(int64_t)blockIdx.x * 2 * d + c] = ((red[0][c] + red[1][c]) + red[2][c]) + red[3][c];
}

// dgamma / dbeta: the block partials added in block order
__global__ __launch_bounds__(256) void ln_partials_final_f32_kernel(const float* __restrict__ part,
                                                                    int64_t nb, int64_t d,
                                                                    float* __restrict__ dgamma,
                                                                    float* __restrict__ dbeta) {
  const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= 2 * d) return;
  float s = 0.0f;
  for (int64_t b = 0; b < nb; ++b) s += part[b * 2 * d + c];
  if (c < d) dgamma[c] = s;
  else dbeta[c - d] = s;
}

__global__ __launch_bounds__(256) void softmax_fwd_f32_kernel(const float* __restrict__ S, float* __restrict__ P,
                                                              int64_t rows, int64_t n, int64_t ld, float scale) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const float* s = S + r * ld;
  float* p = P + r * ld;
  float mx = -INFINITY;
  for (int64_t c = lane; c < n; c += 64) mx = fmaxf(mx, scale * s[c]);
  mx = wave_max(mx);
  float sum = 0.0f;
  for (int64_t c = lane; c < n; c += 64) sum += expf(scale * s[c] - mx);
  const float inv = 1.0f / wave_sum(sum);
  for (int64_t c = lane; c < ld; c += 64) p[c] = c < n ? expf(scale * s[c] - mx) * inv : 0.0f;
}

__global__ __launch_bounds__(256) void softmax_bwd_f32_kernel(const float* __restrict__ P,
                                                              const float* __restrict__ dP,
                                                              float* __restrict__ dS, int64_t rows,
                                                              int64_t n, int64_t ld, float scale) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const float* p = P + r * ld;
  const float* dp = dP + r * ld;
  float dot = 0.0f;
  for (int64_t c = lane; c < n; c += 64) dot += dp[c] * p[c];
  dot = wave_sum(dot);
  float* ds = dS + r * ld;
  for (int64_t c = lane; c < ld; c += 64) ds[c] = c < n ? scale * p[c] * (dp[c] - dot) : 0.0f;
}

__global__ __launch_bounds__(256) void cross_entropy_f32_kernel(const float* __restrict__ Z, int64_t ldz,
                                                                const int32_t* __restrict__ labels,
                                                                int64_t B, int64_t C,
                                                                const mpx_scale_state* __restrict__ st,
                                                                float* __restrict__ rowloss,
                                                                float* __restrict__ dZ) {
  const int lane = threadIdx.x & 63;
  const int64_t b = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (b >= B) return;
  const float* z = Z + b * ldz;
  const int32_t y = labels[b];
  float mx = -INFINITY;
  for (int64_t c = lane; c < C; c += 64) mx = fmaxf(mx, z[c]);
  mx = wave_max(mx);
  float se = 0.0f;
  for (int64_t c = lane; c < C; c += 64) se += expf(z[c] - mx);
  se = wave_sum(se);
  const float k = st->scale / (float)B;
  for (int64_t c = lane; c < C; c += 64)
    dZ[b * C + c] = k * (expf(z[c] - mx) / se - (c == y ? 1.0f : 0.0f));
  if (lane == 0) {
    const bool ok = y >= 0 && y < C;  // an out-of-range label gives a NaN loss, never a read
    rowloss[b] = ok ? logf(se) - (z[y] - mx) : NAN;
  }
}

__global__ __launch_bounds__(256) void patchify_f32_kernel(const float* __restrict__ img, float* __restrict__ out,
                                                           int64_t B, int64_t H, int64_t W, int64_t C,
                                                           int64_t p) {
  const int64_t pd = p * p * C;
  const int64_t gw = W / p, gh = H / p;
  const int64_t total = B * gh * gw * pd;
  for (int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x; o < total; o += (int64_t)gridDim.x * 256) {
    const int64_t row = o / pd, e = o % pd;
    const int64_t b = row / (gh * gw), g = row % (gh * gw);
    const int64_t gy = g / gw, gx = g % gw;
    const int64_t i = e / (p * C), j = (e / C) % p, c = e % C;
    out[o] = img[((b * H + gy * p + i) * W + gx * p + j) * C + c];
  }
}

__global__ __launch_bounds__(256) void embed_f32_kernel(const float* __restrict__ E, const float* __restrict__ cls,
                                                        const float* __restrict__ pos, float* __restrict__ X,
                                                        int64_t B, int64_t T, int64_t d) {
  const int64_t total = B * T * d;
  for (int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x; o < total; o += (int64_t)gridDim.x * 256) {
    const int64_t b = o / (T * d), t = (o / d) % T, c = o % d;
    const float base = t == 0 ? cls[c] : E[(b * (T - 1) + t - 1) * d + c];
    X[o] = base + pos[t * d + c];
  }
}

__global__ __launch_bounds__(256) void embed_bwd_f32_kernel(const float* __restrict__ dX, float* __restrict__ dE,
                                                            float* __restrict__ dcls, float* __restrict__ dpos,
                                                            int64_t B, int64_t T, int64_t d) {
  const int64_t total = T * d;
  for (int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x; o < total; o += (int64_t)gridDim.x * 256) {
    const int64_t t = o / d, c = o % d;
    float s = 0.0f;
    for (int64_t b = 0; b < B; ++b) {
      const float v = dX[b * T * d + o];
      s += v;
      if (t > 0) dE[(b * (T - 1) + t - 1) * d + c] = v;
    }
    dpos[o] = s;
    if (t == 0) dcls[c] = s;
  }
}

unsigned rows_grid(int64_t rows) { return (unsigned)((rows + 3) / 4); }
unsigned elem_grid(int64_t total) {
  return (unsigned)std::max<int64_t>(1, std::min<int64_t>((total + 255) / 256, 65536));
}

}  // namespace

hipError_t launch_layernorm_fwd_f32(const float* X, int64_t ldx, const float* gamma,
                                    const float* beta, float* Y, float* mean_rstd, int64_t rows,
                                    int64_t d, hipStream_t s) {
  layernorm_fwd_f32_kernel<<<rows_grid(rows), 256, 0, s>>>(X, ldx, gamma, beta, Y, mean_rstd, rows, d);
  return hipGetLastError();
}

int64_t ln_bwd_f32_blocks(int64_t rows) { return std::max<int64_t>(1, std::min<int64_t>((rows + 3) / 4, 512)); }

hipError_t launch_layernorm_bwd_f32(const float* X, int64_t ldx, const float* gamma,
                                    const float* dY, const float* Rgrad, float* dX, int64_t ldo,
                                    float* dgamma, float* dbeta, int64_t rows, int64_t d,
                                    float* part, hipStream_t s) {
  if (d > kLnF32MaxD) return hipErrorInvalidValue;
  const int64_t nb = ln_bwd_f32_blocks(rows);
  float* pt = dgamma ? part : nullptr;
  if (d <= 1024)
    layernorm_bwd_f32_kernel<16><<<(unsigned)nb, 256, 0, s>>>(X, ldx, gamma, dY, Rgrad, dX, ldo, rows, d, pt);
  else
    layernorm_bwd_f32_kernel<32><<<(unsigned)nb, 256, 0, s>>>(X, ldx, gamma, dY, Rgrad, dX, ldo, rows, d, pt);
  if (dgamma)
    ln_partials_final_f32_kernel<<<(unsigned)((2 * d + 255) / 256), 256, 0, s>>>(part, nb, d, dgamma, dbeta);
  return hipGetLastError();
}

hipError_t launch_softmax_f32(bool bwd, const float* A, const float* Bp, float* O, int64_t rows,
                              int64_t n, int64_t ld, float scale, hipStream_t s) {
  if (bwd) softmax_bwd_f32_kernel<<<rows_grid(rows), 256, 0, s>>>(A, Bp, O, rows, n, ld, scale);
  else softmax_fwd_f32_kernel<<<rows_grid(rows), 256, 0, s>>>(A, O, rows, n, ld, scale);
  return hipGetLastError();
}

hipError_t launch_cross_entropy_f32(const float* Z, int64_t ldz, const int32_t* labels, int64_t B,
                                    int64_t C, const mpx_scale_state* st, float* rowloss, float* dZ,
                                    hipStream_t s) {
  cross_entropy_f32_kernel<<<rows_grid(B), 256, 0, s>>>(Z, ldz, labels, B, C, st, rowloss, dZ);
  return hipGetLastError();
}

hipError_t launch_patchify_f32(const float* img, float* out, int64_t B, int64_t H, int64_t W,
                               int64_t C, int64_t p, hipStream_t s) {
  patchify_f32_kernel<<<elem_grid(B * H * W * C), 256, 0, s>>>(img, out, B, H, W, C, p);
  return hipGetLastError();
}

hipError_t launch_embed_assemble_f32(const float* E, const float* cls, const float* pos, float* X,
                                     int64_t B, int64_t T, int64_t d, hipStream_t s) {
  embed_f32_kernel<<<elem_grid(B * T * d), 256, 0, s>>>(E, cls, pos, X, B, T, d);
  return hipGetLastError();
}

hipError_t launch_embed_assemble_bwd_f32(const float* dX, float* dE, float* dcls, float* dpos,
                                         int64_t B, int64_t T, int64_t d, hipStream_t s) {
  embed_bwd_f32_kernel<<<elem_grid(T * d), 256, 0, s>>>(dX, dE, dcls, dpos, B, T, d);
  return hipGetLastError();
}

}  // namespace mpx
