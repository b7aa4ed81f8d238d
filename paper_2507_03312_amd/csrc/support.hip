// Support ops of the half-precision forward/backward passes: the
// full-precision islands MPX keeps in float32 (§3.2 force_full_precision:
// sums, means, softmax) — LayerNorm, softmax, the losses — plus the data
// movement of a ViT's token embedding.  Every op widens half inputs to
// float32, computes in float32 and rounds once to half at its output.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.h"

namespace mpx {

constexpr float kLnEps = 1e-5f;
constexpr int kMaxRowVec = 4;  // LayerNorm rows up to 4 * 64 * 8 = 2048 columns

// Row access helpers: lane `lane` owns columns lane*8 + v*512 + j.
template <int DT>
__device__ __forceinline__ void load_row(const uint16_t* __restrict__ row, int64_t d, int lane,
                                         float (&x)[kMaxRowVec][8]) {
#pragma unroll
  for (int v = 0; v < kMaxRowVec; ++v) {
    const int64_t c = (int64_t)lane * 8 + v * 512;
#pragma unroll
    for (int j = 0; j < 8; ++j) x[v][j] = 0.0f;
    if (c + 8 <= d && (reinterpret_cast<uintptr_t>(row + c) & 15u) == 0) {
      uint4 u = *reinterpret_cast<const uint4*>(row + c);
      const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[v][2 * j] = h2f<DT>((uint16_t)(w[j] & 0xFFFFu));
        x[v][2 * j + 1] = h2f<DT>((uint16_t)(w[j] >> 16));
      }
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (c + j < d) x[v][j] = h2f<DT>(row[c + j]);
    }
  }
}

template <int DT>
__device__ __forceinline__ void store_row(uint16_t* __restrict__ row, int64_t d, int lane,
                                          const uint16_t (&h)[kMaxRowVec][8]) {
#pragma unroll
  for (int v = 0; v < kMaxRowVec; ++v) {
    const int64_t c = (int64_t)lane * 8 + v * 512;
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
  return (int64_t)lane * 8 + v * 512 + j < d;
}

// ------------------------------------------------------------- LayerNorm --

template <int DT>
__global__ __launch_bounds__(256) void layernorm_fwd_kernel(const uint16_t* __restrict__ X, int64_t ldx,
                                                            const uint16_t* __restrict__ gamma,
                                                            const uint16_t* __restrict__ beta,
                                                            uint16_t* __restrict__ Y,
                                                            float* __restrict__ mr, int64_t rows,
                                                            int64_t d) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  float x[kMaxRowVec][8];
  load_row<DT>(X + r * ldx, d, lane, x);
  float s = 0.0f;
#pragma unroll
  for (int v = 0; v < kMaxRowVec; ++v)
#pragma unroll
    for (int j = 0; j < 8; ++j) s += x[v][j];
  const float mean = wave_sum(s) / (float)d;
  float q = 0.0f;
#pragma unroll
  for (int v = 0; v < kMaxRowVec; ++v)
#pragma unroll
    for (int j = 0; j < 8; ++j)
      if (col_ok(d, lane, v, j)) {
        const float c = x[v][j] - mean;
        q += c * c;
      }
  const float var = wave_sum(q) / (float)d;
  const float rstd = 1.0f / sqrtf(var + kLnEps);
  float g[kMaxRowVec][8], b[kMaxRowVec][8];
  load_row<DT>(gamma, d, lane, g);
  load_row<DT>(beta, d, lane, b);
  uint16_t h[kMaxRowVec][8];
#pragma unroll
  for (int v = 0; v < kMaxRowVec; ++v)
#pragma unroll
    for (int j = 0; j < 8; ++j) h[v][j] = f2h<DT>((x[v][j] - mean) * rstd * g[v][j] + b[v][j]);
  store_row<DT>(Y + r * d, d, lane, h);
  if (mr && lane == 0) {
    mr[2 * r] = mean;
    mr[2 * r + 1] = rstd;
  }
}

// dX for each row; per-workgroup column partials of dgamma (sum dy*xhat) and
// dbeta (sum dy) into part[blockIdx][2][d].
template <int DT>
__global__ __launch_bounds__(256) void layernorm_bwd_kernel(
    const uint16_t* __restrict__ X, int64_t ldx, const uint16_t* __restrict__ gamma,
    const uint16_t* __restrict__ dY, const uint16_t* __restrict__ Rg, uint16_t* __restrict__ dX,
    int64_t ldo, int64_t rows, int64_t d, float* __restrict__ part) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  float g[kMaxRowVec][8];
  load_row<DT>(gamma, d, lane, g);
  float pg[kMaxRowVec][8], pb[kMaxRowVec][8];
#pragma unroll
  for (int v = 0; v < kMaxRowVec; ++v)
#pragma unroll
    for (int j = 0; j < 8; ++j) pg[v][j] = pb[v][j] = 0.0f;

  for (int64_t r = (int64_t)blockIdx.x * 4 + wave; r < rows; r += (int64_t)gridDim.x * 4) {
    float x[kMaxRowVec][8], dy[kMaxRowVec][8];
    load_row<DT>(X + r * ldx, d, lane, x);
    load_row<DT>(dY + r * d, d, lane, dy);
    float s = 0.0f;
#pragma unroll
    for (int v = 0; v < kMaxRowVec; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) s += x[v][j];
    const float mean = wave_sum(s) / (float)d;
    float q = 0.0f;
#pragma unroll
    for (int v = 0; v < kMaxRowVec; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (col_ok(d, lane, v, j)) {
          const float c = x[v][j] - mean;
          q += c * c;
        }
    const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + kLnEps);
    float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
    for (int v = 0; v < kMaxRowVec; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float xh = col_ok(d, lane, v, j) ? (x[v][j] - mean) * rstd : 0.0f;
        x[v][j] = xh;
        const float dxh = dy[v][j] * g[v][j];
        s1 += dxh;
        s2 += dxh * xh;
        pg[v][j] += dy[v][j] * xh;
        pb[v][j] += dy[v][j];
      }
    s1 = wave_sum(s1) / (float)d;
    s2 = wave_sum(s2) / (float)d;
    float rg[kMaxRowVec][8];
    if (Rg) load_row<DT>(Rg + r * ldo, d, lane, rg);
    uint16_t h[kMaxRowVec][8];
#pragma unroll
    for (int v = 0; v < kMaxRowVec; ++v)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float dx = rstd * (dy[v][j] * g[v][j] - s1 - x[v][j] * s2);
        uint16_t o = f2h<DT>(dx);
        if (Rg) o = f2h<DT>(rg[v][j] + h2f<DT>(o));
        h[v][j] = o;
      }
    store_row<DT>(dX + r * ldo, d, lane, h);
  }
  // reduce the 4 waves' column partials through LDS, then write this block's
  __shared__ float red[4][2][512];
  float* out = part + (int64_t)blockIdx.x * 2 * d;
#pragma unroll
  for (int v = 0; v < kMaxRowVec; ++v) {
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      red[wave][0][lane * 8 + j] = pg[v][j];
      red[wave][1][lane * 8 + j] = pb[v][j];
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 1024; i += 256) {
      const int which = i >> 9, c = i & 511;
      const int64_t col = (int64_t)(c >> 3) * 8 + v * 512 + (c & 7);
      if (col < d)
        out[which * d + col] =
            ((red[0][which][c] + red[1][which][c]) + red[2][which][c]) + red[3][which][c];
    }
  }
}

template <int DT>
__global__ __launch_bounds__(256) void layernorm_bwd_final_kernel(const float* __restrict__ part,
                                                                  int nparts, int64_t d,
                                                                  uint16_t* __restrict__ dg,
                                                                  uint16_t* __restrict__ db) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= 2 * d) return;
  const int which = (int)(i / d);
  const int64_t col = i % d;
  float s = 0.0f;
  for (int p = 0; p < nparts; ++p) s += part[(int64_t)p * 2 * d + which * d + col];
  (which ? db : dg)[col] = f2h<DT>(s);
}

static int ln_bwd_blocks(int64_t rows) { return (int)std::min<int64_t>((rows + 3) / 4, 512); }

// --------------------------------------------------------------- softmax --

template <int DT>
__global__ __launch_bounds__(256) void softmax_fwd_kernel(const uint16_t* __restrict__ S,
                                                          uint16_t* __restrict__ P, int64_t rows,
                                                          int64_t n, int64_t ld, float scale) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const uint16_t* s = S + r * ld;
  uint16_t* p = P + r * ld;
  float mx = -INFINITY;
  for (int64_t c = lane; c < n; c += 64) mx = fmaxf(mx, scale * h2f<DT>(s[c]));
  mx = wave_max(mx);
  float sum = 0.0f;
  for (int64_t c = lane; c < n; c += 64) sum += expf(scale * h2f<DT>(s[c]) - mx);
  sum = wave_sum(sum);
  const float inv = 1.0f / sum;
  for (int64_t c = lane; c < ld; c += 64)
    p[c] = c < n ? f2h<DT>(expf(scale * h2f<DT>(s[c]) - mx) * inv) : (uint16_t)0;
}

template <int DT>
__global__ __launch_bounds__(256) void softmax_bwd_kernel(const uint16_t* __restrict__ P,
                                                          const uint16_t* __restrict__ dP,
                                                          uint16_t* __restrict__ dS, int64_t rows,
                                                          int64_t n, int64_t ld, float scale) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= rows) return;
  const uint16_t* p = P + r * ld;
  const uint16_t* dp = dP + r * ld;
  uint16_t* ds = dS + r * ld;
  float dot = 0.0f;
  for (int64_t c = lane; c < n; c += 64) dot += h2f<DT>(dp[c]) * h2f<DT>(p[c]);
  dot = wave_sum(dot);
  for (int64_t c = lane; c < ld; c += 64)
    ds[c] = c < n ? f2h<DT>(scale * h2f<DT>(p[c]) * (h2f<DT>(dp[c]) - dot)) : (uint16_t)0;
}

// ----------------------------------------------------------------- losses --

// One workgroup; wave w handles rows w, w+4, ...; losses summed in row order
// per wave, then across waves in wave order.
template <int DT>
__global__ __launch_bounds__(256) void cross_entropy_kernel(const uint16_t* __restrict__ Z, int64_t ldz,
                                                            const int32_t* __restrict__ labels,
                                                            int64_t B, int64_t C,
                                                            const mpx_scale_state* __restrict__ st,
                                                            float* __restrict__ loss,
                                                            uint16_t* __restrict__ dZ) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float scale = st->scale;
  float acc = 0.0f;
  for (int64_t b = wave; b < B; b += 4) {
    const uint16_t* z = Z + b * ldz;
    const int32_t y = labels[b];
    float mx = -INFINITY;
    for (int64_t c = lane; c < C; c += 64) mx = fmaxf(mx, h2f<DT>(z[c]));
    mx = wave_max(mx);
    float se = 0.0f;
    for (int64_t c = lane; c < C; c += 64) se += expf(h2f<DT>(z[c]) - mx);
    se = wave_sum(se);
    const float lse = logf(se);
    const bool ok = y >= 0 && y < C;  // an out-of-range label gives a NaN loss, never a read
    acc += ok ? lse - (h2f<DT>(z[y]) - mx) : NAN;
    const float k = scale / (float)B;
    for (int64_t c = lane; c < C; c += 64) {
      const float pr = expf(h2f<DT>(z[c]) - mx) / se;
      dZ[b * C + c] = f2h<DT>(k * (pr - (c == y ? 1.0f : 0.0f)));
    }
  }
  __shared__ float part[4];
  if (lane == 0) part[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) *loss = (((part[0] + part[1]) + part[2]) + part[3]) / (float)B;
}

template <int DT>
__global__ __launch_bounds__(256) void mse_kernel(const uint16_t* __restrict__ Y, const uint16_t* __restrict__ T,
                                                  int64_t n, const mpx_scale_state* __restrict__ st,
                                                  float* __restrict__ loss, uint16_t* __restrict__ dY) {
  const float k = 2.0f * st->scale / (float)n;
  float acc = 0.0f;
  for (int64_t i = threadIdx.x; i < n; i += 256) {
    const float df = h2f<DT>(Y[i]) - h2f<DT>(T[i]);
    acc += df * df;
    dY[i] = f2h<DT>(k * df);
  }
  __shared__ float part[4];
  acc = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) *loss = (((part[0] + part[1]) + part[2]) + part[3]) / (float)n;
}

// ------------------------------------------------------------ embeddings --

template <int DT>
__global__ __launch_bounds__(256) void patchify_cast_kernel(const float* __restrict__ img,
                                                            uint16_t* __restrict__ out, int64_t B,
                                                            int64_t H, int64_t W, int64_t C, int64_t p) {
  const int64_t pd = p * p * C;
  const int64_t gw = W / p, gh = H / p;
  const int64_t total = B * gh * gw * pd;
  for (int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x; o < total; o += (int64_t)gridDim.x * 256) {
    const int64_t row = o / pd, e = o % pd;
    const int64_t b = row / (gh * gw), g = row % (gh * gw);
    const int64_t gy = g / gw, gx = g % gw;
    const int64_t i = e / (p * C), j = (e / C) % p, c = e % C;
    out[o] = f2h<DT>(img[((b * H + gy * p + i) * W + gx * p + j) * C + c]);
  }
}

template <int DT>
__global__ __launch_bounds__(256) void embed_assemble_kernel(const uint16_t* __restrict__ E,
                                                             const uint16_t* __restrict__ cls,
                                                             const uint16_t* __restrict__ pos,
                                                             uint16_t* __restrict__ X, int64_t B,
                                                             int64_t T, int64_t d) {
  const int64_t total = B * T * d;
  for (int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x; o < total; o += (int64_t)gridDim.x * 256) {
    const int64_t b = o / (T * d), t = (o / d) % T, c = o % d;
    const float base = t == 0 ? h2f<DT>(cls[c]) : h2f<DT>(E[(b * (T - 1) + t - 1) * d + c]);
    X[o] = f2h<DT>(base + h2f<DT>(pos[t * d + c]));
  }
}

template <int DT>
__global__ __launch_bounds__(256) void embed_assemble_bwd_kernel(const uint16_t* __restrict__ dX,
                                                                 uint16_t* __restrict__ dE,
                                                                 uint16_t* __restrict__ dcls,
                                                                 uint16_t* __restrict__ dpos,
                                                                 int64_t B, int64_t T, int64_t d) {
  const int64_t total = T * d;
  for (int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x; o < total; o += (int64_t)gridDim.x * 256) {
    const int64_t t = o / d, c = o % d;
    float s = 0.0f;
    for (int64_t b = 0; b < B; ++b) {
      const uint16_t v = dX[b * T * d + o];
      s += h2f<DT>(v);
      if (t > 0) dE[(b * (T - 1) + t - 1) * d + c] = v;
    }
    const uint16_t h = f2h<DT>(s);
    dpos[o] = h;
    if (t == 0) dcls[c] = h;
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

extern "C" int mpx_layernorm_fwd(const void* X, int64_t ldx, const void* gamma, const void* beta,
                                 void* Y, float* mean_rstd, int64_t rows, int64_t d, mpx_dtype dt,
                                 void* stream) {
  clear_error();
  MPX_REQUIRE(X && gamma && beta && Y, "NULL argument");
  MPX_REQUIRE(rows >= 1 && d >= 1 && d <= 2048 && ldx >= d, "bad sizes (1 <= d <= 2048, ldx >= d)");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_DT_DISPATCH(dt, layernorm_fwd_kernel, (unsigned)((rows + 3) / 4), 256, stream,
                  (const uint16_t*)X, ldx, (const uint16_t*)gamma, (const uint16_t*)beta,
                  (uint16_t*)Y, mean_rstd, rows, d);
  return MPX_OK;
}

extern "C" size_t mpx_layernorm_bwd_workspace(int64_t rows, int64_t d) {
  if (rows < 1 || d < 1) return 0;
  return (size_t)ln_bwd_blocks(rows) * 2 * d * sizeof(float);
}

extern "C" int mpx_layernorm_bwd(const void* X, int64_t ldx, const void* gamma, const void* dY,
                                 const void* Rgrad, void* dX, int64_t ldo, void* dgamma, void* dbeta,
                                 int64_t rows, int64_t d, mpx_dtype dt, void* workspace,
                                 size_t ws_bytes, void* stream) {
  clear_error();
  MPX_REQUIRE(X && gamma && dY && dX && dgamma && dbeta, "NULL argument");
  MPX_REQUIRE(rows >= 1 && d >= 1 && d <= 2048 && ldx >= d && ldo >= d, "bad sizes");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  const size_t need = mpx_layernorm_bwd_workspace(rows, d);
  if (!workspace || ws_bytes < need) {
    set_error("mpx_layernorm_bwd: workspace of " + std::to_string(need) + " bytes required");
    return MPX_ERR_WORKSPACE;
  }
  const int nb = ln_bwd_blocks(rows);
  MPX_DT_DISPATCH(dt, layernorm_bwd_kernel, (unsigned)nb, 256, stream, (const uint16_t*)X, ldx,
                  (const uint16_t*)gamma, (const uint16_t*)dY, (const uint16_t*)Rgrad,
                  (uint16_t*)dX, ldo, rows, d, (float*)workspace);
  MPX_DT_DISPATCH(dt, layernorm_bwd_final_kernel, (unsigned)((2 * d + 255) / 256), 256, stream,
                  (const float*)workspace, nb, d, (uint16_t*)dgamma, (uint16_t*)dbeta);
  return MPX_OK;
}

extern "C" int mpx_softmax_fwd(const void* S, void* P, int64_t rows, int64_t n, int64_t ld, float scale,
                               mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(S && P, "NULL argument");
  MPX_REQUIRE(rows >= 1 && n >= 1 && ld >= n, "bad sizes");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_DT_DISPATCH(dt, softmax_fwd_kernel, (unsigned)((rows + 3) / 4), 256, stream,
                  (const uint16_t*)S, (uint16_t*)P, rows, n, ld, scale);
  return MPX_OK;
}

extern "C" int mpx_softmax_bwd(const void* P, const void* dP, void* dS, int64_t rows, int64_t n,
                               int64_t ld, float scale, mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(P && dP && dS, "NULL argument");
  MPX_REQUIRE(rows >= 1 && n >= 1 && ld >= n, "bad sizes");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_DT_DISPATCH(dt, softmax_bwd_kernel, (unsigned)((rows + 3) / 4), 256, stream,
                  (const uint16_t*)P, (const uint16_t*)dP, (uint16_t*)dS, rows, n, ld, scale);
  return MPX_OK;
}

extern "C" int mpx_cross_entropy(const void* Z, int64_t ldz, const int32_t* labels, int64_t B,
                                 int64_t C, const mpx_scale_state* d_state, float* d_loss, void* dZ,
                                 mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(Z && labels && d_state && d_loss && dZ, "NULL argument");
  MPX_REQUIRE(B >= 1 && C >= 1 && ldz >= C, "bad sizes");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_DT_DISPATCH(dt, cross_entropy_kernel, 1, 256, stream, (const uint16_t*)Z, ldz, labels, B, C,
                  d_state, d_loss, (uint16_t*)dZ);
  return MPX_OK;
}

extern "C" int mpx_mse(const void* Y, const void* T, int64_t n, const mpx_scale_state* d_state,
                       float* d_loss, void* dY, mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(Y && T && d_state && d_loss && dY, "NULL argument");
  MPX_REQUIRE(n >= 1, "n must be >= 1");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_DT_DISPATCH(dt, mse_kernel, 1, 256, stream, (const uint16_t*)Y, (const uint16_t*)T, n, d_state,
                  d_loss, (uint16_t*)dY);
  return MPX_OK;
}

extern "C" int mpx_patchify_cast(const float* images, void* patches, int64_t B, int64_t H, int64_t W,
                                 int64_t C, int64_t p, mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(images && patches, "NULL argument");
  MPX_REQUIRE(B >= 1 && C >= 1 && p >= 1 && H >= p && W >= p && H % p == 0 && W % p == 0,
              "bad sizes (H and W must be multiples of p)");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_DT_DISPATCH(dt, patchify_cast_kernel, grid_for(B * H * W * C), 256, stream, images,
                  (uint16_t*)patches, B, H, W, C, p);
  return MPX_OK;
}

extern "C" int mpx_embed_assemble(const void* E, const void* cls, const void* pos, void* X, int64_t B,
                                  int64_t T, int64_t d, mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(E && cls && pos && X, "NULL argument");
  MPX_REQUIRE(B >= 1 && T >= 2 && d >= 1, "bad sizes");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_DT_DISPATCH(dt, embed_assemble_kernel, grid_for(B * T * d), 256, stream, (const uint16_t*)E,
                  (const uint16_t*)cls, (const uint16_t*)pos, (uint16_t*)X, B, T, d);
  return MPX_OK;
}

extern "C" int mpx_embed_assemble_bwd(const void* dX, void* dE, void* dcls, void* dpos, int64_t B,
                                      int64_t T, int64_t d, mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(dX && dE && dcls && dpos, "NULL argument");
  MPX_REQUIRE(B >= 1 && T >= 2 && d >= 1, "bad sizes");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_DT_DISPATCH(dt, embed_assemble_bwd_kernel, grid_for(T * d), 256, stream, (const uint16_t*)dX,
                  (uint16_t*)dE, (uint16_t*)dcls, (uint16_t*)dpos, B, T, d);
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
