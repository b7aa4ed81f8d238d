// Half-precision GEMMs with float32 accumulation on gfx950 MFMA, for the
// forward and backward passes of MPX's mixed-precision step (§2: forward and
// backward in half precision; the products accumulate in float32).
//
// One kernel template computes  C[m,n] = sum_k A(m,k) B(n,k)  where each
// operand is stored either with the reduction index contiguous ("k-major") or
// with the output index contiguous ("mn-major"):
//   forward  Y  = X W^T   : A = X  k-major,  B = W  k-major
//   backward dX = dY W    : A = dY k-major,  B = W  mn-major
//   backward dW = dY^T X  : A = dY mn-major, B = X  mn-major
// Tiles are staged through LDS in one layout, [row][k] with k contiguous, so
// the MFMA operand reads are always 16-byte ds_read_b128.  An mn-major operand
// is transposed on the way in: each lane loads 4 rows of 8 contiguous values
// and writes them as 8 rows of 4 k-values (a register transpose of 16-bit
// pairs).  The MFMA is v_mfma_f32_32x32x16_{f16,bf16}: lane l holds 8 k-values
// of row l%32 for A and of column l%32 for B; the 16 accumulators of lane l are
// column l%32, rows 8*(i/4) + 4*(l/32) + i%4.
//
// Epilogue (all optional, in this order, each rounding once to half):
//   h = half(acc + bias[n]);  pre_out = h;  h = half(gelu(h));
//   h = half(h * gelu'(dact[m,n]));  h = half(h + resid[m,n]);  C = h
// or, for split-K, the float32 partial sums go to a workspace and a second
// kernel adds the partials in a fixed order and rounds once.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "common.h"

namespace mpx {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

struct GemmArgs {
  const uint16_t* A;
  const uint16_t* B;
  uint16_t* C;
  float* ws;  // split-K partials [splits][M][N] (when splits > 1)
  int64_t M, N, K, lda, ldb, ldc;
  int64_t sA0, sA1, sB0, sB1, sC0, sC1, nb1;
  int32_t splits;
  int64_t k_split;  // reduction length per split (multiple of the k tile)
  const uint16_t* bias;
  const uint16_t* resid;
  int64_t ldr;
  uint16_t* pre;
  const uint16_t* dact;
  int32_t act;
};

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

// Loader of one operand tile (ROWS output rows x BK reduction values) into
// registers, then into LDS as [row][k].  KMAJ: element (r,k) at base[r*ld + k];
// otherwise at base[k*ld + r].
template <int ROWS, int BK, int NT, bool KMAJ, bool VEC>
struct TileLoader {
  // k rows per lane for an mn-major operand: 4 when the tile is large enough,
  // else 2, so that every lane owns whole units
  static constexpr int KR = (ROWS * BK / 8) / NT >= 4 ? 4 : 2;
  static constexpr int UNITS = KMAJ ? ROWS * BK / 8 : ROWS * BK / (8 * KR);
  static constexpr int PER = UNITS / NT;                         // units per lane
  static_assert(UNITS % NT == 0, "tile does not split evenly over the workgroup");
  uint4 reg[KMAJ ? PER : PER * KR];

  // rows_valid: rows r < rows_valid exist; k_valid: reduction values k < k_valid exist
  __device__ __forceinline__ void load(const uint16_t* __restrict__ base, int64_t ld, int rows_valid,
                                       int k_valid, int tid) {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int unit = tid + u * NT;
      if constexpr (KMAJ) {
        const int r = unit / (BK / 8);
        const int k = (unit % (BK / 8)) * 8;
        const uint16_t* p = base + (int64_t)r * ld + k;
        if (VEC && r < rows_valid && k + 8 <= k_valid) {
          reg[u] = *reinterpret_cast<const uint4*>(p);
        } else {
          uint16_t h[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) h[j] = (r < rows_valid && k + j < k_valid) ? p[j] : (uint16_t)0;
          reg[u] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16),
                              h[6] | (h[7] << 16));
        }
      } else {
        const int r = (unit % (ROWS / 8)) * 8;
        const int k = (unit / (ROWS / 8)) * KR;
#pragma unroll
        for (int q = 0; q < KR; ++q) {
          const uint16_t* p = base + (int64_t)(k + q) * ld + r;
          if (VEC && k + q < k_valid && r + 8 <= rows_valid) {
            reg[u * KR + q] = *reinterpret_cast<const uint4*>(p);
          } else {
            uint16_t h[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) h[j] = (k + q < k_valid && r + j < rows_valid) ? p[j] : (uint16_t)0;
            reg[u * KR + q] = make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16),
                                         h[4] | (h[5] << 16), h[6] | (h[7] << 16));
          }
        }
      }
    }
  }

  // LDS tile: ROWS rows of pitch LDSP halves.
  template <int LDSP>
  __device__ __forceinline__ void store(uint16_t* __restrict__ lds, int tid) const {
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int unit = tid + u * NT;
      if constexpr (KMAJ) {
        const int r = unit / (BK / 8);
        const int k = (unit % (BK / 8)) * 8;
        *reinterpret_cast<uint4*>(lds + r * LDSP + k) = reg[u];
      } else {
        const int r = (unit % (ROWS / 8)) * 8;
        const int k = (unit / (ROWS / 8)) * KR;
        // register transpose: lane holds rows k..k+KR-1 of 8 consecutive
        // output indices; write output index r+j as KR consecutive k values
        uint32_t w[KR][4];
#pragma unroll
        for (int q = 0; q < KR; ++q) {
          w[q][0] = reg[u * KR + q].x;
          w[q][1] = reg[u * KR + q].y;
          w[q][2] = reg[u * KR + q].z;
          w[q][3] = reg[u * KR + q].w;
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int i = j >> 1;
          uint32_t d[KR / 2];
#pragma unroll
          for (int q = 0; q < KR / 2; ++q) {
            const uint32_t a = w[2 * q][i], b = w[2 * q + 1][i];
            d[q] = (j & 1) ? ((a >> 16) | (b & 0xFFFF0000u)) : ((a & 0xFFFFu) | (b << 16));
          }
          if constexpr (KR == 4)
            *reinterpret_cast<uint2*>(lds + (r + j) * LDSP + k) = make_uint2(d[0], d[1]);
          else
            *reinterpret_cast<uint32_t*>(lds + (r + j) * LDSP + k) = d[0];
        }
      }
    }
  }
};

template <int DT, int BM, int BN, int BK, int WM, int WN, bool AK, bool BKM, bool VEC>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64) void gemm_kernel(GemmArgs g) {
  constexpr int NW = (BM / WM) * (BN / WN);
  constexpr int NT = NW * 64;
  constexpr int PAD = 8;
  constexpr int LDSP = BK + PAD;
  constexpr int TM = WM / 32, TN = WN / 32;
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * LDSP];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * LDSP];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm0 = (wave / (BN / WN)) * WM;
  const int wn0 = (wave % (BN / WN)) * WN;

  // tile coordinates
  const int64_t tiles_n = (g.N + BN - 1) / BN;
  const int64_t tile = blockIdx.x;
  const int64_t m0 = (tile / tiles_n) * BM;
  const int64_t n0 = (tile % tiles_n) * BN;
  // batch / split
  int64_t z = blockIdx.y;
  int split = 0;
  int64_t offA = 0, offB = 0, offC = 0;
  if (g.splits > 1) {
    split = (int)z;
  } else {
    const int64_t i0 = z / g.nb1, i1 = z % g.nb1;
    offA = i0 * g.sA0 + i1 * g.sA1;
    offB = i0 * g.sB0 + i1 * g.sB1;
    offC = i0 * g.sC0 + i1 * g.sC1;
  }
  const int64_t kbeg = (int64_t)split * g.k_split;
  const int64_t kend = min(g.K, kbeg + g.k_split);
  const int nk = (int)((kend - kbeg + BK - 1) / BK);

  const uint16_t* A = g.A + offA;
  const uint16_t* B = g.B + offB;
  // operand tile base pointers at k = kbeg
  const uint16_t* Ab = AK ? A + m0 * g.lda + kbeg : A + kbeg * g.lda + m0;
  const uint16_t* Bb = BKM ? B + n0 * g.ldb + kbeg : B + kbeg * g.ldb + n0;
  const int64_t Astep = AK ? BK : BK * g.lda;
  const int64_t Bstep = BKM ? BK : BK * g.ldb;
  const int rowsA = (int)min<int64_t>(BM, g.M - m0);
  const int rowsB = (int)min<int64_t>(BN, g.N - n0);

  TileLoader<BM, BK, NT, AK, VEC> la;
  TileLoader<BN, BK, NT, BKM, VEC> lb;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  if (nk > 0) {
    la.load(Ab, g.lda, rowsA, (int)min<int64_t>(BK, kend - kbeg), tid);
    lb.load(Bb, g.ldb, rowsB, (int)min<int64_t>(BK, kend - kbeg), tid);
    la.template store<LDSP>(sA[0], tid);
    lb.template store<LDSP>(sB[0], tid);
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      const int64_t kv = kend - (kbeg + (int64_t)(kt + 1) * BK);
      const int kval = (int)min<int64_t>(BK, kv);
      la.load(Ab + (kt + 1) * Astep, g.lda, rowsA, kval, tid);
      lb.load(Bb + (kt + 1) * Bstep, g.ldb, rowsB, kval, tid);
    }
    const uint16_t* a_s = sA[cur];
    const uint16_t* b_s = sB[cur];
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int kofs = kk * 16 + 8 * (lane >> 5);
      uint4 af[TM], bf[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const uint4*>(a_s + (wm0 + i * 32 + (lane & 31)) * LDSP + kofs);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bf[j] = *reinterpret_cast<const uint4*>(b_s + (wn0 + j * 32 + (lane & 31)) * LDSP + kofs);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32<DT>(af[i], bf[j], acc[i][j]);
    }
    if (more) {
      la.template store<LDSP>(sA[cur ^ 1], tid);
      lb.template store<LDSP>(sB[cur ^ 1], tid);
    }
    __syncthreads();
  }

  // ---- epilogue ----
  const int col_l = lane & 31;
  const int row_l = 4 * (lane >> 5);
  if (g.splits > 1) {
    float* W = g.ws + (int64_t)split * g.M * g.N;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int64_t n = n0 + wn0 + j * 32 + col_l;
        if (n >= g.N) continue;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int64_t m = m0 + wm0 + i * 32 + 8 * (e >> 2) + row_l + (e & 3);
          if (m < g.M) W[m * g.N + n] = acc[i][j][e];
        }
      }
    return;
  }
  uint16_t* C = g.C + offC;
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int64_t n = n0 + wn0 + j * 32 + col_l;
      if (n >= g.N) continue;
      const float bias = g.bias ? h2f<DT>(g.bias[n]) : 0.0f;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t m = m0 + wm0 + i * 32 + 8 * (e >> 2) + row_l + (e & 3);
        if (m >= g.M) continue;
        uint16_t h = f2h<DT>(acc[i][j][e] + bias);
        if (g.pre) g.pre[m * g.ldc + n] = h;
        if (g.act == MPX_ACT_GELU_TANH) h = f2h<DT>(gelu_tanh(h2f<DT>(h)));
        if (g.dact) h = f2h<DT>(h2f<DT>(h) * gelu_tanh_grad(h2f<DT>(g.dact[m * g.ldc + n])));
        if (g.resid) h = f2h<DT>(h2f<DT>(h) + h2f<DT>(g.resid[m * g.ldr + n]));
        C[m * g.ldc + n] = h;
      }
    }
}

// Sum of split-K partials in split order, one rounding: C = half(sum_s W[s]).
template <int DT>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ ws, int splits,
                                                            int64_t MN, uint16_t* __restrict__ C) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= MN) return;
  float s = ws[i];
  for (int k = 1; k < splits; ++k) s += ws[(int64_t)k * MN + i];
  C[i] = f2h<DT>(s);
}

// Column sums of a half matrix [rows, cols] (dense), float32 accumulation.
// Phase 1: workgroup (x: 64-column block, y: row slice) -> partial[y][col].
template <int DT>
__global__ __launch_bounds__(256) void colsum_partial_kernel(const uint16_t* __restrict__ X, int64_t rows,
                                                             int64_t cols, int64_t rows_per,
                                                             float* __restrict__ part) {
  __shared__ float red[4][64];
  const int c = threadIdx.x & 63, rl = threadIdx.x >> 6;
  const int64_t col = (int64_t)blockIdx.x * 64 + c;
  const int64_t r0 = (int64_t)blockIdx.y * rows_per;
  const int64_t r1 = min(rows, r0 + rows_per);
  float s = 0.0f;
  if (col < cols)
    for (int64_t r = r0 + rl; r < r1; r += 4) s += h2f<DT>(X[r * cols + col]);
  red[rl][c] = s;
  __syncthreads();
  if (rl == 0 && col < cols)
    part[(int64_t)blockIdx.y * cols + col] = ((red[0][c] + red[1][c]) + red[2][c]) + red[3][c];
}
// Phase 2: out[col] = half(sum_y partial[y][col]) in slice order.
template <int DT>
__global__ __launch_bounds__(256) void colsum_final_kernel(const float* __restrict__ part, int nparts,
                                                           int64_t cols, uint16_t* __restrict__ out) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (col >= cols) return;
  float s = 0.0f;
  for (int y = 0; y < nparts; ++y) s += part[(int64_t)y * cols + col];
  out[col] = f2h<DT>(s);
}

// ------------------------------------------------------------ dispatch --

struct Cfg {
  int bm, bn;
};

static bool aligned_vec(const void* p, int64_t ld, int64_t s0, int64_t s1) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0 && ld % 8 == 0 && s0 % 8 == 0 && s1 % 8 == 0;
}

template <int DT, int BM, int BN, int WM, int WN>
static hipError_t launch_cfg(const GemmArgs& g, bool ak, bool bk, bool vec, int64_t nbatch,
                             hipStream_t s) {
  constexpr int BK = 64;
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  dim3 grid((unsigned)tiles, (unsigned)(g.splits > 1 ? g.splits : nbatch));
#define MPX_G(AKv, BKv, VECv) \
  gemm_kernel<DT, BM, BN, BK, WM, WN, AKv, BKv, VECv><<<grid, NT, 0, s>>>(g)
  if (vec) {
    if (ak && bk) MPX_G(true, true, true);
    else if (ak && !bk) MPX_G(true, false, true);
    else if (!ak && bk) MPX_G(false, true, true);
    else MPX_G(false, false, true);
  } else {
    if (ak && bk) MPX_G(true, true, false);
    else if (ak && !bk) MPX_G(true, false, false);
    else if (!ak && bk) MPX_G(false, true, false);
    else MPX_G(false, false, false);
  }
#undef MPX_G
  return hipGetLastError();
}

// ak: A is k-major; bk: B is k-major.
template <int DT>
static hipError_t run_gemm(GemmArgs g, bool ak, bool bk, int64_t nbatch, hipStream_t s) {
  const bool vec = aligned_vec(g.A, g.lda, g.sA0, g.sA1) && aligned_vec(g.B, g.ldb, g.sB0, g.sB1);
  if (g.M <= 64 || g.N <= 64) return launch_cfg<DT, 64, 64, 32, 32>(g, ak, bk, vec, nbatch, s);
  return launch_cfg<DT, 128, 128, 64, 64>(g, ak, bk, vec, nbatch, s);
}

static hipError_t gemm_dispatch(mpx_dtype dt, const GemmArgs& g, bool ak, bool bk, int64_t nbatch,
                                hipStream_t s) {
  return dt == MPX_F16 ? run_gemm<MPX_F16>(g, ak, bk, nbatch, s) : run_gemm<MPX_BF16>(g, ak, bk, nbatch, s);
}

static GemmArgs base_args() {
  GemmArgs g{};
  g.nb1 = 1;
  g.splits = 1;
  g.k_split = INT64_MAX / 4;
  return g;
}

// split-K plan for a reduction of length K over an MxN output
static int choose_splits(int64_t M, int64_t N, int64_t K) {
  const int64_t tiles = ((M + 127) / 128) * ((N + 127) / 128);
  int64_t s = (512 + tiles - 1) / tiles;
  s = std::min<int64_t>(s, 8);
  s = std::min<int64_t>(s, std::max<int64_t>(1, K / 512));
  return (int)std::max<int64_t>(s, 1);
}

static int64_t colsum_slices(int64_t rows) { return std::max<int64_t>(1, std::min<int64_t>(64, rows / 256)); }

static size_t colsum_ws(int64_t rows, int64_t cols) { return (size_t)colsum_slices(rows) * cols * sizeof(float); }

template <int DT>
static hipError_t colsum_run(const uint16_t* X, int64_t rows, int64_t cols, float* ws, uint16_t* out,
                             hipStream_t s) {
  const int64_t sl = colsum_slices(rows);
  const int64_t per = (rows + sl - 1) / sl;
  dim3 g1((unsigned)((cols + 63) / 64), (unsigned)sl);
  colsum_partial_kernel<DT><<<g1, 256, 0, s>>>(X, rows, cols, per, ws);
  colsum_final_kernel<DT><<<(unsigned)((cols + 255) / 256), 256, 0, s>>>(ws, (int)sl, cols, out);
  return hipGetLastError();
}

}  // namespace mpx

using namespace mpx;

extern "C" int mpx_linear_fwd(const void* X, const void* W, const void* b, const void* R, void* Y,
                              void* Ypre, int64_t M, int64_t N, int64_t K, mpx_dtype dt, int32_t act,
                              void* stream) {
  clear_error();
  MPX_REQUIRE(X && W && Y, "NULL operand");
  MPX_REQUIRE(M >= 1 && N >= 1 && K >= 1, "M, N, K must be >= 1");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_REQUIRE(act == MPX_ACT_NONE || act == MPX_ACT_GELU_TANH, "unknown activation");
  MPX_REQUIRE(act == MPX_ACT_NONE || Ypre, "Ypre is required with an activation");
  GemmArgs g = base_args();
  g.A = (const uint16_t*)X;
  g.B = (const uint16_t*)W;
  g.C = (uint16_t*)Y;
  g.M = M; g.N = N; g.K = K;
  g.lda = K; g.ldb = K; g.ldc = N;
  g.bias = (const uint16_t*)b;
  g.resid = (const uint16_t*)R;
  g.ldr = N;
  g.pre = act ? (uint16_t*)Ypre : nullptr;
  g.act = act;
  MPX_HIP(gemm_dispatch(dt, g, true, true, 1, (hipStream_t)stream));
  return MPX_OK;
}

extern "C" size_t mpx_linear_bwd_workspace(int64_t M, int64_t N, int64_t K) {
  if (M < 1 || N < 1 || K < 1) return 0;
  const int s = choose_splits(N, K, M);
  size_t ws = s > 1 ? (size_t)s * N * K * sizeof(float) : 0;
  return std::max(ws, colsum_ws(M, N)) + 256;
}

extern "C" int mpx_linear_bwd(const void* X, const void* W, const void* dY, const void* Xpre,
                              int32_t x_act, void* dX, void* dW, void* db, int64_t M, int64_t N,
                              int64_t K, mpx_dtype dt, void* workspace, size_t ws_bytes, void* stream) {
  clear_error();
  MPX_REQUIRE(X && dY && dW, "NULL operand");
  MPX_REQUIRE(!dX || W, "W is required for dX");
  MPX_REQUIRE(M >= 1 && N >= 1 && K >= 1, "M, N, K must be >= 1");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_REQUIRE(x_act == MPX_ACT_NONE || x_act == MPX_ACT_GELU_TANH, "unknown activation");
  MPX_REQUIRE(x_act == MPX_ACT_NONE || !dX || Xpre, "Xpre is required with x_act");
  const size_t need = mpx_linear_bwd_workspace(M, N, K);
  if (ws_bytes < need || !workspace) {
    set_error("mpx_linear_bwd: workspace of " + std::to_string(need) + " bytes required");
    return MPX_ERR_WORKSPACE;
  }
  hipStream_t s = (hipStream_t)stream;
  // dX[M,K] = dY[M,N] W[N,K]: A = dY (k-major over N), B(n=k', k=n) = W[n*K + k'] (mn-major)
  if (dX) {
    GemmArgs g = base_args();
    g.A = (const uint16_t*)dY;
    g.B = (const uint16_t*)W;
    g.C = (uint16_t*)dX;
    g.M = M; g.N = K; g.K = N;
    g.lda = N; g.ldb = K; g.ldc = K;
    g.dact = x_act ? (const uint16_t*)Xpre : nullptr;
    MPX_HIP(gemm_dispatch(dt, g, true, false, 1, s));
  }
  // dW[N,K] = dY^T X: A(m=n, k=m_tok) = dY[m_tok*N + n] (mn-major), B(n=k', k=m_tok) = X[m_tok*K + k']
  {
    GemmArgs g = base_args();
    g.A = (const uint16_t*)dY;
    g.B = (const uint16_t*)X;
    g.C = (uint16_t*)dW;
    g.M = N; g.N = K; g.K = M;
    g.lda = N; g.ldb = K; g.ldc = K;
    const int sp = choose_splits(N, K, M);
    if (sp > 1) {
      g.splits = sp;
      g.k_split = ((M + sp - 1) / sp + 63) / 64 * 64;
      g.splits = (int)((M + g.k_split - 1) / g.k_split);
      g.ws = (float*)workspace;
      MPX_HIP(gemm_dispatch(dt, g, false, false, 1, s));
      const int64_t MN = N * K;
      if (dt == MPX_F16)
        splitk_reduce_kernel<MPX_F16><<<(unsigned)((MN + 255) / 256), 256, 0, s>>>(g.ws, g.splits, MN, (uint16_t*)dW);
      else
        splitk_reduce_kernel<MPX_BF16><<<(unsigned)((MN + 255) / 256), 256, 0, s>>>(g.ws, g.splits, MN, (uint16_t*)dW);
      MPX_LAUNCHED();
    } else {
      MPX_HIP(gemm_dispatch(dt, g, false, false, 1, s));
    }
  }
  if (db) {
    if (dt == MPX_F16)
      MPX_HIP(colsum_run<MPX_F16>((const uint16_t*)dY, M, N, (float*)workspace, (uint16_t*)db, s));
    else
      MPX_HIP(colsum_run<MPX_BF16>((const uint16_t*)dY, M, N, (float*)workspace, (uint16_t*)db, s));
  }
  return MPX_OK;
}

extern "C" int mpx_gemm_batched(int32_t trans_a, int32_t trans_b, int64_t M, int64_t N, int64_t K,
                                int64_t nb0, int64_t nb1, const void* A, int64_t lda, int64_t sA0,
                                int64_t sA1, const void* B, int64_t ldb, int64_t sB0, int64_t sB1,
                                void* C, int64_t ldc, int64_t sC0, int64_t sC1, mpx_dtype dt,
                                void* stream) {
  clear_error();
  MPX_REQUIRE(A && B && C, "NULL operand");
  MPX_REQUIRE(M >= 1 && N >= 1 && K >= 1 && nb0 >= 1 && nb1 >= 1, "sizes must be >= 1");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_REQUIRE(nb0 * nb1 <= 65535, "at most 65535 batch entries");
  MPX_REQUIRE(ldc >= N && (trans_a ? lda >= M : lda >= K) && (trans_b ? ldb >= K : ldb >= N),
              "leading dimension too small");
  GemmArgs g = base_args();
  g.A = (const uint16_t*)A;
  g.B = (const uint16_t*)B;
  g.C = (uint16_t*)C;
  g.M = M; g.N = N; g.K = K;
  g.lda = lda; g.ldb = ldb; g.ldc = ldc;
  g.sA0 = sA0; g.sA1 = sA1; g.sB0 = sB0; g.sB1 = sB1; g.sC0 = sC0; g.sC1 = sC1;
  g.nb1 = nb1;
  // opA(m,k): trans_a == 0 -> A[m*lda + k] (k-major); opB(k,n): trans_b == 1 -> B[n*ldb + k] (k-major)
  MPX_HIP(gemm_dispatch(dt, g, trans_a == 0, trans_b != 0, nb0 * nb1, (hipStream_t)stream));
  return MPX_OK;
}
