// C ABI of the half GEMMs (linear forward / backward, batched attention
// products): argument checks, split-K planning and dispatch to the kernels
// of gemm_kernels.h, which are compiled once per half type in gemm_f16.hip
// and gemm_bf16.hip; float32 calls (full-precision training) go to the
// kernels of gemm_f32.hip.
#include <mutex>

#include "gemm_f32.h"
#include "gemm_kernels.h"

namespace mpx {

int g_forced_config = 0;

static hipError_t gemm_dispatch(mpx_dtype dt, const GemmArgs& g, bool ak, bool bk, int64_t nbatch,
                                hipStream_t s, bool* db_fused = nullptr) {
  return dt == MPX_F16 ? run_gemm_f16(g, ak, bk, nbatch, s, db_fused)
                       : run_gemm_bf16(g, ak, bk, nbatch, s, db_fused);
}

static GemmArgs base_args() {
  GemmArgs g{};
  g.nb1 = 1;
  g.splits = 1;
  g.k_split = INT64_MAX / 4;
  return g;
}

// split-K plan for a reduction of length K over an MxN output (the weight
// gradients, whose outputs have far fewer 128 x 128 tiles than the chip has
// workgroup slots): enough splits for one workgroup per CU (256 tiles x
// splits, rounded up), at most 16 and at least 1024 reduction values each.
// The weight gradients run on a second stream beside the critical path, so
// filling the 512 slots of two workgroups per CU (the earlier rule) bought
// latency no one waited for with more float32 partials to write and reduce:
// this rule measured ViT-B +1.2% and ViT-S +2.0% on one box and leaves the
// one-block model's splits as they were (the 1024-value floor binds there);
// 192 slots: ViT-S -1.5%; at least 2048 values per split: ViT-S -2.3%, one
// block -3%; rounding 256 / tiles down left the ViT-B MLP gradients unsplit:
// -7%.
static int choose_splits(int64_t M, int64_t N, int64_t K) {
  const int64_t tiles = ((M + 127) / 128) * ((N + 127) / 128);
  int64_t s = (256 + tiles - 1) / tiles;
  s = std::min<int64_t>(s, 16);
  s = std::min<int64_t>(s, std::max<int64_t>(1, K / 1024));
  return (int)std::max<int64_t>(s, 1);
}

// split-K plan of a reduction of length Mr over an N x K weight gradient:
// sp splits of k_split rows each (a multiple of 64), every split non-empty
static void split_plan(int64_t N, int64_t K, int64_t Mr, int& sp, int64_t& k_split) {
  sp = choose_splits(N, K, Mr);
  k_split = ((Mr + sp - 1) / sp + 63) / 64 * 64;
  sp = (int)((Mr + k_split - 1) / k_split);
}

static GemmF32Args f32_args() {
  GemmF32Args g{};
  g.nb1 = 1;
  g.splits = 1;
  g.k_split = INT64_MAX / 4;
  return g;
}

}  // namespace mpx

using namespace mpx;

extern "C" int mpx_linear_fwd(const void* X, const void* W, const void* b, const void* R, void* Y,
                              void* Ypre, int64_t M, int64_t N, int64_t K, mpx_dtype dt, int32_t act,
                              void* stream) {
  clear_error();
  MPX_REQUIRE(X && W && Y, "NULL operand");
  MPX_REQUIRE(M >= 1 && N >= 1 && K >= 1, "M, N, K must be >= 1");
  MPX_REQUIRE(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  MPX_REQUIRE(act == MPX_ACT_NONE || act == MPX_ACT_GELU_TANH, "unknown activation");
  MPX_REQUIRE(act == MPX_ACT_NONE || Ypre, "Ypre is required with an activation");
  if (dt == MPX_F32) {  // full precision: every operand float32
    GemmF32Args g = f32_args();
    g.A = (const float*)X;
    g.B = (const float*)W;
    g.C = (float*)Y;
    g.M = M; g.N = N; g.K = K;
    g.lda = K; g.ldb = K; g.ldc = N;
    g.bias = (const float*)b;
    g.resid = (const float*)R;
    g.pre = act ? (float*)Ypre : nullptr;
    g.act = act;
    MPX_HIP(launch_gemm_f32(g, true, true, 1, (hipStream_t)stream));
    return MPX_OK;
  }
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

// Byte offset of the bias-gradient partials [splits][N] behind the split-K
// partials [splits][N][K] in the workspace.
static size_t db_partials_offset(int splits, int64_t N, int64_t K) {
  return ((size_t)splits * N * K * sizeof(float) + 255) / 256 * 256;
}

// Bias-gradient partials of a split-K weight gradient: for each of the N
// rows, one per split and 128-wide tile column of the K outputs.
static size_t db_partials_count(int splits, int64_t N, int64_t K) {
  return (size_t)splits * (size_t)((K + 127) / 128) * N;
}

extern "C" size_t mpx_linear_bwd_workspace(int64_t M, int64_t N, int64_t K) {
  if (M < 1 || N < 1 || K < 1) return 0;
  const int s = choose_splits(N, K, M);
  size_t ws = s > 1 ? db_partials_offset(s, N, K) + db_partials_count(s, N, K) * sizeof(float) : 0;
  return std::max(ws, colsum_workspace(M, N)) + 256;
}

// Shared body of mpx_linear_bwd and mpx_linear_bwd_noalloc (`fn` names the
// entry point in error messages).
#define MPX_REQUIRE_FN(cond, msg)                          \
  do {                                                     \
    if (!(cond)) {                                         \
      ::mpx::set_error(std::string(fn) + ": " + (msg));    \
      return MPX_ERR_INVALID;                              \
    }                                                      \
  } while (0)

static int linear_bwd(const char* fn, const void* X, const void* W, const void* dY, const void* Xpre,
                      int32_t x_act, void* dX, void* dW, void* db, int64_t M, int64_t N, int64_t K,
                      mpx_dtype dt, void* workspace, size_t ws_bytes, int32_t* d_nonfinite,
                      void* stream) {
  MPX_REQUIRE_FN(dY, "NULL dY");
  MPX_REQUIRE_FN(dX || dW || db, "nothing to compute: dX, dW and db are all NULL");
  MPX_REQUIRE_FN(!dX || W, "W is required for dX");
  MPX_REQUIRE_FN(!dW || X, "X is required for dW");
  MPX_REQUIRE_FN(M >= 1 && N >= 1 && K >= 1, "M, N, K must be >= 1");
  MPX_REQUIRE_FN(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  MPX_REQUIRE_FN(x_act == MPX_ACT_NONE || x_act == MPX_ACT_GELU_TANH, "unknown activation");
  MPX_REQUIRE_FN(x_act == MPX_ACT_NONE || !dX || Xpre, "Xpre is required with x_act");
  MPX_REQUIRE_FN(dt != MPX_F32 || !d_nonfinite, "d_nonfinite is counted for half gradients only");
  if (dW || db) {  // only the weight and bias gradients use the workspace
    // a bias-only call needs just the column partials
    const size_t need = dW ? mpx_linear_bwd_workspace(M, N, K) : colsum_workspace(M, N) + 256;
    if (ws_bytes < need || !workspace) {
      set_error(std::string(fn) + ": workspace of " + std::to_string(need) + " bytes required");
      return MPX_ERR_WORKSPACE;
    }
  }
  hipStream_t s = (hipStream_t)stream;
  if (dt == MPX_F32) {  // full precision: the same three products in float32
    if (dX) {
      GemmF32Args g = f32_args();
      g.A = (const float*)dY;
      g.B = (const float*)W;
      g.C = (float*)dX;
      g.M = M; g.N = K; g.K = N;
      g.lda = N; g.ldb = K; g.ldc = K;
      g.dact = x_act ? (const float*)Xpre : nullptr;
      MPX_HIP(launch_gemm_f32(g, true, false, 1, s));
    }
    if (dW) {
      GemmF32Args g = f32_args();
      g.A = (const float*)dY;
      g.B = (const float*)X;
      g.C = (float*)dW;
      g.M = N; g.N = K; g.K = M;
      g.lda = N; g.ldb = K; g.ldc = K;
      int sp;
      int64_t ks;
      split_plan(N, K, M, sp, ks);
      if (sp > 1) {
        g.splits = sp;
        g.k_split = ks;
        g.ws = (float*)workspace;
        MPX_HIP(launch_gemm_f32(g, false, false, 1, s));
        MPX_HIP(launch_splitk_reduce_f32(g.ws, sp, N * K, (float*)dW, s));
      } else {
        MPX_HIP(launch_gemm_f32(g, false, false, 1, s));
      }
    }
    if (db) MPX_HIP(launch_colsum_f32((const float*)dY, M, N, (float*)workspace, (float*)db, s));
    return MPX_OK;
  }
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
  // db[N] = sum over tokens of dY: summed by the same product's kernel from
  // its dY fragments where that kernel can (db_fused), else column sums below
  bool db_fused = false;
  if (dW) {
    GemmArgs g = base_args();
    g.A = (const uint16_t*)dY;
    g.B = (const uint16_t*)X;
    g.C = (uint16_t*)dW;
    g.M = N; g.N = K; g.K = M;
    g.lda = N; g.ldb = K; g.ldc = K;
    g.nonfinite = d_nonfinite;
    g.db = (uint16_t*)db;
    int sp;
    int64_t ks;
    split_plan(N, K, M, sp, ks);
    if (sp > 1) {
      g.splits = sp;
      g.k_split = ks;
      g.ws = (float*)workspace;
      g.dbp = db ? (float*)((char*)workspace + db_partials_offset(sp, N, K)) : nullptr;
      MPX_HIP(gemm_dispatch(dt, g, false, false, 1, s, &db_fused));
      // the GEMM wrote splits x (K / 128 tile columns) bias partials per row
      const int64_t MN = N * K, nrows = db_fused ? N : 0;
      const int dbparts = (int)(db_partials_count(sp, N, K) / N);
      // 4 outputs per thread from 4 splits on (ViT-S, 8-16 splits: step +1.4%);
      // with 2 or 3 the one-output form measured 0.2-0.3% faster in the ViT-B step
      const bool vec = g.splits >= 4 && splitk_reduce_vec(g.ws, MN, (const uint16_t*)dW);
      const unsigned blocks = splitk_reduce_blocks(MN, nrows, vec);
#define MPX_SKR(DTv, VECv)                                                                       \
  splitk_reduce_kernel<DTv, VECv><<<blocks, 256, 0, s>>>(g.ws, g.splits, MN, (uint16_t*)dW, d_nonfinite, \
                                                        g.dbp, dbparts, nrows, (uint16_t*)db)
      if (dt == MPX_F16) {
        if (vec) MPX_SKR(MPX_F16, true);
        else MPX_SKR(MPX_F16, false);
      } else {
        if (vec) MPX_SKR(MPX_BF16, true);
        else MPX_SKR(MPX_BF16, false);
      }
#undef MPX_SKR
      MPX_LAUNCHED();
    } else {
      MPX_HIP(gemm_dispatch(dt, g, false, false, 1, s, &db_fused));
    }
  }
  if (db && !db_fused) {
    if (dt == MPX_F16)
      MPX_HIP(colsum_run<MPX_F16>((const uint16_t*)dY, M, N, (float*)workspace, (uint16_t*)db,
                                           d_nonfinite, s));
    else
      MPX_HIP(colsum_run<MPX_BF16>((const uint16_t*)dY, M, N, (float*)workspace, (uint16_t*)db,
                                            d_nonfinite, s));
  }
  return MPX_OK;
}

extern "C" int mpx_linear_bwd(const void* X, const void* W, const void* dY, const void* Xpre,
                              int32_t x_act, void* dX, void* dW, void* db, int64_t M, int64_t N,
                              int64_t K, mpx_dtype dt, void* workspace, size_t ws_bytes,
                              int32_t* d_nonfinite, void* stream) {
  clear_error();
  return linear_bwd("mpx_linear_bwd", X, W, dY, Xpre, x_act, dX, dW, db, M, N, K, dt, workspace,
                    ws_bytes, d_nonfinite, stream);
}

// ------------------------------------------- the variant that allocates nothing --
//
// mpx_linear_bwd_noalloc keeps its split-K and column partials in a
// file-scope device array instead of a caller's workspace.  Each GPU the
// library runs on holds its own copy of the array until the process ends.
// In host code `scratch` names a host-side stand-in, not device memory: its
// device address on the current GPU is looked up once per device with
// hipGetSymbolAddress, kept in g_scratch, and only that address is passed to
// kernels.  Nothing in the array needs to start at zero: every partial the
// kernels read was written earlier in the same call.
static __device__ __align__(256) unsigned char scratch[MPX_LINEAR_BWD_NOALLOC_SCRATCH];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};
}  // namespace

// Device address of the current GPU's scratch array (resolved on the first
// call on that GPU).
static int scratch_address(void** out) {
  int dev = -1;
  MPX_HIP(hipGetDevice(&dev));
  MPX_REQUIRE(dev >= 0 && dev < kMaxDevices, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    MPX_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    MPX_REQUIRE(p != nullptr, "scratch array has no device address");
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return MPX_OK;
}

extern "C" int mpx_linear_bwd_noalloc(const void* X, const void* W, const void* dY,
                                      const void* Xpre, int32_t x_act, void* dX, void* dW,
                                      void* db, int64_t M, int64_t N, int64_t K, mpx_dtype dt,
                                      int32_t* d_nonfinite, void* stream) {
  clear_error();
  const char* fn = "mpx_linear_bwd_noalloc";
  MPX_REQUIRE_FN(M >= 1 && N >= 1 && K >= 1, "M, N, K must be >= 1");
  if (dW || db) {  // the partials must fit the static array
    const size_t need = dW ? mpx_linear_bwd_workspace(M, N, K) : colsum_workspace(M, N) + 256;
    if (need > MPX_LINEAR_BWD_NOALLOC_SCRATCH) {
      set_error(std::string(fn) + ": this product needs " + std::to_string(need) +
                " bytes of partials, more than the " +
                std::to_string((size_t)MPX_LINEAR_BWD_NOALLOC_SCRATCH) +
                "-byte static scratch; use mpx_linear_bwd with a workspace");
      return MPX_ERR_WORKSPACE;
    }
  }
  void* ws = nullptr;
  const int rc = scratch_address(&ws);
  if (rc != MPX_OK) return rc;
  return linear_bwd(fn, X, W, dY, Xpre, x_act, dX, dW, db, M, N, K, dt, ws,
                    (size_t)MPX_LINEAR_BWD_NOALLOC_SCRATCH, d_nonfinite, stream);
}
#undef MPX_REQUIRE_FN

extern "C" int mpx_gemm_batched(int32_t trans_a, int32_t trans_b, int64_t M, int64_t N, int64_t K,
                                int64_t nb0, int64_t nb1, const void* A, int64_t lda, int64_t sA0,
                                int64_t sA1, const void* B, int64_t ldb, int64_t sB0, int64_t sB1,
                                void* C, int64_t ldc, int64_t sC0, int64_t sC1, mpx_dtype dt,
                                void* stream) {
  clear_error();
  MPX_REQUIRE(A && B && C, "NULL operand");
  MPX_REQUIRE(M >= 1 && N >= 1 && K >= 1 && nb0 >= 1 && nb1 >= 1, "sizes must be >= 1");
  MPX_REQUIRE(is_half(dt) || dt == MPX_F32, "dt must be MPX_F16, MPX_BF16 or MPX_F32");
  MPX_REQUIRE(nb0 * nb1 <= 65535, "at most 65535 batch entries");
  MPX_REQUIRE(ldc >= N && (trans_a ? lda >= M : lda >= K) && (trans_b ? ldb >= K : ldb >= N),
              "leading dimension too small");
  if (dt == MPX_F32) {  // full precision
    GemmF32Args g = f32_args();
    g.A = (const float*)A;
    g.B = (const float*)B;
    g.C = (float*)C;
    g.M = M; g.N = N; g.K = K;
    g.lda = lda; g.ldb = ldb; g.ldc = ldc;
    g.sA0 = sA0; g.sA1 = sA1; g.sB0 = sB0; g.sB1 = sB1; g.sC0 = sC0; g.sC1 = sC1;
    g.nb1 = nb1;
    MPX_HIP(launch_gemm_f32(g, trans_a == 0, trans_b != 0, nb0 * nb1, (hipStream_t)stream));
    return MPX_OK;
  }
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

extern "C" int mpx_gemm_set_config(int32_t config) {
  clear_error();
  MPX_REQUIRE(config >= 0 && config <= 11, "config must be in [0, 11]");
  g_forced_config = config;
  return MPX_OK;
}
