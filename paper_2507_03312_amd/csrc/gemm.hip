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
#include <utility>

#include "colsum.h"
#include "common.h"

namespace mpx {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
// Clang vector types for 8- and 16-byte global accesses (a store through the
// HIP uint2 / float4 structs is split into 4-byte stores)
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

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

// Compile-time loop: f(std::integral_constant<int, I>) for I in [0, N).  The
// accumulator tiles are indexed only with such constants, so they stay in
// registers (a runtime index would force them into scratch memory).
template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

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

  // rows_valid: rows r < rows_valid exist; k_valid: reduction values k < k_valid exist.
  //
  // VEC (16-byte aligned base, leading dimension a multiple of 8): every load
  // is a plain 16-byte load with no branch, so the compiler keeps the next
  // stage's loads in flight.  A vector that starts inside the matrix lies
  // wholly inside its row's leading dimension (ld is a multiple of 8 and at
  // least the row length), so it is loaded whole and its elements past the
  // end are zeroed; a vector that starts outside is redirected to the tile's
  // first vector (always inside) and zeroed entirely.
  __device__ __forceinline__ static uint4 mask_vec(uint4 v, int nvalid) {
    // keep elements [0, nvalid) of 8, zero the rest
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint32_t lo = 2 * q < nvalid ? 0x0000FFFFu : 0u;
      const uint32_t hi = 2 * q + 1 < nvalid ? 0xFFFF0000u : 0u;
      o[q] = w[q] & (lo | hi);
    }
    return make_uint4(o[0], o[1], o[2], o[3]);
  }

  // extent of the tile last loaded (the masking happens in store(), next to
  // the LDS writes, so that nothing waits on the loads before then)
  int rv_ = ROWS, kv_ = BK;

  __device__ __forceinline__ void load(const uint16_t* __restrict__ base, int64_t ld, int rows_valid,
                                       int k_valid, int tid) {
    rv_ = rows_valid;
    kv_ = k_valid;
    // a whole tile (the common case) needs no clamping or masking; the test
    // is uniform over the workgroup, so it costs one scalar branch
    const bool full = rows_valid >= ROWS && k_valid >= BK;
    if constexpr (!VEC) {
      load_guarded(base, ld, rows_valid, k_valid, tid);
    } else {
#pragma unroll
      for (int u = 0; u < PER; ++u) {
        const int unit = tid + u * NT;
        if constexpr (KMAJ) {
          const int r = unit / (BK / 8);
          const int k = (unit % (BK / 8)) * 8;
          const bool inside = full || (r < rows_valid && k < k_valid);
          const int64_t off = inside ? (int64_t)r * ld + k : 0;
          reg[u] = *reinterpret_cast<const uint4*>(base + off);
        } else {
          const int r = (unit / (BK / KR)) * 8;
          const int k = (unit % (BK / KR)) * KR;
#pragma unroll
          for (int q = 0; q < KR; ++q) {
            const bool inside = full || (k + q < k_valid && r < rows_valid);
            const int64_t off = inside ? (int64_t)(k + q) * ld + r : 0;
            reg[u * KR + q] = *reinterpret_cast<const uint4*>(base + off);
          }
        }
      }
    }
  }

  __device__ __forceinline__ void load_guarded(const uint16_t* __restrict__ base, int64_t ld,
                                               int rows_valid, int k_valid, int tid) {
    auto pack8 = [](const uint16_t (&h)[8]) {
      return make_uint4(h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16),
                        h[4] | ((uint32_t)h[5] << 16), h[6] | ((uint32_t)h[7] << 16));
    };
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int unit = tid + u * NT;
      if constexpr (KMAJ) {
        const int r = unit / (BK / 8);
        const int k = (unit % (BK / 8)) * 8;
        const uint16_t* p = base + (int64_t)r * ld + k;
        uint16_t h[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) h[j] = (r < rows_valid && k + j < k_valid) ? p[j] : (uint16_t)0;
        reg[u] = pack8(h);
      } else {
        const int r = (unit / (BK / KR)) * 8;
        const int k = (unit % (BK / KR)) * KR;
#pragma unroll
        for (int q = 0; q < KR; ++q) {
          const uint16_t* p = base + (int64_t)(k + q) * ld + r;
          uint16_t h[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) h[j] = (k + q < k_valid && r + j < rows_valid) ? p[j] : (uint16_t)0;
          reg[u * KR + q] = pack8(h);
        }
      }
    }
  }

  // LDS tile: ROWS rows of pitch LDSP halves.
  template <int LDSP>
  __device__ __forceinline__ void store(uint16_t* __restrict__ lds, int tid) const {
    const int rv_ = this->rv_, kv_ = this->kv_;
    const bool full = rv_ >= ROWS && kv_ >= BK;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
      const int unit = tid + u * NT;
      if constexpr (KMAJ) {
        const int r = unit / (BK / 8);
        const int k = (unit % (BK / 8)) * 8;
        uint4 v = reg[u];
        if (VEC && !full) v = mask_vec(v, r < rv_ && k < kv_ ? min(8, kv_ - k) : 0);
        *reinterpret_cast<uint4*>(lds + r * LDSP + k) = v;
      } else {
        const int r = (unit / (BK / KR)) * 8;
        const int k = (unit % (BK / KR)) * KR;
        // register transpose: lane holds rows k..k+KR-1 of 8 consecutive
        // output indices; write output index r+j as KR consecutive k values
        uint32_t w[KR][4];
#pragma unroll
        for (int q = 0; q < KR; ++q) {
          uint4 v = reg[u * KR + q];
          if (VEC && !full) v = mask_vec(v, k + q < kv_ && r < rv_ ? min(8, rv_ - r) : 0);
          w[q][0] = v.x;
          w[q][1] = v.y;
          w[q][2] = v.z;
          w[q][3] = v.w;
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

// Output tile of this workgroup.  Workgroups are dealt to the 8 XCDs
// round-robin (workgroup w runs on XCD w % 8); they are renumbered so that
// each XCD works through one contiguous range of tiles, and that range is
// walked in groups of 8 tile rows, column by column, so the tiles an XCD
// runs at the same time form a compact block: their A row panels and B
// column panels are shared through that XCD's L2 instead of each B panel
// being fetched again for every tile row.
template <int BM, int BN>
__device__ __forceinline__ void tile_origin(int64_t M, int64_t N, int64_t& m0, int64_t& n0) {
  constexpr int64_t GM = 8;
  const int64_t tiles_m = (M + BM - 1) / BM, tiles_n = (N + BN - 1) / BN;
  const int64_t ntiles = gridDim.x;
  const int64_t xcd = blockIdx.x % 8, local = blockIdx.x / 8;
  const int64_t t = xcd * (ntiles / 8) + min(xcd, ntiles % 8) + local;
  const int64_t first = (t / (GM * tiles_n)) * GM;
  const int64_t gm = min(tiles_m - first, GM);
  const int64_t r = t - first * tiles_n;
  m0 = (first + r % gm) * BM;
  n0 = (r / gm) * BN;
}

// Epilogue shared by the GEMM kernels: the wave's TM x TN accumulator
// blocks of 32 x 32 start at output row mw and column nw.
template <int DT, int TM, int TN>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& g, const f32x16 (&acc)[TM][TN],
                                              int64_t mw, int64_t nw, int lane, int split,
                                              int64_t offC) {
  // The accumulators of a 32x32 block hold, per lane, one column and 4 runs
  // of 4 consecutive rows.  A 4x4 transpose across each group of 4 lanes
  // (two butterfly exchanges) turns every run into 4 consecutive columns of
  // one row, so bias / residual / activation inputs are read and outputs
  // written 4 elements (8 bytes; 16 for float partials) at a time.
  const int q4 = lane & 3;
  const int row_l = 4 * (lane >> 5) + q4;        // row within an 8-row group
  const int col_l = 4 * ((lane & 31) >> 2);      // first of the lane's 4 columns
  // exchange (p, p + st) pairs with the lane st apart (st = 1 or 2) through a
  // DPP quad permutation (lane ^ 1: quad_perm [1,0,3,2]; lane ^ 2: [2,3,0,1])
  auto xchg = [&](float& lo, float& hi_v, int st) {
    const bool hi = (q4 & st) != 0;
    const int send = __builtin_bit_cast(int, hi ? lo : hi_v);
    const int got = st == 1 ? __builtin_amdgcn_mov_dpp(send, 0xB1, 0xF, 0xF, false)
                            : __builtin_amdgcn_mov_dpp(send, 0x4E, 0xF, 0xF, false);
    if (hi) lo = __builtin_bit_cast(float, got);
    else hi_v = __builtin_bit_cast(float, got);
  };
  auto transpose4 = [&](float (&v)[4]) {
    xchg(v[0], v[1], 1);
    xchg(v[2], v[3], 1);
    xchg(v[0], v[2], 2);
    xchg(v[1], v[3], 2);
  };
  auto al8 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; };
  if (g.splits > 1) {
    float* W = g.ws + (int64_t)split * g.M * g.N;
    const bool v16 = g.N % 4 == 0 && (reinterpret_cast<uintptr_t>(W) & 15u) == 0;
    static_for<TM>([&](auto i) {
      static_for<TN>([&](auto j) {
        const f32x16 a = acc[i][j];
#pragma unroll
        for (int qd = 0; qd < 4; ++qd) {
          float v[4] = {a[4 * qd], a[4 * qd + 1], a[4 * qd + 2], a[4 * qd + 3]};
          transpose4(v);
          const int64_t m = mw + i * 32 + 8 * qd + row_l;
          const int64_t n = nw + j * 32 + col_l;
          if (m < g.M && n < g.N) {
            float* out = W + m * g.N + n;
            if (v16 && n + 4 <= g.N) *reinterpret_cast<f32x4*>(out) = f32x4{v[0], v[1], v[2], v[3]};
            else
#pragma unroll
              for (int c = 0; c < 4; ++c)
                if (n + c < g.N) out[c] = v[c];
          }
        }
      });
    });
    return;
  }
  uint16_t* C = g.C + offC;
  const bool v8 = g.ldc % 4 == 0 && al8(C) && (!g.pre || al8(g.pre)) && (!g.dact || al8(g.dact)) &&
                  (!g.resid || (al8(g.resid) && g.ldr % 4 == 0)) && (!g.bias || al8(g.bias));
  auto ld4 = [&](const uint16_t* p, bool vec, int nv, uint16_t (&d)[4]) {
    if (vec) {
      const u32x2 w = *reinterpret_cast<const u32x2*>(p);
      d[0] = (uint16_t)(w.x & 0xFFFFu);
      d[1] = (uint16_t)(w.x >> 16);
      d[2] = (uint16_t)(w.y & 0xFFFFu);
      d[3] = (uint16_t)(w.y >> 16);
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c) d[c] = c < nv ? p[c] : (uint16_t)0;
    }
  };
  auto st4 = [&](uint16_t* p, bool vec, int nv, const uint16_t (&d)[4]) {
    if (vec) {
      *reinterpret_cast<u32x2*>(p) = u32x2{d[0] | ((uint32_t)d[1] << 16), d[2] | ((uint32_t)d[3] << 16)};
    } else {
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (c < nv) p[c] = d[c];
    }
  };
  static_for<TM>([&](auto i) {
    static_for<TN>([&](auto j) {
      const f32x16 a = acc[i][j];
      const int64_t n = nw + j * 32 + col_l;
      const int nv = (int)max<int64_t>(0, min<int64_t>(4, g.N - n));
      const bool vec = v8 && nv == 4;
      uint16_t bias[4] = {0, 0, 0, 0};
      if (g.bias && nv > 0) ld4(g.bias + n, vec, nv, bias);
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        float v[4] = {a[4 * qd], a[4 * qd + 1], a[4 * qd + 2], a[4 * qd + 3]};
        transpose4(v);
        const int64_t m = mw + i * 32 + 8 * qd + row_l;
        if (m >= g.M || nv == 0) continue;
        uint16_t h[4], da[4], res[4];
        if (g.dact) ld4(g.dact + m * g.ldc + n, vec, nv, da);
        if (g.resid) ld4(g.resid + m * g.ldr + n, vec, nv, res);
#pragma unroll
        for (int c = 0; c < 4; ++c) h[c] = f2h<DT>(v[c] + (g.bias ? h2f<DT>(bias[c]) : 0.0f));
        if (g.pre) st4(g.pre + m * g.ldc + n, vec, nv, h);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          uint16_t o = h[c];
          if (g.act == MPX_ACT_GELU_TANH) o = f2h<DT>(gelu_tanh(h2f<DT>(o)));
          if (g.dact) o = f2h<DT>(h2f<DT>(o) * gelu_tanh_grad(h2f<DT>(da[c])));
          if (g.resid) o = f2h<DT>(h2f<DT>(o) + h2f<DT>(res[c]));
          h[c] = o;
        }
        st4(C + m * g.ldc + n, vec, nv, h);
      }
    });
  });
}

// OCC: waves per SIMD the register budget is sized for.
template <int DT, int BM, int BN, int BK, int WM, int WN, bool AK, bool BKM, bool VEC, int OCC>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(OCC, OCC)))
void gemm_kernel(GemmArgs g) {
  constexpr int NW = (BM / WM) * (BN / WN);
  constexpr int NT = NW * 64;
  constexpr int PAD = 8;
  constexpr int LDSP = BK + PAD;
  constexpr int TM = WM / 32, TN = WN / 32;
  // one LDS block: the double-buffered A and B tiles during the main loop,
  // then the float32 staging area of the epilogue
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (BM + BN) * LDSP];
  uint16_t (*sA)[BM * LDSP] = reinterpret_cast<uint16_t (*)[BM * LDSP]>(smem);
  uint16_t (*sB)[BN * LDSP] = reinterpret_cast<uint16_t (*)[BN * LDSP]>(smem + 2 * BM * LDSP);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm0 = (wave / (BN / WN)) * WM;
  const int wn0 = (wave % (BN / WN)) * WN;

  int64_t m0, n0;
  tile_origin<BM, BN>(g.M, g.N, m0, n0);
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

  // One register stage: the loads of k tile kt+1 are issued before the MFMAs
  // of tile kt and land in LDS (the other buffer) after them.
  TileLoader<BM, BK, NT, AK, VEC> la;
  TileLoader<BN, BK, NT, BKM, VEC> lb;

  f32x16 acc[TM][TN];
  static_for<TM>([&](auto i) {
    static_for<TN>([&](auto j) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;
    });
  });

  auto kvalid = [&](int kt) { return (int)min<int64_t>(BK, kend - (kbeg + (int64_t)kt * BK)); };
  if (nk > 0) {
    la.load(Ab, g.lda, rowsA, kvalid(0), tid);
    lb.load(Bb, g.ldb, rowsB, kvalid(0), tid);
    la.template store<LDSP>(sA[0], tid);
    lb.template store<LDSP>(sB[0], tid);
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int c = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load(Ab + (kt + 1) * Astep, g.lda, rowsA, kvalid(kt + 1), tid);
      lb.load(Bb + (kt + 1) * Bstep, g.ldb, rowsB, kvalid(kt + 1), tid);
    }
    const uint16_t* a_s = sA[c];
    const uint16_t* b_s = sB[c];
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
      static_for<TM>([&](auto i) {
        static_for<TN>([&](auto j) { acc[i][j] = mfma32<DT>(af[i], bf[j], acc[i][j]); });
      });
    }
    if (more) {
      la.template store<LDSP>(sA[c ^ 1], tid);
      lb.template store<LDSP>(sB[c ^ 1], tid);
    }
    __syncthreads();
  }

  gemm_epilogue<DT, TM, TN>(g, acc, m0 + wm0, n0 + wn0, lane, split, offC);
}

// ------------------------------------------------- direct-to-LDS kernel --
//
// The main loop of the kernel below moves operand tiles from global memory
// straight into LDS (global_load_lds_dwordx4: each lane's 16 bytes land at
// M0 + 16 * lane, so one wave instruction fills 1 KiB of LDS) and keeps
// S - 1 k tiles of 64 in flight while the MFMAs consume the oldest one.  No
// registers stage the tiles, so deep pipelines cost LDS only.  The compiler
// does not track these copies: each k step waits for its own tile with an
// explicit vmcnt and one barrier makes the tile visible to every wave.
//
// LDS layouts (no padding: a copy fills 1 KiB contiguously, so bank
// conflicts are avoided by permuting 16-byte chunks instead):
//   k-major operand   [row][64 k], 128 B per row; chunk c of row r sits at
//                     position c ^ ((r >> 1) & 7).  The 16 lanes reading one
//                     ds_read_b128 phase (16 rows, one chunk) hit all 64 banks.
//   mn-major operand  [k][ROWS] (ROWS = 128 or 256 outputs, 16 or 32 chunks
//                     per k row); chunk c of k row kr sits at c ^ (4*(kr & 3)).
//                     MFMA fragments are read with ds_read_b64_tr_b16, which
//                     transposes 16-bit elements across groups of 16 lanes, so
//                     the operand needs no transposition on the way in.
// Requirements (checked by the dispatcher): 16-byte aligned operands with
// leading dimensions and batch strides that are multiples of 8, and every
// split's k range a multiple of 64.  Rows past M or N read clamped (valid)
// addresses; their results are never stored.

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane from base + off (bytes) into LDS at lds + 16 * lane
__device__ __forceinline__ void dma16(const void* base, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(off), "s"(base), "s"(lds)
               : "memory", "m0");
}
#pragma clang diagnostic pop

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

__device__ __forceinline__ uint32_t lds_u32(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

typedef short s16x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint2 lds_tr_b64(uint32_t addr) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(uintptr_t)addr);
  return __builtin_bit_cast(uint2, v);
}

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 lds_b128(uint32_t addr) {
  const u32x4 v = *(const __attribute__((address_space(3))) u32x4*)(uintptr_t)addr;
  return __builtin_bit_cast(uint4, v);
}

// One operand of the direct-to-LDS kernel: ROWS output rows (of M or N) by
// 64 k per stage, copied by NWAVES waves, Q copies per wave.
template <int ROWS, bool KMAJ, int NWAVES>
struct DmaOperand {
  static constexpr int BLOCKS = ROWS / 8;  // 1 KiB copies per stage
  static constexpr int Q = BLOCKS / NWAVES;
  static_assert(BLOCKS % NWAVES == 0, "copies do not split evenly over the waves");
  static_assert(KMAJ || ROWS == 128 || ROWS == 256, "mn-major tiles are 128 or 256 wide");
  uint32_t off[Q];  // per-lane byte offsets of the copies, relative to the tile base
  int64_t step;     // bytes from one k tile to the next

  // rv: valid rows (>= 1) of the tile; ld: leading dimension in elements
  __device__ __forceinline__ void init(int64_t ld, int rv, int wave, int lane) {
    if constexpr (KMAJ) {
      step = 128;
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int r = 8 * (wave + NWAVES * q) + (lane >> 3);
        const int c = (lane & 7) ^ ((r >> 1) & 7);
        off[q] = (uint32_t)(min(r, rv - 1) * ld * 2 + c * 16);
      }
    } else {
      constexpr int CH = ROWS / 8;   // 16-byte chunks per k row
      constexpr int RPB = 64 / CH;   // k rows per 1 KiB copy
      step = 64 * ld * 2;
#pragma unroll
      for (int q = 0; q < Q; ++q) {
        const int kr = RPB * (wave + NWAVES * q) + lane / CH;
        const int c = (lane % CH) ^ (4 * (kr & 3));
        off[q] = (uint32_t)(kr * ld * 2 + (8 * c < rv ? 16 * c : 0));
      }
    }
  }
  // copy the tile whose first element is at base into LDS at lds
  __device__ __forceinline__ void issue(const uint16_t* base, uint32_t lds, int wave) const {
#pragma unroll
    for (int q = 0; q < Q; ++q)
      dma16(base, off[q], lds + 1024u * (uint32_t)(wave + NWAVES * q));
  }
};

// Per-lane LDS byte offsets of the MFMA fragments of one operand, for a
// wave whose rows start at w0 within the tile (relative to the tile base).
template <int ROWS, bool KMAJ, int T>
struct FragReader {
  uint32_t base[KMAJ ? 4 : T];
  __device__ __forceinline__ void init(int w0, int lane) {
    if constexpr (KMAJ) {
      const int r = w0 + (lane & 31);
      const int sw = (r >> 1) & 7;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) base[kk] = (uint32_t)(r * 128 + (((2 * kk + (lane >> 5)) ^ sw) << 4));
    } else {
      const int g = lane >> 4, e = (lane >> 2) & 3, t = lane & 3;
      const int kr = 8 * (g >> 1) + e;  // + 16 kk + 4 h
#pragma unroll
      for (int i = 0; i < T; ++i) {
        const int m = w0 + 32 * i + 16 * (g & 1) + 4 * t;
        base[i] = (uint32_t)(kr * ROWS * 2 + (((m >> 3) ^ (4 * e)) << 4) + (m & 7) * 2);
      }
    }
  }
  // fragment i (rows w0 + 32 i ..) at k step kk of the tile at lds
  template <int I, int KK>
  __device__ __forceinline__ uint4 read(uint32_t lds) const {
    if constexpr (KMAJ) {
      return lds_b128(lds + base[KK] + I * 32 * 128);
    } else {
      const uint2 lo = lds_tr_b64(lds + base[I] + KK * 16 * ROWS * 2);
      const uint2 hi = lds_tr_b64(lds + base[I] + KK * 16 * ROWS * 2 + 4 * ROWS * 2);
      return make_uint4(lo.x, lo.y, hi.x, hi.y);
    }
  }
};

// OCC: waves per SIMD the register budget is sized for.
template <int DT, int BM, int BN, int WM, int WN, int S, int OCC, bool AK, bool BKM>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(OCC, OCC)))
void gemm_dma_kernel(GemmArgs g) {
  constexpr int NWAVES = (BM / WM) * (BN / WN);
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int A_BYTES = BM * 64 * 2, B_BYTES = BN * 64 * 2;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int L = (BM + BN) / 8 / NWAVES;  // copies per lane per stage
  static_assert((S - 2) * L <= 63, "vmcnt range");
  __shared__ __attribute__((aligned(1024))) uint8_t smem[S * STAGE];
  const uint32_t lds0 = lds_u32(smem);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave / (BN / WN)) * WM;
  const int wn0 = (wave % (BN / WN)) * WN;

  int64_t m0, n0;
  tile_origin<BM, BN>(g.M, g.N, m0, n0);
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
  const int nk = (int)((kend - kbeg) / 64);

  const uint16_t* Ab = g.A + offA + (AK ? m0 * g.lda + kbeg : kbeg * g.lda + m0);
  const uint16_t* Bb = g.B + offB + (BKM ? n0 * g.ldb + kbeg : kbeg * g.ldb + n0);
  DmaOperand<BM, AK, NWAVES> da;
  DmaOperand<BN, BKM, NWAVES> db;
  da.init(g.lda, (int)min<int64_t>(BM, g.M - m0), wave, lane);
  db.init(g.ldb, (int)min<int64_t>(BN, g.N - n0), wave, lane);
  FragReader<BM, AK, TM> fa;
  FragReader<BN, BKM, TN> fb;
  fa.init(wm0, lane);
  fb.init(wn0, lane);

  f32x16 acc[TM][TN];
  static_for<TM>([&](auto i) {
    static_for<TN>([&](auto j) {
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;
    });
  });

  auto issue = [&](int kt) {
    const uint32_t st = lds0 + (uint32_t)((kt % S) * STAGE);
    da.issue(reinterpret_cast<const uint16_t*>(reinterpret_cast<const uint8_t*>(Ab) + kt * da.step), st, wave);
    db.issue(reinterpret_cast<const uint16_t*>(reinterpret_cast<const uint8_t*>(Bb) + kt * db.step),
             st + A_BYTES, wave);
  };
#pragma unroll
  for (int s = 0; s < S - 1; ++s)
    if (s < nk) issue(s);

  for (int kt = 0; kt < nk; ++kt) {
    // tile kt has landed once at most min(S - 2, nk - 1 - kt) later tiles are in flight
    const int later = min(S - 2, nk - 1 - kt);
    static_for<S - 1>([&](auto p) {
      if (later == p) wait_vmcnt<p * L>();
    });
    __syncthreads();
    if (kt + S - 1 < nk) issue(kt + S - 1);
    const uint32_t sa = lds0 + (uint32_t)((kt % S) * STAGE), sb = sa + A_BYTES;
    // fragments double-buffered over the four k steps of 16: the LDS reads
    // of step kk + 1 are issued ahead of the MFMAs of step kk (the scheduling
    // barriers keep the compiler from sinking them next to their uses)
    uint4 af[2][TM], bf[2][TN];
    static_for<TM>([&](auto i) { af[0][i] = fa.template read<i, 0>(sa); });
    static_for<TN>([&](auto j) { bf[0][j] = fb.template read<j, 0>(sb); });
    static_for<4>([&](auto kk) {
      constexpr int cur = kk & 1, nxt = cur ^ 1;
      if constexpr (kk + 1 < 4) {
        static_for<TM>([&](auto i) { af[nxt][i] = fa.template read<i, kk + 1>(sa); });
        static_for<TN>([&](auto j) { bf[nxt][j] = fb.template read<j, kk + 1>(sb); });
      }
      __builtin_amdgcn_sched_barrier(0);
      static_for<TM>([&](auto i) {
        static_for<TN>([&](auto j) { acc[i][j] = mfma32<DT>(af[cur][i], bf[cur][j], acc[i][j]); });
      });
      __builtin_amdgcn_sched_barrier(0);
    });
  }
  gemm_epilogue<DT, TM, TN>(g, acc, m0 + wm0, n0 + wn0, lane, split, offC);
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

// ------------------------------------------------------------ dispatch --

struct Cfg {
  int bm, bn;
};

static bool aligned_vec(const void* p, int64_t ld, int64_t s0, int64_t s1) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0 && ld % 8 == 0 && s0 % 8 == 0 && s1 % 8 == 0;
}

template <int DT, int BM, int BN, int WM, int WN, int BK = 64, int OCC = 2>
static hipError_t launch_cfg(const GemmArgs& g, bool ak, bool bk, bool vec, int64_t nbatch,
                             hipStream_t s) {
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  dim3 grid((unsigned)tiles, (unsigned)(g.splits > 1 ? g.splits : nbatch));
#define MPX_G(AKv, BKv, VECv) \
  gemm_kernel<DT, BM, BN, BK, WM, WN, AKv, BKv, VECv, OCC><<<grid, NT, 0, s>>>(g)
  if (vec) {
    if (ak && bk) MPX_G(true, true, true);
    else if (ak && !bk) MPX_G(true, false, true);
    else if (!ak && bk) MPX_G(false, true, true);
    else MPX_G(false, false, true);
  } else if constexpr (BM * BN <= 128 * 128) {  // unaligned operands: small tiles only
    if (ak && bk) MPX_G(true, true, false);
    else if (ak && !bk) MPX_G(true, false, false);
    else if (!ak && bk) MPX_G(false, true, false);
    else MPX_G(false, false, false);
  } else {
    return hipErrorInvalidValue;
  }
#undef MPX_G
  return hipGetLastError();
}

template <int DT, int BM, int BN, int WM, int WN, int S, int OCC>
static hipError_t launch_dma(const GemmArgs& g, bool ak, bool bk, int64_t nbatch, hipStream_t s) {
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  dim3 grid((unsigned)tiles, (unsigned)(g.splits > 1 ? g.splits : nbatch));
#define MPX_D(AKv, BKv) gemm_dma_kernel<DT, BM, BN, WM, WN, S, OCC, AKv, BKv><<<grid, NT, 0, s>>>(g)
  if (ak && bk) MPX_D(true, true);
  else if (ak && !bk) MPX_D(true, false);
  else if (!ak && bk) MPX_D(false, true);
  else MPX_D(false, false);
#undef MPX_D
  return hipGetLastError();
}

// Tile configurations (the value of mpx_gemm_set_config):
//   1  register-staged 64 x 64, 4 waves          (any operands)
//   2  register-staged 128 x 128, 8 waves        (16-byte aligned operands)
//   3  direct-to-LDS 256 x 256, 4 waves, 2 stages
//   4  direct-to-LDS 256 x 128, 4 waves, 3 stages
//   5  direct-to-LDS 128 x 256, 4 waves, 3 stages
//   6  direct-to-LDS 128 x 128, 4 waves, 4 stages
//   7  direct-to-LDS 128 x 128, 4 waves, 2 stages, two workgroups per CU
static int g_forced_config = 0;

// The direct-to-LDS kernel needs 16-byte aligned operands and whole k tiles
// of 64 in every split, and 32-bit per-lane copy offsets.
static bool dma_ok(const GemmArgs& g, bool vec, bool ak, bool bk) {
  if (!vec || g.K % 64 != 0) return false;
  if (g.splits > 1 && g.k_split % 64 != 0) return false;
  const int64_t lim = (int64_t)1 << 31;
  const int64_t spanA = (ak ? 256 : 64) * g.lda * 2, spanB = (bk ? 256 : 64) * g.ldb * 2;
  return spanA < lim && spanB < lim;
}

// Measured on MI355X over the transformer layer shapes (M 8320..25216, N and K
// 384..3072) and 8192^3: configuration 7 (two co-resident workgroups hide
// each other's epilogue and pipeline bubbles) is the fastest direct-to-LDS
// variant for every shape, forward and backward; the register-staged
// kernels serve operands the copies cannot take.
static int choose_config(const GemmArgs& g, bool vec, bool ak, bool bk) {
  const bool dma = dma_ok(g, vec, ak, bk);
  const int f = g_forced_config;
  if (f >= 3 && dma) return f;
  if (f == 1 || (f == 2 && vec)) return f;
  if (g.M <= 64 || g.N <= 64) return 1;
  if (dma) return 7;
  return vec ? 2 : 0;
}

// ak: A is k-major; bk: B is k-major.
template <int DT>
static hipError_t run_gemm(GemmArgs g, bool ak, bool bk, int64_t nbatch, hipStream_t s) {
  const bool vec = aligned_vec(g.A, g.lda, g.sA0, g.sA1) && aligned_vec(g.B, g.ldb, g.sB0, g.sB1);
  switch (choose_config(g, vec, ak, bk)) {
    case 1: return launch_cfg<DT, 64, 64, 32, 32>(g, ak, bk, vec, nbatch, s);
    case 2: return launch_cfg<DT, 128, 128, 64, 32, 64, 4>(g, ak, bk, vec, nbatch, s);
    case 3: return launch_dma<DT, 256, 256, 128, 128, 2, 1>(g, ak, bk, nbatch, s);
    case 4: return launch_dma<DT, 256, 128, 128, 64, 3, 1>(g, ak, bk, nbatch, s);
    case 5: return launch_dma<DT, 128, 256, 64, 128, 3, 1>(g, ak, bk, nbatch, s);
    case 6: return launch_dma<DT, 128, 128, 64, 64, 4, 1>(g, ak, bk, nbatch, s);
    case 7: return launch_dma<DT, 128, 128, 64, 64, 2, 2>(g, ak, bk, nbatch, s);
    default:  // unaligned operands (rare: odd leading dimensions)
      return launch_cfg<DT, 128, 128, 64, 64>(g, ak, bk, vec, nbatch, s);
  }
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
  return std::max(ws, colsum_workspace(M, N)) + 256;
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

extern "C" int mpx_gemm_set_config(int32_t config) {
  clear_error();
  MPX_REQUIRE(config >= 0 && config <= 7, "config must be in [0, 7]");
  g_forced_config = config;
  return MPX_OK;
}
