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
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <utility>

#include "colsum.h"
#include "common.h"
#include "mfma.h"

namespace mpx {

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
  int32_t full_epi;  // set by the dispatcher: whole tiles may use gemm_epilogue_lds
  // if set, the number of non-finite half outputs C is added to *nonfinite
  // (split-K partials are counted by the reduction that rounds them
  // instead); such calls take the generic epilogue or the whole-tile one
  // compiled with EPI_COUNT
  int32_t* nonfinite;
  // weight-gradient products (both operands mn-major) may also return the
  // bias gradient db[m] = half(sum_k A(m, k)), summed from the A fragments
  // the MFMAs read: set by the dispatcher only for the kernel variant that
  // does it.  Split-K calls write float32 partial sums dbp[split][M] instead,
  // which the split-K reduction adds in split order.
  uint16_t* db;
  float* dbp;
};

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
__device__ __forceinline__ void tile_origin_of(uint32_t tile, uint32_t ntiles, int64_t M, int64_t N,
                                               int64_t& m0, int64_t& n0) {
  // 32-bit index arithmetic (tile counts stay far below 2^32; a 64-bit
  // division is a long software sequence)
  constexpr uint32_t GM = 8;
  const uint32_t tiles_m = (uint32_t)((M + BM - 1) / BM), tiles_n = (uint32_t)((N + BN - 1) / BN);
  const uint32_t xcd = tile % 8, local = tile / 8;
  const uint32_t t = xcd * (ntiles / 8) + min(xcd, ntiles % 8) + local;
  const uint32_t first = (t / (GM * tiles_n)) * GM;
  const uint32_t gm = min(tiles_m - first, GM);
  const uint32_t r = t - first * tiles_n;
  m0 = (int64_t)(first + r % gm) * BM;
  n0 = (int64_t)(r / gm) * BN;
}

template <int BM, int BN>
__device__ __forceinline__ void tile_origin(int64_t M, int64_t N, int64_t& m0, int64_t& n0) {
  tile_origin_of<BM, BN>(blockIdx.x, gridDim.x, M, N, m0, n0);
}

// Epilogue variants chosen at compile time (a mask of these bits), used for
// tiles that lie wholly inside the output when every epilogue operand is
// 8-byte aligned: no per-element masks, no runtime flag tests, one 64-bit
// base per wave and 32-bit lane offsets.  The arithmetic is the generic
// epilogue's, step for step, so both give identical bits.
// EPI_COUNT: add the number of non-finite outputs to g.nonfinite (weight
// gradients, which have no other epilogue operation)
enum : int { EPI_BIAS = 1, EPI_GELU = 2, EPI_DACT = 4, EPI_RESID = 8, EPI_COUNT = 16,
             EPI_GENERIC = -1 };

// Whole-tile epilogue through LDS, for the transposed accumulator layout and
// 32 x 64 or 64 x 64 wave tiles.  Step 1 (accumulator layout: lane = one row, runs of 4
// consecutive columns): h = half(acc + bias), written to the wave's own
// [rows][68] half region of the LDS the main loop no longer needs.  Step 2 (row
// layout: lane = 8 consecutive columns of one row): the pre-activation store,
// GELU, GELU' of the previous layer and the residual add with 16-byte
// accesses, each store writing 8 rows x 128 contiguous bytes.
// pf (nullable): the wave's GELU' or residual operand rows, already loaded
// in the row layout (16 bytes of row (lane >> 3) + 8 t per entry t).
template <int DT, int TM, int TN, int E>
__device__ __forceinline__ void gemm_epilogue_lds(const GemmArgs& g, const f32x16 (&acc)[TM][TN],
                                                  int64_t mw, int64_t nw, int lane, int64_t offC,
                                                  uint16_t* lds, const u32x4* pf = nullptr) {
  static_assert((TM == 1 || TM == 2) && TN == 2, "32 x 64 or 64 x 64 wave tiles");
  constexpr int PITCH = 68;  // halves (34 banks): a column of 32 rows spreads over all banks
  const int hi = lane >> 5, r32 = lane & 31;
  auto unpack = [](u32x2 w, float (&f)[4]) {
    f[0] = h2f<DT>((uint16_t)(w.x & 0xFFFFu));
    f[1] = h2f<DT>((uint16_t)(w.x >> 16));
    f[2] = h2f<DT>((uint16_t)(w.y & 0xFFFFu));
    f[3] = h2f<DT>((uint16_t)(w.y >> 16));
  };
  static_for<TN>([&](auto j) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int col = 32 * j + 8 * q + 4 * hi;
      float b[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      if constexpr ((E & EPI_BIAS) != 0) unpack(ld_u2(g.bias + nw + col), b);
      static_for<TM>([&](auto i) {
        const int row = 32 * i + r32;
        uint16_t h[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) h[c] = f2h<DT>(acc[i][j][4 * q + c] + b[c]);
        *reinterpret_cast<u32x2*>(lds + row * PITCH + col) =
            u32x2{h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16)};
      });
    }
  });
  const int c8 = 8 * (lane & 7);
  const int64_t ldc = g.ldc;
  uint16_t* C = g.C + (offC + mw * ldc + nw);
  uint16_t* pre = (E & EPI_GELU) ? g.pre + (mw * ldc + nw) : nullptr;
  const uint16_t* dact = (E & EPI_DACT) ? g.dact + (mw * ldc + nw) : nullptr;
  const uint16_t* res = (E & EPI_RESID) ? g.resid + (mw * g.ldr + nw) : nullptr;
  auto h8 = [](u32x4 w, uint16_t (&h)[8]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      h[2 * k] = (uint16_t)(w[k] & 0xFFFFu);
      h[2 * k + 1] = (uint16_t)(w[k] >> 16);
    }
  };
  auto p8 = [](const uint16_t (&h)[8]) {
    return u32x4{h[0] | ((uint32_t)h[1] << 16), h[2] | ((uint32_t)h[3] << 16),
                 h[4] | ((uint32_t)h[5] << 16), h[6] | ((uint32_t)h[7] << 16)};
  };
  int bad = 0;
#pragma unroll
  for (int t = 0; t < 4 * TM; ++t) {
    const int row = (lane >> 3) + 8 * t;
    const u32x2 w0 = *reinterpret_cast<const u32x2*>(lds + row * PITCH + c8);
    const u32x2 w1 = *reinterpret_cast<const u32x2*>(lds + row * PITCH + c8 + 4);
    uint16_t h[8];
    h8(u32x4{w0.x, w0.y, w1.x, w1.y}, h);
    const uint32_t off = (uint32_t)(row * ldc + c8);
    if constexpr ((E & EPI_GELU) != 0) {
      *reinterpret_cast<u32x4*>(pre + off) = p8(h);
#pragma unroll
      for (int c = 0; c < 8; ++c) h[c] = f2h<DT>(gelu_tanh(h2f<DT>(h[c])));
    }
    if constexpr ((E & EPI_DACT) != 0) {
      uint16_t da[8];
      h8(pf ? pf[t] : *reinterpret_cast<const u32x4*>(dact + off), da);
#pragma unroll
      for (int c = 0; c < 8; ++c) h[c] = f2h<DT>(h2f<DT>(h[c]) * gelu_tanh_grad(h2f<DT>(da[c])));
    }
    if constexpr ((E & EPI_RESID) != 0) {
      uint16_t rv[8];
      h8(pf ? pf[t] : *reinterpret_cast<const u32x4*>(res + (uint32_t)(row * g.ldr + c8)), rv);
#pragma unroll
      for (int c = 0; c < 8; ++c) h[c] = f2h<DT>(h2f<DT>(h[c]) + h2f<DT>(rv[c]));
    }
    const u32x4 o = p8(h);
    if constexpr ((E & EPI_COUNT) != 0)  // no branch inside the store loop
      bad += nonfinite2<DT>(o[0]) + nonfinite2<DT>(o[1]) + nonfinite2<DT>(o[2]) +
             nonfinite2<DT>(o[3]);
    *reinterpret_cast<u32x4*>(C + off) = o;
  }
  if constexpr ((E & EPI_COUNT) != 0) add_nonfinite(g.nonfinite, bad);
}

// Generic epilogue shared by the GEMM kernels: any tile, any operand
// alignment, split-K partials.  The wave's TM x TN accumulator blocks of
// 32 x 32 start at output row mw and column nw.  Two accumulator layouts:
//   TRANS = false (C = A B^T blocks): lane l holds column l % 32 and 4 runs of
//     4 consecutive rows; a 4x4 transpose across lane quads (two DPP
//     butterfly exchanges) turns each run into 4 consecutive columns of one row;
//   TRANS = true (the MFMA operands swapped, C^T blocks): lane l already holds
//     row l % 32, columns 8 q + 4 (l / 32) + (0..3) for q = 0..3.
// Either way bias / residual / activation inputs are read and outputs written
// 4 elements (8 bytes; 16 for float partials) at a time.
template <int DT, int TM, int TN, bool TRANS = false>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& g, const f32x16 (&acc)[TM][TN],
                                              int64_t mw, int64_t nw, int lane, int split,
                                              int64_t offC) {
  const int q4 = lane & 3;
  // run q of block (i, j): its 4 values, output row and first column
  auto run = [&](const f32x16& a, int i, int j, int q, float (&v)[4], int64_t& m, int64_t& n) {
#pragma unroll
    for (int c = 0; c < 4; ++c) v[c] = a[4 * q + c];
    if constexpr (TRANS) {
      m = mw + i * 32 + (lane & 31);
      n = nw + j * 32 + 8 * q + 4 * (lane >> 5);
    } else {
      quad_transpose(v, q4);
      m = mw + i * 32 + 8 * q + 4 * (lane >> 5) + q4;
      n = nw + j * 32 + 4 * ((lane & 31) >> 2);
    }
  };
  auto al8 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; };
  if (g.splits > 1) {
    float* W = g.ws + (int64_t)split * g.M * g.N;
    const bool v16 = g.N % 4 == 0 && (reinterpret_cast<uintptr_t>(W) & 15u) == 0;
    static_for<TM>([&](auto i) {
      static_for<TN>([&](auto j) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float v[4];
          int64_t m, n;
          run(acc[i][j], i, j, q, v, m, n);
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
  int bad = 0;
  static_for<TM>([&](auto i) {
    static_for<TN>([&](auto j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v[4];
        int64_t m, n;
        run(acc[i][j], i, j, q, v, m, n);
        const int nv = (int)max<int64_t>(0, min<int64_t>(4, g.N - n));
        if (m >= g.M || nv == 0) continue;
        const bool vec = v8 && nv == 4;
        uint16_t bias[4] = {0, 0, 0, 0}, h[4], da[4], res[4];
        if (g.bias) ld4(g.bias + n, vec, nv, bias);
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
#pragma unroll
        for (int c = 0; c < 4; ++c) bad += (c < nv && h_nonfinite<DT>(h[c])) ? 1 : 0;
        st4(C + m * g.ldc + n, vec, nv, h);
      }
    });
  });
  if (g.nonfinite) add_nonfinite(g.nonfinite, bad);
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
    const int64_t i0 = (uint32_t)z / (uint32_t)g.nb1, i1 = (uint32_t)z % (uint32_t)g.nb1;
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
  // copy the tile whose first element is at base into LDS at lds (both
  // wave-uniform; made explicitly scalar for the copy instruction)
  __device__ __forceinline__ void issue(const uint16_t* base, uint32_t lds, int wave) const {
    const uint64_t p = reinterpret_cast<uint64_t>(base);
    const uint64_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)p);
    const uint64_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(p >> 32));
    const void* sbase = reinterpret_cast<const void*>(lo | (hi << 32));
    const uint32_t slds = (uint32_t)__builtin_amdgcn_readfirstlane((int)lds);
#pragma unroll
    for (int q = 0; q < Q; ++q)
      dma16(sbase, off[q], slds + 1024u * (uint32_t)(wave + NWAVES * q));
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

// OCC: waves per SIMD the register budget is sized for.  E: the epilogue
// variant of whole tiles (EPI_GENERIC: always the generic epilogue).
// Sum of the 8 half values of an MFMA operand fragment, in a fixed pairwise order.
template <int DT>
__device__ __forceinline__ float frag_sum8(const uint4& f) {
  const uint32_t w[4] = {f.x, f.y, f.z, f.w};
  float p[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) p[k] = h2f<DT>((uint16_t)(w[k] & 0xFFFFu)) + h2f<DT>((uint16_t)(w[k] >> 16));
  return (p[0] + p[1]) + (p[2] + p[3]);
}

// DBS: also sum the rows of A over this workgroup's k range (the bias
// gradient of a weight-gradient product; see GemmArgs::db).  The waves of
// the left half of the tile (wn0 == 0) add up their A fragments as the MFMAs
// consume them: lane l holds 8 consecutive k of row l % 32 (k half l / 32),
// so per lane a running float32 sum per fragment, in k order, and at the end
// lane l plus lane l + 32 give the row's sum.  With split-K the work is
// spread over the C tile columns that share the A rows: the workgroup of
// column c sums the k tiles kt = c, c + C, ... of its split and writes
// partial dbp[row][split * C + c] (the reduction adds a row's C x splits
// partials with one wave, in a fixed order); without split-K column 0 sums
// every k tile and writes db itself.
template <int DT, int BM, int BN, int WM, int WN, int S, int OCC, bool AK, bool BKM, int E,
          bool DBS = false>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(OCC, OCC)))
void gemm_dma_kernel(GemmArgs g) {
  constexpr int NWAVES = (BM / WM) * (BN / WN);
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int A_BYTES = BM * 64 * 2, B_BYTES = BN * 64 * 2;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int L = (BM + BN) / 8 / NWAVES;  // copies per lane per stage
  static_assert((S - 2) * L <= 63, "vmcnt range");
  // LDS read instructions per k step (a k-major fragment is one 16-byte
  // read, an mn-major one two transposing 8-byte reads), per MFMA
  constexpr int kReads = TM * (AK ? 1 : 2) + TN * (BKM ? 1 : 2);
  constexpr int kReadsPerMfma = (kReads + TM * TN - 1) / (TM * TN);
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
    const int64_t i0 = (uint32_t)z / (uint32_t)g.nb1, i1 = (uint32_t)z % (uint32_t)g.nb1;
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
  // bias-gradient sums: tile columns sharing the A rows, this one's index,
  // and the next k tile this wave adds up (uniform over the wave)
  const int db_cols = g.splits > 1 ? (int)((g.N + BN - 1) / BN) : 1;
  const int db_col = g.splits > 1 ? (int)(n0 / BN) : 0;
  const bool dbw = DBS && wn0 == 0 && (g.splits > 1 || n0 == 0);
  int db_next = db_col;
  float dbs[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) dbs[i] = 0.0f;

  // A whole tile's GELU' or residual operand is loaded into registers before
  // the first copies (the oldest loads, so the first tile's wait covers
  // them): the epilogue then starts without a memory round trip.
  constexpr bool kPF = E != EPI_GENERIC && (E & (EPI_DACT | EPI_RESID)) != 0;
  const bool whole = E != EPI_GENERIC && g.full_epi && m0 + BM <= g.M && n0 + BN <= g.N;
  u32x4 pf[kPF ? 4 * TM : 1];
  if constexpr (kPF) {
    if (whole) {
      const int64_t ldp = (E & EPI_DACT) ? g.ldc : g.ldr;
      const uint16_t* src = ((E & EPI_DACT) ? g.dact : g.resid) + ((m0 + wm0) * ldp + n0 + wn0);
#pragma unroll
      for (int t = 0; t < 4 * TM; ++t)
        pf[t] = *reinterpret_cast<const u32x4*>(src + (uint32_t)(((lane >> 3) + 8 * t) * ldp + 8 * (lane & 7)));
    }
  }

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
    const bool db_now = dbw && kt == db_next;
    if (db_now) db_next += db_cols;
    // tile kt has landed once at most min(S - 2, nk - 1 - kt) later tiles are in flight
    const int later = min(S - 2, nk - 1 - kt);
    static_for<S - 1>([&](auto p) {
      if (later == p) wait_vmcnt<p * L>();
    });
    __syncthreads();
    if (kt + S - 1 < nk) issue(kt + S - 1);
    const uint32_t sa = lds0 + (uint32_t)((kt % S) * STAGE), sb = sa + A_BYTES;
    // fragments double-buffered over the four k steps of 16: the LDS reads
    // of step kk + 1 are issued ahead of the MFMAs of step kk.  Products
    // with an mn-major operand (dX, dW: transposing reads, two per
    // fragment) interleave one MFMA with its share of those reads
    // (scheduling group barriers: dW +8-17% on the ViT-B layers); the
    // forward products (both operands k-major) issue the step's reads as a
    // group before its MFMAs (scheduling barriers), which measured 1-2%
    // faster for them.
    constexpr bool kInterleave = !(AK && BKM);
    uint4 af[2][TM], bf[2][TN];
    static_for<TM>([&](auto i) { af[0][i] = fa.template read<i, 0>(sa); });
    static_for<TN>([&](auto j) { bf[0][j] = fb.template read<j, 0>(sb); });
    static_for<4>([&](auto kk) {
      constexpr int cur = kk & 1, nxt = cur ^ 1;
      if constexpr (kk + 1 < 4) {
        static_for<TM>([&](auto i) { af[nxt][i] = fa.template read<i, kk + 1>(sa); });
        static_for<TN>([&](auto j) { bf[nxt][j] = fb.template read<j, kk + 1>(sb); });
      }
      if constexpr (!kInterleave) __builtin_amdgcn_sched_barrier(0);
      static_for<TM>([&](auto i) {
        static_for<TN>([&](auto j) { acc[i][j] = mfma32<DT>(bf[cur][j], af[cur][i], acc[i][j]); });
      });
      if constexpr (DBS) {
        if (db_now) static_for<TM>([&](auto i) { dbs[i] += frag_sum8<DT>(af[cur][i]); });
      }
      if constexpr (!kInterleave) {
        __builtin_amdgcn_sched_barrier(0);
      } else if constexpr (kk + 1 < 4) {
        static_for<TM * TN>([&](auto) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);              // one MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, kReadsPerMfma, 0);  // its LDS reads
        });
      }
    });
  }
  if constexpr (DBS) {
    if (dbw) {
      int bad = 0;
      static_for<TM>([&](auto i) {
        const float other = __shfl_xor(dbs[i], 32);  // the row's other 8 k of every step
        const int64_t row = m0 + wm0 + 32 * i + lane;
        if (lane < 32 && row < g.M) {
          const float v = dbs[i] + other;
          if (g.splits > 1) {
            g.dbp[row * ((int64_t)g.splits * db_cols) + (int64_t)split * db_cols + db_col] = v;
          } else {
            const uint16_t h = f2h<DT>(v);
            g.db[row] = h;
            bad += h_nonfinite<DT>(h) ? 1 : 0;
          }
        }
      });
      if (g.nonfinite) add_nonfinite(g.nonfinite, bad);
    }
  }
  // the accumulators hold C^T blocks (the MFMA operands are swapped above)
  if constexpr (E != EPI_GENERIC) {
    if (whole) {  // uniform over the workgroup
      __syncthreads();  // every wave is done reading the stage buffers
      gemm_epilogue_lds<DT, TM, TN, E>(g, acc, m0 + wm0, n0 + wn0, lane, offC,
                                       reinterpret_cast<uint16_t*>(smem) + wave * (WM * 68),
                                       kPF ? pf : nullptr);
      return;
    }
  }
  gemm_epilogue<DT, TM, TN, true>(g, acc, m0 + wm0, n0 + wn0, lane, split, offC);
}

// Persistent form of the direct-to-LDS kernel for one product without
// split-K or batching: a grid of (workgroups per CU) x 256 workgroups walks
// the tiles in strides of the grid, so every workgroup stays on one XCD and
// its tiles keep the XCD-contiguous order of tile_origin.  Between two tiles
// the next tile's first k tile is copied into stage 0 while the current
// tile's epilogue stages its output through the LDS above stage 0, so the
// copy's latency overlaps the epilogue instead of opening the next tile.
template <int DT, int BM, int BN, int WM, int WN, int OCC, bool AK, bool BKM, int E>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64)
__attribute__((amdgpu_waves_per_eu(OCC, OCC)))
void gemm_dma_persistent_kernel(GemmArgs g) {
  constexpr int NWAVES = (BM / WM) * (BN / WN);
  constexpr int TM = WM / 32, TN = WN / 32;
  constexpr int A_BYTES = BM * 64 * 2, B_BYTES = BN * 64 * 2;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int EPI = NWAVES * WM * 68 * 2;  // epilogue staging, from the start of stage 1
  constexpr int SMEM = STAGE + (STAGE > EPI ? STAGE : EPI);
  __shared__ __attribute__((aligned(1024))) uint8_t smem[SMEM];
  const uint32_t lds0 = lds_u32(smem);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm0 = (wave / (BN / WN)) * WM;
  const int wn0 = (wave % (BN / WN)) * WN;
  const uint32_t ntiles = (uint32_t)(((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN));
  const int nk = (int)(g.K / 64);

  FragReader<BM, AK, TM> fa;
  FragReader<BN, BKM, TN> fb;
  fa.init(wm0, lane);
  fb.init(wn0, lane);
  DmaOperand<BM, AK, NWAVES> da;
  DmaOperand<BN, BKM, NWAVES> db;
  int64_t m0, n0;
  const uint16_t* Ab;
  const uint16_t* Bb;
  auto setup = [&](uint32_t t) {
    tile_origin_of<BM, BN>(t, ntiles, g.M, g.N, m0, n0);
    Ab = g.A + (AK ? m0 * g.lda : m0);
    Bb = g.B + (BKM ? n0 * g.ldb : n0);
    da.init(g.lda, (int)min<int64_t>(BM, g.M - m0), wave, lane);
    db.init(g.ldb, (int)min<int64_t>(BN, g.N - n0), wave, lane);
  };
  auto issue = [&](int kt) {
    const uint32_t st = lds0 + (uint32_t)((kt & 1) * STAGE);
    da.issue(reinterpret_cast<const uint16_t*>(reinterpret_cast<const uint8_t*>(Ab) + kt * da.step), st, wave);
    db.issue(reinterpret_cast<const uint16_t*>(reinterpret_cast<const uint8_t*>(Bb) + kt * db.step),
             st + A_BYTES, wave);
  };

  uint32_t t = blockIdx.x;
  if (t >= ntiles) return;  // uniform over the workgroup
  setup(t);
  issue(0);
  for (;;) {
    f32x16 acc[TM][TN];
    static_for<TM>([&](auto i) {
      static_for<TN>([&](auto j) {
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;
      });
    });
    for (int kt = 0; kt < nk; ++kt) {
      wait_vmcnt<0>();  // k tile kt (and everything issued before it) has landed
      __syncthreads();
      if (kt + 1 < nk) issue(kt + 1);
      const uint32_t sa = lds0 + (uint32_t)((kt & 1) * STAGE), sb = sa + A_BYTES;
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
          static_for<TN>([&](auto j) { acc[i][j] = mfma32<DT>(bf[cur][j], af[cur][i], acc[i][j]); });
        });
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    const int64_t me = m0, ne = n0;
    const uint32_t tn = t + gridDim.x;
    __syncthreads();  // every wave is done reading the stage buffers
    if (tn < ntiles) {
      setup(tn);
      issue(0);  // lands in stage 0 while this tile's epilogue runs above it
    }
    if (E != EPI_GENERIC && g.full_epi && me + BM <= g.M && ne + BN <= g.N) {
      if constexpr (E != EPI_GENERIC)
        gemm_epilogue_lds<DT, TM, TN, E>(g, acc, me + wm0, ne + wn0, lane, 0,
                                         reinterpret_cast<uint16_t*>(smem + STAGE) + wave * (WM * 68));
    } else {
      gemm_epilogue<DT, TM, TN, true>(g, acc, me + wm0, ne + wn0, lane, 0, 0);
    }
    if (tn >= ntiles) break;
    t = tn;
    __syncthreads();  // the epilogue's LDS (stage 1) is free for the next copies
  }
}

// Sum of split-K partials in split order, one rounding: C = half(sum_s W[s]),
// one thread per output in the first ceil(MN / 256) workgroups.  The
// workgroups after them reduce the bias-gradient partials dbp[row][p],
// p < dbparts, one wave per row (nrows rows; 0: none): lane l adds p = l,
// l + 64, ... in order, then the fixed wave tree of wave_sum; db = half of
// that.  Non-finite results are added to *nonfinite when it is set.
// VEC (MN a multiple of 4, ws 16-byte and C 8-byte aligned): each thread
// reduces 4 consecutive outputs with 16-byte loads and one 8-byte store, each
// output summed in the same split order as the scalar form (the same bits):
// 3072 x 768 from 2 splits alone 6.3 -> 5.4 us, 768 x 768 from 8 splits 6.2 -> 4.9.
template <int DT, bool VEC>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ ws, int splits,
                                                            int64_t MN, uint16_t* __restrict__ C,
                                                            int32_t* __restrict__ nonfinite,
                                                            const float* __restrict__ dbp, int dbparts,
                                                            int64_t nrows, uint16_t* __restrict__ db) {
  constexpr int PER = VEC ? 4 : 1;
  const int64_t mn_blocks = (MN + 256 * PER - 1) / (256 * PER);
  if ((int64_t)blockIdx.x < mn_blocks) {
    const int64_t i = ((int64_t)blockIdx.x * 256 + threadIdx.x) * PER;
    if (i >= MN) return;
    if constexpr (VEC) {
      f32x4 s = *reinterpret_cast<const f32x4*>(ws + i);
      for (int k = 1; k < splits; ++k) {
        const f32x4 t = *reinterpret_cast<const f32x4*>(ws + (int64_t)k * MN + i);
#pragma unroll
        for (int e = 0; e < 4; ++e) s[e] += t[e];
      }
      uint16_t h[4];
      int bad = 0;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        h[e] = f2h<DT>(s[e]);
        bad += h_nonfinite<DT>(h[e]) ? 1 : 0;
      }
      *reinterpret_cast<uint2*>(C + i) =
          make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
      if (nonfinite) add_nonfinite(nonfinite, bad);
    } else {
      float s = ws[i];
      for (int k = 1; k < splits; ++k) s += ws[(int64_t)k * MN + i];
      const uint16_t h = f2h<DT>(s);
      C[i] = h;
      if (nonfinite) add_nonfinite(nonfinite, h_nonfinite<DT>(h) ? 1 : 0);
    }
    return;
  }
  const int64_t row = ((int64_t)blockIdx.x - mn_blocks) * 4 + (threadIdx.x >> 6);
  if (row >= nrows) return;  // uniform over the wave
  const int lane = threadIdx.x & 63;
  const float* p = dbp + row * dbparts;
  float s = 0.0f;
  for (int k = lane; k < dbparts; k += 64) s += p[k];
  s = wave_sum(s);
  if (lane == 0) {
    const uint16_t h = f2h<DT>(s);
    db[row] = h;
    if (nonfinite) add_nonfinite(nonfinite, h_nonfinite<DT>(h) ? 1 : 0);
  }
}

// launch shape of splitk_reduce_kernel: MN outputs and nrows bias rows
inline unsigned splitk_reduce_blocks(int64_t MN, int64_t nrows, bool vec) {
  const int64_t per = vec ? 1024 : 256;
  return (unsigned)((MN + per - 1) / per + (nrows + 3) / 4);
}

inline bool splitk_reduce_vec(const float* ws, int64_t MN, const uint16_t* C) {
  return MN % 4 == 0 && (reinterpret_cast<uintptr_t>(ws) & 15u) == 0 &&
         (reinterpret_cast<uintptr_t>(C) & 7u) == 0;
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

// Epilogue mask of a call, or EPI_GENERIC when it has no compiled variant
static int epilogue_mask(const GemmArgs& g) {
  if (g.splits > 1) return EPI_GENERIC;
  return (g.bias ? EPI_BIAS : 0) | (g.act == MPX_ACT_GELU_TANH ? EPI_GELU : 0) |
         (g.dact ? EPI_DACT : 0) | (g.resid ? EPI_RESID : 0);
}

// Whole-tile epilogue preconditions that do not depend on the tile: output,
// pre-activation, GELU' and residual operands 16-byte aligned with row
// strides a multiple of 8, the bias 8-byte aligned, and the per-lane 32-bit
// offsets in range.
static bool full_epilogue_ok(const GemmArgs& g, int bm) {
  auto al8 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 7u) == 0; };
  auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
  const bool strides = g.sC0 % 8 == 0 && g.sC1 % 8 == 0;
  return g.splits == 1 && strides && g.ldc % 8 == 0 && al16(g.C) && (!g.bias || al8(g.bias)) &&
         (!g.pre || al16(g.pre)) && (!g.dact || al16(g.dact)) &&
         (!g.resid || (al16(g.resid) && g.ldr % 8 == 0)) && g.ldc * bm < ((int64_t)1 << 30) &&
         g.ldr * bm < ((int64_t)1 << 30);
}

template <int DT, int BM, int BN, int WM, int WN, int S, int OCC>
static hipError_t launch_dma(GemmArgs g, bool ak, bool bk, int64_t nbatch, hipStream_t s) {
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  dim3 grid((unsigned)tiles, (unsigned)(g.splits > 1 ? g.splits : nbatch));
  g.full_epi = full_epilogue_ok(g, BM) ? 1 : 0;
  // a call that counts non-finite outputs (weight gradients: both operands
  // mn-major, no epilogue operation) has a whole-tile variant of its own;
  // any other counting call takes the generic epilogue
  const int e = g.full_epi ? epilogue_mask(g) | (g.nonfinite ? EPI_COUNT : 0) : EPI_GENERIC;
#define MPX_D(AKv, BKv, Ev) gemm_dma_kernel<DT, BM, BN, WM, WN, S, OCC, AKv, BKv, Ev><<<grid, NT, 0, s>>>(g)
#define MPX_DB(Ev) gemm_dma_kernel<DT, BM, BN, WM, WN, S, OCC, false, false, Ev, true><<<grid, NT, 0, s>>>(g)
  if constexpr (BM == 64) {
    // 64 x 128 tiles (outputs too small to fill the CUs with 128 x 128): the
    // A operand must be k-major (dma_ok rejects the rest)
    if (!ak) return hipErrorInvalidValue;
    if (bk) {
      switch (e) {
        case 0: MPX_D(true, true, 0); break;
        case EPI_BIAS: MPX_D(true, true, EPI_BIAS); break;
        case EPI_BIAS | EPI_GELU: MPX_D(true, true, EPI_BIAS | EPI_GELU); break;
        case EPI_BIAS | EPI_RESID: MPX_D(true, true, EPI_BIAS | EPI_RESID); break;
        default: MPX_D(true, true, EPI_GENERIC);
      }
    } else {
      switch (e) {
        case 0: MPX_D(true, false, 0); break;
        case EPI_DACT: MPX_D(true, false, EPI_DACT); break;
        default: MPX_D(true, false, EPI_GENERIC);
      }
    }
  } else if constexpr (BM == 128 && BN == 128 && S == 2) {
    // the configuration the dispatcher picks: whole tiles get the
    // specialised epilogue of each call pattern of the training step
    if (ak && bk) {
      switch (e) {
        case 0: MPX_D(true, true, 0); break;
        case EPI_BIAS: MPX_D(true, true, EPI_BIAS); break;
        case EPI_BIAS | EPI_GELU: MPX_D(true, true, EPI_BIAS | EPI_GELU); break;
        case EPI_BIAS | EPI_RESID: MPX_D(true, true, EPI_BIAS | EPI_RESID); break;
        default: MPX_D(true, true, EPI_GENERIC);
      }
    } else if (ak && !bk) {
      switch (e) {
        case 0: MPX_D(true, false, 0); break;
        case EPI_DACT: MPX_D(true, false, EPI_DACT); break;
        default: MPX_D(true, false, EPI_GENERIC);
      }
    } else if (!ak && bk) {
      if (e == 0) MPX_D(false, true, 0);
      else MPX_D(false, true, EPI_GENERIC);
    } else if (g.db) {  // weight gradient with the bias gradient summed alongside
      if (e == 0) MPX_DB(0);
      else if (e == EPI_COUNT) MPX_DB(EPI_COUNT);
      else MPX_DB(EPI_GENERIC);
    } else {
      if (e == 0) MPX_D(false, false, 0);
      else if (e == EPI_COUNT) MPX_D(false, false, EPI_COUNT);
      else MPX_D(false, false, EPI_GENERIC);
    }
  } else {
    if (ak && bk) MPX_D(true, true, EPI_GENERIC);
    else if (ak && !bk) MPX_D(true, false, EPI_GENERIC);
    else if (!ak && bk) MPX_D(false, true, EPI_GENERIC);
    else MPX_D(false, false, EPI_GENERIC);
  }
#undef MPX_D
#undef MPX_DB
  return hipGetLastError();
}

template <int DT, int BM, int BN, int WM, int WN, int OCC>
static hipError_t launch_persistent(GemmArgs g, bool ak, bool bk, hipStream_t s) {
  constexpr int NT = (BM / WM) * (BN / WN) * 64;
  const int64_t tiles = ((g.M + BM - 1) / BM) * ((g.N + BN - 1) / BN);
  const unsigned grid = (unsigned)std::min<int64_t>(tiles, 256 * OCC);
  g.full_epi = full_epilogue_ok(g, BM) ? 1 : 0;
  // a call that counts non-finite outputs takes the generic epilogue
  const int e = g.full_epi && !g.nonfinite ? epilogue_mask(g) : EPI_GENERIC;
  if (!ak) return hipErrorInvalidValue;
#define MPX_P(BKv, Ev) gemm_dma_persistent_kernel<DT, BM, BN, WM, WN, OCC, true, BKv, Ev><<<grid, NT, 0, s>>>(g)
  if (bk) {
    switch (e) {
      case 0: MPX_P(true, 0); break;
      case EPI_BIAS: MPX_P(true, EPI_BIAS); break;
      case EPI_BIAS | EPI_GELU: MPX_P(true, EPI_BIAS | EPI_GELU); break;
      case EPI_BIAS | EPI_RESID: MPX_P(true, EPI_BIAS | EPI_RESID); break;
      default: MPX_P(true, EPI_GENERIC);
    }
  } else {
    switch (e) {
      case 0: MPX_P(false, 0); break;
      case EPI_DACT: MPX_P(false, EPI_DACT); break;
      default: MPX_P(false, EPI_GENERIC);
    }
  }
#undef MPX_P
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
//   8  skinny products: one wave (K > 32) or one lane (K <= 32) per output
//   9  direct-to-LDS 64 x 128, 4 waves of 32 x 64, 2 stages, three workgroups
//      per CU (A k-major only)
//  10  configuration 7, persistent (A k-major, no split-K or batch)
//  11  configuration 9, persistent (A k-major, no split-K or batch)
extern int g_forced_config;  // defined in gemm.hip

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
// variant at full occupancy, forward and backward; the register-staged
// kernels serve operands the copies cannot take.  What remains is tile
// quantisation: 128 x 128 tiles run 512 at a time (2 per CU), 64 x 128
// tiles 768 at a time (3 per CU) with half the work each, so an output
// whose 128 x 128 tile count sits just above a multiple of 512 runs a
// nearly empty last round.  Cost of a configuration = rounds x
// (workgroups per CU) x (tile area), with 5% added for the smaller tiles'
// lower MFMA efficiency; the 64 x 128 tiles are taken when they save more
// than 3% (on the ViT layer shapes this picks the faster of the two in
// every measured case, e.g. 12608 x 768 outputs: 22 us instead of 29).
static bool small_ok(const GemmArgs& g, int64_t nbatch);

static bool prefer_64x128(const GemmArgs& g, int64_t nbatch) {
  const int64_t nb = g.splits > 1 ? g.splits : nbatch;
  const int64_t tn = (g.N + 127) / 128;
  const int64_t t128 = ((g.M + 127) / 128) * tn * nb, t64 = ((g.M + 63) / 64) * tn * nb;
  const double cost128 = (double)((t128 + 511) / 512) * 2.0 * 2.0;
  const double cost64 = (double)((t64 + 767) / 768) * 3.0 * 1.05;
  return cost64 < 0.97 * cost128;
}

static int choose_config(const GemmArgs& g, bool vec, bool ak, bool bk, int64_t nbatch) {
  const bool dma = dma_ok(g, vec, ak, bk);
  const bool small = small_ok(g, nbatch);
  const int f = g_forced_config;
  if (f == 8 && small) return 8;
  if (f == 9 && dma && ak) return 9;
  if ((f == 10 || f == 11) && dma && ak) return g.splits == 1 && nbatch == 1 ? f : (f == 10 ? 7 : 9);
  if (f >= 3 && f <= 7 && dma) return f;
  if (f == 1 || (f == 2 && vec)) return f;
  if (small && (g.M <= 32 || g.N <= 32 || g.K <= 32)) return 8;
  if (g.M <= 64 || g.N <= 64) return 1;
  // (the persistent forms 10 and 11 are 1-5% faster on a product alone, but
  // they hold every workgroup slot of the chip until they end, so the
  // weight-gradient stream of the training step cannot interleave: the ViT
  // steps ran 2-4% slower with them)
  if (dma) return ak && prefer_64x128(g, nbatch) ? 9 : 7;
  return vec ? 2 : 0;
}

// ----------------------------------------------------------- skinny GEMMs --
//
// Products with a dimension of 32 or less (a classifier head: 10 outputs, or
// a reduction over 10 classes) waste most of a 32x32 MFMA tile and run a
// long dependent k loop on very few workgroups.  Here every output element
// gets its own wave when K > 32 (lane l sums k = l, l + 64, ... in float32,
// then a fixed butterfly adds the 64 lane sums) or its own lane when K <= 32
// (a plain k loop).  Both orders are fixed, so results are reproducible.
// Epilogue: bias and residual, h = half(acc + bias[n]), then half(h + R[m,n]).
template <int DT, bool WAVE>
__global__ __launch_bounds__(256) void gemm_small_kernel(GemmArgs g, bool ak, bool bk) {
  const int64_t MN = g.M * g.N;
  const int64_t idx = WAVE ? ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6))
                           : ((int64_t)blockIdx.x * 256 + threadIdx.x);
  if (idx >= MN) return;
  const int64_t m = idx / g.N, n = idx % g.N;
  // opA(m,k) = A[m*lda + k] (k-major) or A[k*lda + m]; opB(n,k) likewise
  const int64_t sam = ak ? g.lda : 1, sak = ak ? 1 : g.lda;
  const int64_t sbn = bk ? g.ldb : 1, sbk = bk ? 1 : g.ldb;
  const uint16_t* a = g.A + m * sam;
  const uint16_t* b = g.B + n * sbn;
  float acc = 0.0f;
  if constexpr (WAVE) {
    const int lane = threadIdx.x & 63;
    for (int64_t k = lane; k < g.K; k += 64) acc += h2f<DT>(a[k * sak]) * h2f<DT>(b[k * sbk]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o);
    if (lane != 0) return;
  } else {
    for (int64_t k = 0; k < g.K; ++k) acc += h2f<DT>(a[k * sak]) * h2f<DT>(b[k * sbk]);
  }
  const float bias = g.bias ? h2f<DT>(g.bias[n]) : 0.0f;
  uint16_t h = f2h<DT>(acc + bias);
  if (g.resid) h = f2h<DT>(h2f<DT>(h) + h2f<DT>(g.resid[m * g.ldr + n]));
  g.C[m * g.ldc + n] = h;
  if (g.nonfinite) add_nonfinite(g.nonfinite, h_nonfinite<DT>(h) ? 1 : 0);
}

static bool small_ok(const GemmArgs& g, int64_t nbatch) {
  return nbatch == 1 && g.splits == 1 && !g.pre && !g.dact && g.act == MPX_ACT_NONE &&
         g.M * g.N <= ((int64_t)1 << 22);
}

template <int DT>
static hipError_t launch_small(const GemmArgs& g, bool ak, bool bk, hipStream_t s) {
  const int64_t MN = g.M * g.N;
  if (g.K > 32)
    gemm_small_kernel<DT, true><<<(unsigned)((MN + 3) / 4), 256, 0, s>>>(g, ak, bk);
  else
    gemm_small_kernel<DT, false><<<(unsigned)((MN + 255) / 256), 256, 0, s>>>(g, ak, bk);
  return hipGetLastError();
}

// ak: A is k-major; bk: B is k-major.  A call with g.db set (a weight
// gradient whose bias gradient is wanted) gets it from the GEMM when the
// chosen kernel can sum it (the two-stage 128 x 128 direct-to-LDS kernel
// with both operands mn-major); *db_fused tells the caller whether it did,
// and otherwise the caller computes the column sums itself.
template <int DT>
static hipError_t run_gemm(GemmArgs g, bool ak, bool bk, int64_t nbatch, hipStream_t s,
                           bool* db_fused) {
  const bool vec = aligned_vec(g.A, g.lda, g.sA0, g.sA1) && aligned_vec(g.B, g.ldb, g.sB0, g.sB1);
  const int cfg = choose_config(g, vec, ak, bk, nbatch);
  const bool fuse = g.db && cfg == 7 && !ak && !bk && nbatch == 1 && (g.splits == 1 || g.dbp);
  if (db_fused) *db_fused = fuse;
  if (!fuse) {
    g.db = nullptr;
    g.dbp = nullptr;
  }
  switch (cfg) {
    case 8: return launch_small<DT>(g, ak, bk, s);
    case 1: return launch_cfg<DT, 64, 64, 32, 32>(g, ak, bk, vec, nbatch, s);
    case 2: return launch_cfg<DT, 128, 128, 64, 32, 64, 4>(g, ak, bk, vec, nbatch, s);
    case 3: return launch_dma<DT, 256, 256, 128, 128, 2, 1>(g, ak, bk, nbatch, s);
    case 4: return launch_dma<DT, 256, 128, 128, 64, 3, 1>(g, ak, bk, nbatch, s);
    case 5: return launch_dma<DT, 128, 256, 64, 128, 3, 1>(g, ak, bk, nbatch, s);
    case 6: return launch_dma<DT, 128, 128, 64, 64, 4, 1>(g, ak, bk, nbatch, s);
    case 7: return launch_dma<DT, 128, 128, 64, 64, 2, 2>(g, ak, bk, nbatch, s);
    case 9: return launch_dma<DT, 64, 128, 32, 64, 2, 3>(g, ak, bk, nbatch, s);
    case 10: return launch_persistent<DT, 128, 128, 64, 64, 2>(g, ak, bk, s);
    case 11: return launch_persistent<DT, 64, 128, 32, 64, 3>(g, ak, bk, s);
    default:  // unaligned operands (rare: odd leading dimensions)
      return launch_cfg<DT, 128, 128, 64, 64>(g, ak, bk, vec, nbatch, s);
  }
}

hipError_t run_gemm_f16(const GemmArgs& g, bool ak, bool bk, int64_t nbatch, hipStream_t s,
                        bool* db_fused = nullptr);
hipError_t run_gemm_bf16(const GemmArgs& g, bool ak, bool bk, int64_t nbatch, hipStream_t s,
                         bool* db_fused = nullptr);

}  // namespace mpx
