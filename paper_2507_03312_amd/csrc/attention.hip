// Fused multi-head self-attention core for short sequences (T <= 256, head
// dimension 64), forward and backward, with the half-precision policy of
// MPX (§2.1: products in half with float32 accumulation; §3.2: the softmax
// and its backward run in full precision as a force_full_precision island):
//
//   forward   S = half(Q K^T),  P = half(softmax(scale S)) in float32,
//             O = half(P V)                                (scale = 1/sqrt(hd))
//   backward  dP = half(dO V^T),  dV = half(P^T dO),
//             dS = half(scale P (dP - sum_k dP P)) in float32,
//             dQ = half(dS K),  dK = half(dS^T Q)
//
// One workgroup per (batch, head) with one wave per 32-row block of the
// sequence (up to 8 waves).  Each wave computes the transposed score block S^T = K Q^T for
// its 32 queries, so that a lane holds one query (column) and half of every
// key block (rows): the softmax reductions over keys are lane-local plus one
// exchange with the lane 32 apart.  The probabilities then feed the P V
// product straight from registers: a v_permlane32_swap turns the
// accumulator layout into the MFMA B-operand layout (8 consecutive keys per
// lane).  V, and in the backward K, Q, dO, P and dS, are staged in LDS and
// read as transposed MFMA operands with ds_read_b64_tr_b16.  Up to T = 128
// the backward keeps the [T, T] probability and dS blocks in LDS; beyond,
// they no longer fit next to K, V, Q and dO, and each wave keeps its own
// query block's P and dS in registers and hands them to the others through
// a [32, T] slab in LDS, one query block at a time (attn_bwd_fused_kernel).
//
// Layouts: qkv [B*T, 3*H*64] (Q | K | V, head h at columns h*64 of each
// third), O and dO [B*T, H*64], dqkv like qkv, P [B*H, T, ldP] with
// ldP = T rounded up to 8 (columns T..ldP-1 hold 0).
#include <hip/hip_runtime.h>

#include <cmath>

#include "common.h"
#include "mfma.h"

namespace mpx {
namespace {

constexpr int HD = 64;               // head dimension
constexpr int PD = HD + 8;           // LDS row pitch (halves) of [row][d] arrays:
                                     // 144 B, so the 4 consecutive rows of a
                                     // transposed read fall in distinct banks

// MFMA operand fragment (32 rows of m or n, 16 k) from an LDS array stored
// [k][mn] with mn contiguous and a pitch of `pitch` halves: two
// ds_read_b64_tr_b16, each giving 4 consecutive k of one mn per lane.
__device__ __forceinline__ uint4 frag_tr(uint32_t base, int pitch, int k0, int mn0, int lane) {
  const int g = lane >> 4, e = (lane >> 2) & 3, t = lane & 3;
  const int kr = k0 + 8 * (g >> 1) + e;
  const int mn = mn0 + 16 * (g & 1) + 4 * t;
  const uint2 lo = lds_tr_b64(base + (uint32_t)((kr * pitch + mn) * 2));
  const uint2 hi = lds_tr_b64(base + (uint32_t)(((kr + 4) * pitch + mn) * 2));
  return make_uint4(lo.x, lo.y, hi.x, hi.y);
}

// The rows of a [T, 64] head slice (row stride ld) staged into LDS
// [PER * nthreads / 8][PD] in two steps, PER 16-byte chunks per thread:
// load() puts every global load of the thread in flight, store() writes
// them.  No branches: rows past T load row T - 1 and are written as zeros.
// A loop that stores each chunk before loading the next waits one memory
// latency per chunk.
template <int PER>
struct RowStage {
  u32x4 v[PER];
  __device__ __forceinline__ void load_clamped(const uint16_t* src, int64_t ld, int T, int tid,
                                               int nthreads) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * nthreads;
      v[i] = *reinterpret_cast<const u32x4*>(src + min(c >> 3, T - 1) * ld + (c & 7) * 8);
    }
  }
  __device__ __forceinline__ void store_clamped(uint16_t* lds, int T, int tid, int nthreads) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * nthreads;
      asm volatile("" : "+v"(v[i]));  // keeps the load unconditional
      if ((c >> 3) >= T) v[i] = u32x4{0u, 0u, 0u, 0u};
      *reinterpret_cast<u32x4*>(lds + (c >> 3) * PD + (c & 7) * 8) = v[i];
    }
  }
};

// Packs 4 halves.
__device__ __forceinline__ u32x2 pack4(uint16_t a, uint16_t b, uint16_t c, uint16_t d) {
  return u32x2{a | ((uint32_t)b << 16), c | ((uint32_t)d << 16)};
}

// Two halves packed in a dword <-> float32 (exact widening; narrowing
// rounds to nearest even, as f2h).
typedef float f32x2v __attribute__((ext_vector_type(2)));
template <int DT> __device__ __forceinline__ void unpack2(uint32_t v, float& a, float& b);
template <> __device__ __forceinline__ void unpack2<MPX_BF16>(uint32_t v, float& a, float& b) {
  a = __builtin_bit_cast(float, v << 16);
  b = __builtin_bit_cast(float, v & 0xFFFF0000u);
}
template <> __device__ __forceinline__ void unpack2<MPX_F16>(uint32_t v, float& a, float& b) {
  a = (float)__builtin_bit_cast(_Float16, (uint16_t)(v & 0xFFFFu));
  b = (float)__builtin_bit_cast(_Float16, (uint16_t)(v >> 16));
}
template <int DT> __device__ __forceinline__ uint32_t pack2(float a, float b);
template <> __device__ __forceinline__ uint32_t pack2<MPX_BF16>(float a, float b) {
  typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2v){a, b}, bf16x2v));
}
template <> __device__ __forceinline__ uint32_t pack2<MPX_F16>(float a, float b) {
  // two scalar conversions: they keep half subnormals, as f2h does
  return (uint32_t)f2h<MPX_F16>(a) | ((uint32_t)f2h<MPX_F16>(b) << 16);
}

// A 32 x 32 accumulator block whose rows run along a stored row (lane =
// column n, rows 8 gq + 4 hi + 0..3 in entries 4 gq + 0..3), rounded to
// half and stored as that row's 32 consecutive elements: one exchange with
// the lane 32 apart gives each lane 8 consecutive ones, so the row goes out
// in two 16-byte stores per lane.  row must be 16-byte aligned.
template <int DT>
__device__ __forceinline__ void store_acc_row32(const f32x16& o, uint16_t* row, int hi) {
#pragma unroll
  for (int m = 0; m < 2; ++m) {
    u32x2 x = pack4(f2h<DT>(o[8 * m]), f2h<DT>(o[8 * m + 1]), f2h<DT>(o[8 * m + 2]), f2h<DT>(o[8 * m + 3]));
    u32x2 y = pack4(f2h<DT>(o[8 * m + 4]), f2h<DT>(o[8 * m + 5]), f2h<DT>(o[8 * m + 6]),
                    f2h<DT>(o[8 * m + 7]));
    half_swap(x, y);
    *reinterpret_cast<u32x4*>(row + 16 * m + 8 * hi) = u32x4{x.x, x.y, y.x, y.y};
  }
}

// B operand (n = query, 16 keys starting at 16 ks) from the packed
// probabilities of the lane's query: R[j][gq] holds keys 32 j + 8 gq + 4 hi +
// (0..3).  Half 0 needs keys 8 g' + 0..7 with g' = 2s, half 1 with g' = 2s+1;
// swapping the upper half of group 2s with the lower half of group 2s+1
// leaves the first 4 keys in x and the next 4 in y on every lane.
template <int NB>
__device__ __forceinline__ uint4 keys_operand(const u32x2 (&R)[NB][4], int ks) {
  u32x2 x = R[ks / 2][2 * (ks % 2)], y = R[ks / 2][2 * (ks % 2) + 1];
  half_swap(x, y);
  return make_uint4(x.x, x.y, y.x, y.y);
}

// ----------------------------------------------------------------- forward --

// Up to 4 key blocks (T <= 128): the single-pass form, a lane holding its
// query's whole score row in registers (K read straight from global memory).
// It measured faster there than the two-pass kernel below (13.8-15.1 vs
// 16.6-17.4 us at 65 tokens, batch 128, 6 heads).
template <int DT, int NB>
__global__ __launch_bounds__(NB * 64) void attn_fwd_rows_kernel(const uint16_t* __restrict__ qkv,
                                                           uint16_t* __restrict__ O,
                                                           uint16_t* __restrict__ P, int T, int H,
                                                           int ldP, float scale) {
  constexpr int TK = 32 * NB;
  __shared__ __attribute__((aligned(16))) uint16_t sV[TK * PD];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, hi = lane >> 5;
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int dm = H * HD;
  const int64_t ld = 3 * (int64_t)dm;
  const uint16_t* Q = qkv + (int64_t)b * T * ld + h * HD;
  const uint16_t* K = Q + dm;
  const uint16_t* V = Q + 2 * dm;

  RowStage<4> vst;  // V: 32 NB rows over 64 NB threads
  vst.load_clamped(V, ld, T, tid, NB * 64);

  // S^T blocks: rows = keys of block j, columns = the wave's 32 queries
  const int q = 32 * w + (lane & 31);
  const int qc = min(q, T - 1);
  uint4 qf[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) qf[kk] = ld_u4(Q + qc * ld + 16 * kk + 8 * hi);
  f32x16 s[NB];
  static_for<NB>([&](auto j) {
    const int key = min(32 * j + (lane & 31), T - 1);
    f32x16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) acc = mfma32<DT>(ld_u4(K + key * ld + 16 * kk + 8 * hi), qf[kk], acc);
    s[j] = acc;
  });

  // softmax over the keys of query q (float32; S rounded to half first)
  // (blocks below nfull have no key past T: no masks there)
  const int nfull = T / 32;
  float mx = -INFINITY;
  static_for<NB>([&](auto j) {
#pragma unroll
    for (int e = 0; e < 16; e += 2) {
      float a, c;
      unpack2<DT>(pack2<DT>(s[j][e], s[j][e + 1]), a, c);
      s[j][e] = a * scale;
      s[j][e + 1] = c * scale;
    }
    if (j >= nfull) {
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (32 * j + 8 * (e >> 2) + 4 * hi + (e & 3) >= T) s[j][e] = -INFINITY;
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[j][e]);
  });
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  float sum = 0.0f;
  static_for<NB>([&](auto j) {
#pragma unroll
    for (int e = 0; e < 16; ++e) s[j][e] = __expf(s[j][e] - mx);
    if (j >= nfull) {  // exact zeros past T, whatever mx is
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (32 * j + 8 * (e >> 2) + 4 * hi + (e & 3) >= T) s[j][e] = 0.0f;
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) sum += s[j][e];
  });
  sum += __shfl_xor(sum, 32);
  const float inv = 1.0f / sum;
  u32x2 R[NB][4];
  static_for<NB>([&](auto j) {
#pragma unroll
    for (int gq = 0; gq < 4; ++gq)
      R[j][gq] = u32x2{pack2<DT>(s[j][4 * gq] * inv, s[j][4 * gq + 1] * inv),
                       pack2<DT>(s[j][4 * gq + 2] * inv, s[j][4 * gq + 3] * inv)};
  });

  // O^T = V^T P^T: rows = d (two blocks of 32), columns = the wave's queries
  vst.store_clamped(sV, T, tid, NB * 64);
  __syncthreads();
  const uint32_t vbase = lds_u32(sV);
  f32x16 o[2];
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[db][e] = 0.0f;
  uint16_t* prow = P + ((int64_t)bh * T + q) * ldP;
  static_for<2 * NB>([&](auto ks) {
    const uint4 bf = keys_operand<NB>(R, ks);  // keys 16 ks + 8 hi + 0..7
    if (q < T && 16 * ks + 8 * hi < ldP) *reinterpret_cast<uint4*>(prow + 16 * ks + 8 * hi) = bf;
#pragma unroll
    for (int db = 0; db < 2; ++db) o[db] = mfma32<DT>(frag_tr(vbase, PD, 16 * ks, 32 * db, lane), bf, o[db]);
  });
  if (q < T) {
    uint16_t* out = O + ((int64_t)b * T + q) * dm + h * HD;
#pragma unroll
    for (int db = 0; db < 2; ++db) store_acc_row32<DT>(o[db], out + 32 * db, hi);
  }
}

// B operand of one key block's 16 keys 16 h .. 16 h + 15 (h = 0, 1) from the
// block's packed probabilities R4[gq] (keys 8 gq + 4 hi + 0..3), as above.
__device__ __forceinline__ uint4 block_keys_operand(const u32x2 (&R4)[4], int h) {
  u32x2 x = R4[2 * h], y = R4[2 * h + 1];
  half_swap(x, y);
  return make_uint4(x.x, x.y, y.x, y.y);
}

// More than 4 key blocks: one workgroup per (batch, head), one wave per block
// of 32 queries; K and V of the head staged in LDS.  The wave's scores are produced one key block
// at a time (S^T block j = K_j Q^T: a lane holds one query and half of the
// block's keys), in two passes so that no lane holds a whole score row:
//   pass 1: per lane, the running maximum m and the running sum l of
//           exp(z - m) over its keys (z = half(S) * scale), rescaled when
//           m grows; the two halves of a query's keys are then merged;
//   pass 2: the same scores again, p = half(exp(z - M) / L) written to P
//           and fed from registers to O^T += V_j^T P_j^T.
// p differs from a single pass over the whole row only in the rounding of
// the float32 sum L.
template <int DT, int NB>
__global__ __launch_bounds__(NB * 64) void attn_fwd_kernel(const uint16_t* __restrict__ qkv,
                                                           uint16_t* __restrict__ O,
                                                           uint16_t* __restrict__ P, int T, int H,
                                                           int ldP, float scale) {
  constexpr int TK = 32 * NB;
  __shared__ __attribute__((aligned(16))) uint16_t sK[TK * PD];
  __shared__ __attribute__((aligned(16))) uint16_t sV[TK * PD];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, hi = lane >> 5;
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int dm = H * HD;
  const int64_t ld = 3 * (int64_t)dm;
  const uint16_t* Q = qkv + (int64_t)b * T * ld + h * HD;
  const uint16_t* K = Q + dm;
  const uint16_t* V = Q + 2 * dm;

  const int q = 32 * w + (lane & 31);
  const int qc = min(q, T - 1);
  uint4 qf[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) qf[kk] = ld_u4(Q + qc * ld + 16 * kk + 8 * hi);
  RowStage<4> kst, vst;  // K and V: 32 NB rows over 64 NB threads
  kst.load_clamped(K, ld, T, tid, NB * 64);
  vst.load_clamped(V, ld, T, tid, NB * 64);
  kst.store_clamped(sK, T, tid, NB * 64);
  __syncthreads();
  const uint32_t kbase = lds_u32(sK), vbase = lds_u32(sV);

  // z = half(S) * scale for the lane's 16 keys of block j (-inf past T;
  // blocks below nfull have no key past T)
  const int nfull = T / 32;
  auto scores = [&](int j, float (&z)[16]) {
    f32x16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
    const uint32_t row = kbase + (uint32_t)(((32 * j + (lane & 31)) * PD + 8 * hi) * 2);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) acc = mfma32<DT>(lds_b128(row + 32 * kk), qf[kk], acc);
#pragma unroll
    for (int e = 0; e < 16; e += 2) {
      unpack2<DT>(pack2<DT>(acc[e], acc[e + 1]), z[e], z[e + 1]);
      z[e] *= scale;
      z[e + 1] *= scale;
    }
    if (j >= nfull) {
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (32 * j + 8 * (e >> 2) + 4 * hi + (e & 3) >= T) z[e] = -INFINITY;
    }
  };

  // pass 1
  float m = -INFINITY, l = 0.0f;
  for (int j = 0; j < NB; ++j) {
    float z[16];
    scores(j, z);
    float bm = z[0];
#pragma unroll
    for (int e = 1; e < 16; ++e) bm = fmaxf(bm, z[e]);
    if (bm == -INFINITY) continue;  // every key of this half-block is past T
    const float mn = fmaxf(m, bm);
    float t = 0.0f;
#pragma unroll
    for (int e = 0; e < 16; ++e) t += __expf(z[e] - mn);
    l = (m == -INFINITY ? 0.0f : l * __expf(m - mn)) + t;
    m = mn;
  }
  vst.store_clamped(sV, T, tid, NB * 64);
  __syncthreads();
  const float M = fmaxf(m, __shfl_xor(m, 32));  // finite: key 0 is in every row
  const float lc = m == -INFINITY ? 0.0f : l * __expf(m - M);
  const float inv = 1.0f / (lc + __shfl_xor(lc, 32));

  // pass 2
  f32x16 o[2];
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[db][e] = 0.0f;
  uint16_t* prow = P + ((int64_t)bh * T + q) * ldP;
  for (int j = 0; j < NB; ++j) {
    float z[16];
    scores(j, z);
    u32x2 R4[4];
    float ex[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) ex[e] = __expf(z[e] - M) * inv;
    if (j >= nfull) {  // exact zeros past T, whatever M is
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (32 * j + 8 * (e >> 2) + 4 * hi + (e & 3) >= T) ex[e] = 0.0f;
    }
#pragma unroll
    for (int gq = 0; gq < 4; ++gq)
      R4[gq] = u32x2{pack2<DT>(ex[4 * gq], ex[4 * gq + 1]), pack2<DT>(ex[4 * gq + 2], ex[4 * gq + 3])};
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const uint4 bf = block_keys_operand(R4, hh);  // keys 32 j + 16 hh + 8 hi + 0..7
      const int key0 = 32 * j + 16 * hh + 8 * hi;
      if (q < T && key0 < ldP) *reinterpret_cast<uint4*>(prow + key0) = bf;
#pragma unroll
      for (int db = 0; db < 2; ++db)
        o[db] = mfma32<DT>(frag_tr(vbase, PD, 32 * j + 16 * hh, 32 * db, lane), bf, o[db]);
    }
  }
  if (q < T) {
    uint16_t* out = O + ((int64_t)b * T + q) * dm + h * HD;
#pragma unroll
    for (int db = 0; db < 2; ++db) store_acc_row32<DT>(o[db], out + 32 * db, hi);
  }
}

// ---------------------------------------------------------------- backward --

// From the float32 accumulators dp (dP^T of the wave's queries, one block of
// 32 keys each; lane = query, entry [j][gq] holding keys 32 j + 8 gq + 4 hi
// + (0..3)) and the probabilities Pr of the lane's query in the same
// layout: dP rounded to half, the row sum rs = sum_k dP P, and
// dS = half(scale P (dP - rs)) packed like Pr.  The operands' rows past T
// are zero where these come from, so dP is 0 for keys >= T and for queries
// >= T and so are the probabilities: the sums and products need no masks (a
// masked term is an exact 0, and dS there is a zero of either sign).
// Conversions go two values at a time.
template <int DT, int NB>
__device__ __forceinline__ void probs_to_ds_zero_padded(f32x16 (&dp)[NB], const u32x2 (&Pr)[NB][4],
                                                        float scale, u32x2 (&Sr)[NB][4]) {
  float rs = 0.0f;
  static_for<NB>([&](auto j) {
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      float p[4], d[4];
      unpack2<DT>(Pr[j][gq].x, p[0], p[1]);
      unpack2<DT>(Pr[j][gq].y, p[2], p[3]);
      unpack2<DT>(pack2<DT>(dp[j][4 * gq], dp[j][4 * gq + 1]), d[0], d[1]);
      unpack2<DT>(pack2<DT>(dp[j][4 * gq + 2], dp[j][4 * gq + 3]), d[2], d[3]);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        dp[j][4 * gq + c] = d[c];
        rs += d[c] * p[c];
      }
    }
  });
  rs += __shfl_xor(rs, 32);
  static_for<NB>([&](auto j) {
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      float p[4], ds[4];
      unpack2<DT>(Pr[j][gq].x, p[0], p[1]);
      unpack2<DT>(Pr[j][gq].y, p[2], p[3]);
#pragma unroll
      for (int c = 0; c < 4; ++c) ds[c] = (scale * p[c]) * (dp[j][4 * gq + c] - rs);
      Sr[j][gq] = u32x2{pack2<DT>(ds[0], ds[1]), pack2<DT>(ds[2], ds[3])};
    }
  });
}

// dQ^T = K^T dS^T for the wave's queries (K staged in LDS as [key][d]):
// the float32 accumulators (lane = query, d in registers).
template <int DT, int NB>
__device__ __forceinline__ void bwd_dq_acc(uint32_t kbase, const u32x2 (&Sr)[NB][4], int lane, f32x16 (&o)[2]) {
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[db][e] = 0.0f;
  static_for<2 * NB>([&](auto ks) {
    const uint4 bf = keys_operand<NB>(Sr, ks);
#pragma unroll
    for (int db = 0; db < 2; ++db) o[db] = mfma32<DT>(frag_tr(kbase, PD, 16 * ks, 32 * db, lane), bf, o[db]);
  });
}

// The lane's dQ row (its query's 64 d) rounded to half: runs of 4 d.
template <int DT>
__device__ __forceinline__ void put_dq_row(const f32x16 (&o)[2], uint16_t* row, int lane) {
#pragma unroll
  for (int db = 0; db < 2; ++db) store_acc_row32<DT>(o[db], row + 32 * db, lane >> 5);
}

// dQ for the wave's queries, stored for queries < T.
template <int DT, int NB>
__device__ __forceinline__ void bwd_dq(uint32_t kbase, const u32x2 (&Sr)[NB][4], uint16_t* dQrow, int q,
                                       int T, int lane) {
  f32x16 o[2];
  bwd_dq_acc<DT, NB>(kbase, Sr, lane, o);
  if (q < T) put_dq_row<DT>(o, dQrow, lane);
}

// Store dK and dV rows of the wave's key block (accumulator runs of 4
// consecutive keys of one d, transposed to 4 consecutive d of one key).
template <int DT>
__device__ __forceinline__ void store_kv_block(const f32x16 (&dk)[2], const f32x16 (&dv)[2], uint16_t* dK,
                                               uint16_t* dV, int64_t ld, int key_base, int T, int lane) {
  const int hi = lane >> 5, q4 = lane & 3;
  const int col = 4 * ((lane & 31) >> 2);
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      float a[4] = {dk[db][4 * gq], dk[db][4 * gq + 1], dk[db][4 * gq + 2], dk[db][4 * gq + 3]};
      float c[4] = {dv[db][4 * gq], dv[db][4 * gq + 1], dv[db][4 * gq + 2], dv[db][4 * gq + 3]};
      quad_transpose(a, q4);
      quad_transpose(c, q4);
      const int key = key_base + 8 * gq + 4 * hi + q4;
      if (key < T) {
        st_u2(dK + key * ld + 32 * db + col, pack4(f2h<DT>(a[0]), f2h<DT>(a[1]), f2h<DT>(a[2]), f2h<DT>(a[3])));
        st_u2(dV + key * ld + 32 * db + col, pack4(f2h<DT>(c[0]), f2h<DT>(c[1]), f2h<DT>(c[2]), f2h<DT>(c[3])));
      }
    }
}

// Per query block (the wave's 32 queries q), V and dO read from global
// memory: dP^T = V dO^T, the probabilities P of query q and dS, without
// branches and with exact zeros past T: V rows of keys >= T and the dO row
// and probabilities of a query >= T are loaded from clamped addresses and
// masked to 0, so dP is 0 there and dS needs no masks
// (probs_to_ds_zero_padded).  The masks are ANDs, not selects: a select lets
// the compiler turn the load into a branch around it.
template <int DT, int NB>
__device__ __forceinline__ void bwd_query_block_zp(const uint16_t* V, int64_t ld, const uint16_t* G, int dm,
                                                   const uint16_t* Pbh, int ldP, int q, int T, float scale,
                                                   int lane, u32x2 (&Pr)[NB][4], u32x2 (&Sr)[NB][4]) {
  const int hi = lane >> 5;
  const int qc = min(q, T - 1);
  const uint32_t qmask = q < T ? 0xFFFFFFFFu : 0u;
  const uint16_t* Prow = Pbh + (int64_t)qc * ldP;
  static_for<NB>([&](auto j) {
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int key0 = 32 * j + 8 * gq + 4 * hi;
      const uint32_t m = key0 < T ? qmask : 0u;
      const u32x2 v = ld_u2(Prow + min(key0, ldP - 4));
      Pr[j][gq] = u32x2{v.x & m, v.y & m};
    }
  });
  uint4 gf[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    const uint4 v = ld_u4(G + qc * dm + 16 * kk + 8 * hi);
    gf[kk] = make_uint4(v.x & qmask, v.y & qmask, v.z & qmask, v.w & qmask);
  }
  f32x16 dp[NB];
  static_for<NB>([&](auto j) {
    const int key = 32 * j + (lane & 31);
    const uint32_t km = key < T ? 0xFFFFFFFFu : 0u;
    const uint16_t* vrow = V + min(key, T - 1) * ld + 8 * hi;
    f32x16 acc;
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const uint4 v = ld_u4(vrow + 16 * kk);
      acc = mfma32<DT>(make_uint4(v.x & km, v.y & km, v.z & km, v.w & km), gf[kk], acc);
    }
    dp[j] = acc;
  });
  probs_to_ds_zero_padded<DT, NB>(dp, Pr, scale, Sr);
}

// T <= 128: the whole backward of one (batch, head) in one workgroup.
template <int DT, int NB>
__global__ __launch_bounds__(NB * 64) void attn_bwd_kernel(const uint16_t* __restrict__ qkv,
                                                           const uint16_t* __restrict__ P,
                                                           const uint16_t* __restrict__ dO,
                                                           uint16_t* __restrict__ dqkv, int T, int H,
                                                           int ldP, float scale) {
  constexpr int TK = 32 * NB;
  // pitch (halves) of the [query][key] arrays: 4 consecutive rows of a
  // transposed read land in distinct banks, and at T <= 96 the whole LDS
  // footprint stays under 80 KiB, so two workgroups share a CU
  constexpr int PK = TK + 8;
  __shared__ __attribute__((aligned(16))) uint16_t sK[TK * PD];
  __shared__ __attribute__((aligned(16))) uint16_t sQ[TK * PD];
  __shared__ __attribute__((aligned(16))) uint16_t sdO[TK * PD];
  __shared__ __attribute__((aligned(16))) uint16_t sP[TK * PK];
  __shared__ __attribute__((aligned(16))) uint16_t sdS[TK * PK];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int dm = H * HD;
  const int64_t ld = 3 * (int64_t)dm;
  const uint16_t* Q = qkv + (int64_t)b * T * ld + h * HD;
  const uint16_t* K = Q + dm;
  const uint16_t* V = Q + 2 * dm;
  const uint16_t* G = dO + (int64_t)b * T * dm + h * HD;
  uint16_t* dQ = dqkv + (int64_t)b * T * ld + h * HD;

  {
    RowStage<4> kst, qst, gst;  // 32 NB rows each over 64 NB threads
    kst.load_clamped(K, ld, T, tid, NB * 64);
    qst.load_clamped(Q, ld, T, tid, NB * 64);
    gst.load_clamped(G, dm, T, tid, NB * 64);
    kst.store_clamped(sK, T, tid, NB * 64);
    qst.store_clamped(sQ, T, tid, NB * 64);
    gst.store_clamped(sdO, T, tid, NB * 64);
  }

  const int q = 32 * w + (lane & 31);
  u32x2 Pr[NB][4], Sr[NB][4];
  bwd_query_block_zp<DT, NB>(V, ld, G, dm, P + (int64_t)bh * T * ldP, ldP, q, T, scale, lane, Pr, Sr);
  // the [query][key] copies for the dK / dV products (rows >= T are 0)
  static_for<NB>([&](auto j) {
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int key0 = 32 * j + 8 * gq + 4 * (lane >> 5);
      *reinterpret_cast<u32x2*>(sP + q * PK + key0) = Pr[j][gq];
      *reinterpret_cast<u32x2*>(sdS + q * PK + key0) = Sr[j][gq];
    }
  });
  __syncthreads();  // sK / sQ / sdO staged, sP / sdS complete

  bwd_dq<DT, NB>(lds_u32(sK), Sr, dQ + q * ld, q, T, lane);

  // per key block (wave w): dK = dS^T Q and dV = P^T dO over all queries
  const uint32_t qbase = lds_u32(sQ), gbase = lds_u32(sdO), pbase = lds_u32(sP), sbase = lds_u32(sdS);
  f32x16 dk[2], dv[2];
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) dk[db][e] = dv[db][e] = 0.0f;
  static_for<2 * NB>([&](auto ks) {
    const uint4 sa = frag_tr(sbase, PK, 16 * ks, 32 * w, lane);
    const uint4 pa = frag_tr(pbase, PK, 16 * ks, 32 * w, lane);
#pragma unroll
    for (int db = 0; db < 2; ++db) {
      dk[db] = mfma32<DT>(sa, frag_tr(qbase, PD, 16 * ks, 32 * db, lane), dk[db]);
      dv[db] = mfma32<DT>(pa, frag_tr(gbase, PD, 16 * ks, 32 * db, lane), dv[db]);
    }
  });
  store_kv_block<DT>(dk, dv, dQ + dm, dQ + 2 * dm, ld, 32 * w, T, lane);
}

// Output staging of one wave: a [32][OP] half block in LDS, written from
// the accumulator layouts and copied out as whole 128-byte rows (16 bytes
// per lane, 8 lanes per row), instead of 8-byte pieces of 32 rows per store.
constexpr int OP = HD + 8;
__device__ __forceinline__ void copy_rows_out(const uint16_t* stage, uint16_t* dst, int64_t ld, int nrows,
                                              int lane) {
  asm volatile("" ::: "memory");  // the wave's writes to stage come first
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 8 * i + (lane >> 3), c = (lane & 7) * 8;
    const u32x4 v = *reinterpret_cast<const u32x4*>(stage + r * OP + c);
    if (r < nrows) *reinterpret_cast<u32x4*>(dst + r * ld + c) = v;
  }
  asm volatile("" ::: "memory");  // ... and the reads finish before it is written again
}

// dK or dV of the wave's key block through the staging block.
template <int DT>
__device__ __forceinline__ void put_kv_block(const f32x16 (&acc)[2], uint16_t* stage, int lane) {
  const int hi = lane >> 5, q4 = lane & 3;
  const int col = 4 * ((lane & 31) >> 2);
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      float a[4] = {acc[db][4 * gq], acc[db][4 * gq + 1], acc[db][4 * gq + 2], acc[db][4 * gq + 3]};
      quad_transpose(a, q4);
      st_u2(stage + (8 * gq + 4 * hi + q4) * OP + 32 * db + col,
            pack4(f2h<DT>(a[0]), f2h<DT>(a[1]), f2h<DT>(a[2]), f2h<DT>(a[3])));
    }
}

// 128 < T <= 256: the whole backward of one (batch, head) in one workgroup,
// without a [T, T] array in LDS.  K, V, Q and dO are staged in four [TK][PD]
// regions.  Pass 1 (wave w = query block w): dP^T = V dO^T from LDS, P rows
// from global memory, dS, then dQ = dS K; the wave keeps its P and dS
// blocks in registers.  Pass 2 (wave w = key block w): dK = dS^T Q and
// dV = P^T dO reduced over the query blocks in order: in round r wave r's
// P and dS blocks ([32 queries][TK keys]) are read from a slab in LDS, the
// slabs alternating between the K and V regions (free after pass 1) so
// that wave r + 1 writes the next one while round r is computed.  The
// arithmetic, and its order, is that of the two-kernel form: the same dS,
// dQ, dK and dV bits.
template <int DT, int NB>
__global__ __launch_bounds__(NB * 64) void attn_bwd_fused_kernel(const uint16_t* __restrict__ qkv,
                                                                 const uint16_t* __restrict__ P,
                                                                 const uint16_t* __restrict__ dO,
                                                                 uint16_t* __restrict__ dqkv, int T, int H,
                                                                 int ldP, float scale) {
  constexpr int TK = 32 * NB;
  constexpr int PK = TK + 16;  // slab pitch (halves)
  static_assert(2 * 32 * PK <= TK * PD, "a P slab and a dS slab fit in one staging region");
  __shared__ __attribute__((aligned(16))) uint16_t sK[TK * PD];  // pass 2: slabs of even rounds
  __shared__ __attribute__((aligned(16))) uint16_t sV[TK * PD];  // pass 2: slabs of odd rounds
  __shared__ __attribute__((aligned(16))) uint16_t sQ[TK * PD];
  __shared__ __attribute__((aligned(16))) uint16_t sdO[TK * PD];
  // per-wave output staging where it fits next to the four regions
  constexpr bool kStage = (4 * TK * PD + NB * 32 * OP) * 2 <= 160 * 1024;
  __shared__ __attribute__((aligned(16))) uint16_t sOut[kStage ? NB * 32 * OP : 8];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6, hi = lane >> 5;
  const int bh = blockIdx.x, b = bh / H, h = bh % H;
  const int dm = H * HD;
  const int64_t ld = 3 * (int64_t)dm;
  const uint16_t* Q = qkv + (int64_t)b * T * ld + h * HD;
  const uint16_t* G = dO + (int64_t)b * T * dm + h * HD;
  uint16_t* dQ = dqkv + (int64_t)b * T * ld + h * HD;
  const int q = 32 * w + (lane & 31);
  uint16_t* stage = sOut + (kStage ? w * 32 * OP : 0);
  const int nrows = min(32, T - 32 * w);  // rows of the wave's block below T (may be <= 0)

  u32x2 Pr[NB][4], Sr[NB][4];
  {
    // every load issued, out-of-range entries replaced by 0 afterwards
    const uint16_t* Prow = P + ((int64_t)bh * T + min(q, T - 1)) * ldP;
    static_for<NB>([&](auto j) {
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int key0 = 32 * j + 8 * gq + 4 * hi;
        Pr[j][gq] = ld_u2(Prow + min(key0, ldP - 4));
      }
    });
  }
  {
    RowStage<4> kst, vst, qst, gst;  // 32 NB rows each over 64 NB threads
    kst.load_clamped(Q + dm, ld, T, tid, NB * 64);
    vst.load_clamped(Q + 2 * dm, ld, T, tid, NB * 64);
    gst.load_clamped(G, dm, T, tid, NB * 64);
    qst.load_clamped(Q, ld, T, tid, NB * 64);
    kst.store_clamped(sK, T, tid, NB * 64);
    vst.store_clamped(sV, T, tid, NB * 64);
    gst.store_clamped(sdO, T, tid, NB * 64);
    qst.store_clamped(sQ, T, tid, NB * 64);
  }
  __syncthreads();
  const uint32_t kbase = lds_u32(sK), vbase = lds_u32(sV), qbase = lds_u32(sQ), gbase = lds_u32(sdO);

  // pass 1: dP^T = V dO^T (rows >= T of the staged arrays are 0), dS, dQ
  {
    uint4 gf[4];
    const uint32_t grow = gbase + (uint32_t)((q * PD + 8 * hi) * 2);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) gf[kk] = lds_b128(grow + 32 * kk);
    f32x16 dp[NB];
    static_for<NB>([&](auto j) {
      const uint32_t vrow = vbase + (uint32_t)(((32 * j + (lane & 31)) * PD + 8 * hi) * 2);
      f32x16 acc;
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[e] = 0.0f;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) acc = mfma32<DT>(lds_b128(vrow + 32 * kk), gf[kk], acc);
      dp[j] = acc;
    });
    static_for<NB>([&](auto j) {
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        asm volatile("" : "+v"(Pr[j][gq]));  // keeps the load above unconditional
        if (!(q < T && 32 * j + 8 * gq + 4 * hi < T)) Pr[j][gq] = u32x2{0u, 0u};
      }
    });
    probs_to_ds_zero_padded<DT, NB>(dp, Pr, scale, Sr);
  }
  if constexpr (kStage) {
    f32x16 o[2];
    bwd_dq_acc<DT, NB>(kbase, Sr, lane, o);
    put_dq_row<DT>(o, stage + (lane & 31) * OP, lane);
    copy_rows_out(stage, dQ + 32 * w * ld, ld, nrows, lane);
  } else {
    bwd_dq<DT, NB>(kbase, Sr, dQ + q * ld, q, T, lane);
  }
  __syncthreads();  // the K and V regions are free

  // pass 2
  auto write_slab = [&](uint16_t* slab) {
    const int ql = lane & 31;
    static_for<NB>([&](auto j) {
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int key0 = 32 * j + 8 * gq + 4 * hi;
        *reinterpret_cast<u32x2*>(slab + ql * PK + key0) = Pr[j][gq];
        *reinterpret_cast<u32x2*>(slab + 32 * PK + ql * PK + key0) = Sr[j][gq];
      }
    });
  };
  f32x16 dk[2], dv[2];
#pragma unroll
  for (int db = 0; db < 2; ++db)
#pragma unroll
    for (int e = 0; e < 16; ++e) dk[db][e] = dv[db][e] = 0.0f;
  if (w == 0) write_slab(sK);
  __syncthreads();
  for (int r = 0; r < NB; ++r) {
    // wave r + 1 fills the other slab: its last readers finished round r - 1
    if (w == r + 1) write_slab((r & 1) ? sK : sV);
    const uint32_t pbase = (r & 1) ? vbase : kbase, sbase = pbase + 32 * PK * 2;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const uint4 sa = frag_tr(sbase, PK, 16 * ks, 32 * w, lane);
      const uint4 pa = frag_tr(pbase, PK, 16 * ks, 32 * w, lane);
#pragma unroll
      for (int db = 0; db < 2; ++db) {
        dk[db] = mfma32<DT>(sa, frag_tr(qbase, PD, 32 * r + 16 * ks, 32 * db, lane), dk[db]);
        dv[db] = mfma32<DT>(pa, frag_tr(gbase, PD, 32 * r + 16 * ks, 32 * db, lane), dv[db]);
      }
    }
    __syncthreads();
  }
  if constexpr (kStage) {
    put_kv_block<DT>(dk, stage, lane);
    copy_rows_out(stage, dQ + dm + 32 * w * ld, ld, nrows, lane);
    put_kv_block<DT>(dv, stage, lane);
    copy_rows_out(stage, dQ + 2 * dm + 32 * w * ld, ld, nrows, lane);
  } else {
    store_kv_block<DT>(dk, dv, dQ + dm, dQ + 2 * dm, ld, 32 * w, T, lane);
  }
}

template <int DT>
hipError_t launch_fwd(const uint16_t* qkv, uint16_t* O, uint16_t* P, int B, int T, int H, int ldP,
                      float scale, hipStream_t s) {
  const dim3 grid((unsigned)(B * H));
  const int nb = (T + 31) / 32;
#define MPX_F(NBv) attn_fwd_kernel<DT, NBv><<<grid, NBv * 64, 0, s>>>(qkv, O, P, T, H, ldP, scale)
#define MPX_FR(NBv) attn_fwd_rows_kernel<DT, NBv><<<grid, NBv * 64, 0, s>>>(qkv, O, P, T, H, ldP, scale)
  switch (nb) {
    case 1: MPX_FR(1); break;
    case 2: MPX_FR(2); break;
    case 3: MPX_FR(3); break;
    case 4: MPX_FR(4); break;
    case 5: MPX_F(5); break;
    case 6: MPX_F(6); break;
    case 7: MPX_F(7); break;
    default: MPX_F(8); break;
  }
#undef MPX_FR
#undef MPX_F
  return hipGetLastError();
}

template <int DT>
hipError_t launch_bwd(const uint16_t* qkv, const uint16_t* P, const uint16_t* dO, uint16_t* dqkv, int B,
                      int T, int H, int ldP, float scale, hipStream_t s) {
  const dim3 grid((unsigned)(B * H));
  const int nb = (T + 31) / 32;
#define MPX_B(NBv) attn_bwd_kernel<DT, NBv><<<grid, NBv * 64, 0, s>>>(qkv, P, dO, dqkv, T, H, ldP, scale)
#define MPX_B2(NBv) attn_bwd_fused_kernel<DT, NBv><<<grid, NBv * 64, 0, s>>>(qkv, P, dO, dqkv, T, H, ldP, scale)
  switch (nb) {
    case 1: MPX_B(1); break;
    case 2: MPX_B(2); break;
    case 3: MPX_B(3); break;
    case 4: MPX_B(4); break;
    case 5: MPX_B2(5); break;
    case 6: MPX_B2(6); break;
    case 7: MPX_B2(7); break;
    default: MPX_B2(8); break;
  }
#undef MPX_B
#undef MPX_B2
  return hipGetLastError();
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace
}  // namespace mpx

using namespace mpx;

extern "C" int mpx_attention_fwd(const void* qkv, void* O, void* P, int64_t B, int64_t T, int64_t H,
                                 int64_t hd, mpx_dtype dt, void* stream) {
  clear_error();
  MPX_REQUIRE(qkv && O && P, "NULL operand");
  MPX_REQUIRE(B >= 1 && T >= 1 && H >= 1, "B, T, H must be >= 1");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_REQUIRE(B * H <= INT32_MAX && B * T * H * 3 * 64 < ((int64_t)1 << 31), "problem too large");
  if (hd != 64 || T > 256) {
    set_error("mpx_attention_fwd: implemented for head dimension 64 and T <= 256");
    return MPX_ERR_UNSUPPORTED;
  }
  MPX_REQUIRE(aligned16(qkv) && aligned16(O) && aligned16(P), "qkv, O and P must be 16-byte aligned");
  const int ldP = (int)((T + 7) / 8 * 8);
  const float scale = (float)(1.0 / std::sqrt((double)hd));
  hipStream_t s = (hipStream_t)stream;
  if (dt == MPX_F16)
    MPX_HIP(launch_fwd<MPX_F16>((const uint16_t*)qkv, (uint16_t*)O, (uint16_t*)P, (int)B, (int)T, (int)H,
                                ldP, scale, s));
  else
    MPX_HIP(launch_fwd<MPX_BF16>((const uint16_t*)qkv, (uint16_t*)O, (uint16_t*)P, (int)B, (int)T,
                                 (int)H, ldP, scale, s));
  return MPX_OK;
}

extern "C" size_t mpx_attention_bwd_workspace(int64_t, int64_t, int64_t, int64_t) { return 0; }

extern "C" int mpx_attention_bwd(const void* qkv, const void* P, const void* dO, void* dqkv, int64_t B,
                                 int64_t T, int64_t H, int64_t hd, mpx_dtype dt, void* workspace,
                                 size_t ws_bytes, void* stream) {
  clear_error();
  MPX_REQUIRE(qkv && P && dO && dqkv, "NULL operand");
  MPX_REQUIRE(B >= 1 && T >= 1 && H >= 1, "B, T, H must be >= 1");
  MPX_REQUIRE(is_half(dt), "dt must be MPX_F16 or MPX_BF16");
  MPX_REQUIRE(B * H <= INT32_MAX && B * T * H * 3 * 64 < ((int64_t)1 << 31), "problem too large");
  if (hd != 64 || T > 256) {
    set_error("mpx_attention_bwd: implemented for head dimension 64 and T <= 256");
    return MPX_ERR_UNSUPPORTED;
  }
  MPX_REQUIRE(aligned16(qkv) && aligned16(dO) && aligned16(dqkv) &&
                  (reinterpret_cast<uintptr_t>(P) & 7u) == 0,
              "qkv, dO and dqkv must be 16-byte aligned, P 8-byte aligned");
  (void)workspace;  // no workspace is used
  (void)ws_bytes;
  const int ldP = (int)((T + 7) / 8 * 8);
  const float scale = (float)(1.0 / std::sqrt((double)hd));
  hipStream_t s = (hipStream_t)stream;
  if (dt == MPX_F16)
    MPX_HIP(launch_bwd<MPX_F16>((const uint16_t*)qkv, (const uint16_t*)P, (const uint16_t*)dO,
                                (uint16_t*)dqkv, (int)B, (int)T, (int)H, ldP, scale, s));
  else
    MPX_HIP(launch_bwd<MPX_BF16>((const uint16_t*)qkv, (const uint16_t*)P, (const uint16_t*)dO,
                                 (uint16_t*)dqkv, (int)B, (int)T, (int)H, ldP, scale, s));
  return MPX_OK;
}
