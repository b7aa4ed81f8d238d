// Multi-tensor sweeps of the mixed-precision step: the float32 -> half cast
// of the parameter tree (MPX §3.1), the unscale + all-finite check (§3.3,
// §3.4), the dynamic loss-scale update (§3.3 adjust, rule of §2.1) and the
// masked AdamW update (§3.5).
//
// All sweeps are HBM-bound.  A tensor list is cut into fixed-size chunks
// once, at list creation; one workgroup owns one chunk and walks it in
// coalesced vector accesses (groups of 4 elements per lane, consecutive lanes
// on consecutive groups, several groups in flight per lane), falling back to
// scalar accesses only for chunk tails and for tensors whose base pointer is
// not 16-byte aligned.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "common.h"

namespace mpx {

static thread_local std::string g_err;
void set_error(const std::string& msg) { g_err = msg; }
void clear_error() { g_err.clear(); }

constexpr int kThreads = 256;

struct Chunk {
  int32_t tensor;
  int32_t len;
  int64_t start;
};

}  // namespace mpx

struct mpx_tlist_s {
  int32_t n = 0;
  int64_t total = 0;
  std::vector<void*> ptrs;
  std::vector<int64_t> numels;
  void** d_ptrs = nullptr;
  mpx::Chunk* d_chunks = nullptr;
  int32_t nchunks = 0;
};

namespace mpx {

// ------------------------------------------------------------- helpers --

__device__ __forceinline__ bool aligned16(const void* p) {
  return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

// Lanes work on groups of 4 consecutive elements so that a wave's float32
// accesses are one contiguous 1 KiB span per instruction (16 bytes per lane)
// and its half accesses one contiguous 512 B span (8 bytes per lane).  Each
// lane handles kUnroll groups per iteration to keep enough bytes in flight.
constexpr int kUnroll = 4;
constexpr int kGroup = 4;
constexpr int kStep = kUnroll * kGroup * kThreads;  // elements per workgroup iteration
// AdamW moves 28 bytes per element over eight streams; it reached more of
// the HBM bandwidth with half the work per workgroup (2048 elements, two
// float4 groups per lane per stream: 5.8 vs 5.65 TB/s on 1e8 elements),
// while the 2-byte check pass is faster on whole chunks
constexpr int kAdamUnroll = 2;
constexpr int kAdamStep = kAdamUnroll * kGroup * kThreads;
static_assert(2 * kAdamStep == kStep, "AdamW runs two workgroups per chunk");

// Chunk length: one workgroup iteration, so that every lane issues all of its
// loads at once and the grid holds as many workgroups as there are chunks
// (measured: the highest sustained bandwidth for these streaming updates).
static int64_t chunk_len(int64_t) { return kStep; }

// Streaming accesses: every byte is touched once per sweep, so loads and
// stores are marked non-temporal.
// The tensor pointers come from a device table, so the compiler cannot tell
// they are global memory; the casts let it use global (not flat) accesses.
typedef float nt_f4 __attribute__((ext_vector_type(4)));
typedef uint32_t nt_u2 __attribute__((ext_vector_type(2)));
#define MPX_GLOBAL __attribute__((address_space(1)))
__device__ __forceinline__ float4 ld_nt(const float* p) {
  const nt_f4 v = __builtin_nontemporal_load((const MPX_GLOBAL nt_f4*)p);
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st_nt(float* p, float4 v) {
  __builtin_nontemporal_store((nt_f4){v.x, v.y, v.z, v.w}, (MPX_GLOBAL nt_f4*)p);
}
__device__ __forceinline__ uint2 ld_nt(const uint16_t* p) {
  const nt_u2 v = __builtin_nontemporal_load((const MPX_GLOBAL nt_u2*)p);
  return make_uint2(v.x, v.y);
}
__device__ __forceinline__ void st_nt(uint16_t* p, uint2 v) {
  __builtin_nontemporal_store((nt_u2){v.x, v.y}, (MPX_GLOBAL nt_u2*)p);
}

__device__ __forceinline__ void unpack_h4(uint2 u, uint16_t (&h)[4]) {
  h[0] = (uint16_t)(u.x & 0xFFFFu);
  h[1] = (uint16_t)(u.x >> 16);
  h[2] = (uint16_t)(u.y & 0xFFFFu);
  h[3] = (uint16_t)(u.y >> 16);
}
__device__ __forceinline__ uint2 pack_h4(const uint16_t (&h)[4]) {
  return make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16));
}
__device__ __forceinline__ float get(const float4& v, int j) {
  return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
}
__device__ __forceinline__ void set(float4& v, int j, float x) {
  if (j == 0) v.x = x; else if (j == 1) v.y = x; else if (j == 2) v.z = x; else v.w = x;
}

// ----------------------------------------------------------------- cast --

template <int HDT>
__global__ __launch_bounds__(kThreads) void cast_kernel(const Chunk* __restrict__ chunks,
                                                        void* const* __restrict__ src_ptrs,
                                                        void* const* __restrict__ dst_ptrs) {
  const Chunk c = chunks[blockIdx.x];
  const float* src = reinterpret_cast<const float*>(src_ptrs[c.tensor]) + c.start;
  uint16_t* dst = reinterpret_cast<uint16_t*>(dst_ptrs[c.tensor]) + c.start;
  const int len = c.len;
  int done = 0;
  if (aligned16(src) && aligned16(dst)) {
    for (; done + kStep <= len; done += kStep) {
      float4 f[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        f[u] = ld_nt(src + done + (u * kThreads + threadIdx.x) * kGroup);
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        uint16_t h[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) h[j] = f2h<HDT>(get(f[u], j));
        st_nt(dst + done + (u * kThreads + threadIdx.x) * kGroup, pack_h4(h));
      }
    }
  }
  for (int i = done + threadIdx.x; i < len; i += kThreads) dst[i] = f2h<HDT>(src[i]);
}

// The inverse direction: half -> float32, exact (every half value is a
// float32 value).
template <int HDT>
__global__ __launch_bounds__(kThreads) void widen_kernel(const Chunk* __restrict__ chunks,
                                                         void* const* __restrict__ src_ptrs,
                                                         void* const* __restrict__ dst_ptrs) {
  const Chunk c = chunks[blockIdx.x];
  const uint16_t* src = reinterpret_cast<const uint16_t*>(src_ptrs[c.tensor]) + c.start;
  float* dst = reinterpret_cast<float*>(dst_ptrs[c.tensor]) + c.start;
  const int len = c.len;
  int done = 0;
  if (aligned16(src) && aligned16(dst)) {
    for (; done + kStep <= len; done += kStep) {
      uint2 raw[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        raw[u] = ld_nt(src + done + (u * kThreads + threadIdx.x) * kGroup);
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        uint16_t h[4];
        unpack_h4(raw[u], h);
        st_nt(dst + done + (u * kThreads + threadIdx.x) * kGroup,
              make_float4(h2f<HDT>(h[0]), h2f<HDT>(h[1]), h2f<HDT>(h[2]), h2f<HDT>(h[3])));
      }
    }
  }
  for (int i = done + threadIdx.x; i < len; i += kThreads) dst[i] = h2f<HDT>(src[i]);
}

// -------------------------------------------------------- unscale/check --

template <int GDT, bool WRITE>
__global__ __launch_bounds__(kThreads) void unscale_check_kernel(
    const Chunk* __restrict__ chunks, void* const* __restrict__ g_ptrs,
    void* const* __restrict__ o_ptrs, const mpx_scale_state* __restrict__ state,
    int32_t* __restrict__ nonfinite) {
  const Chunk c = chunks[blockIdx.x];
  const uint16_t* g = reinterpret_cast<const uint16_t*>(g_ptrs[c.tensor]) + c.start;
  float* out = WRITE ? reinterpret_cast<float*>(o_ptrs[c.tensor]) + c.start : nullptr;
  const float scale = WRITE ? state->scale : 1.0f;
  const int len = c.len;
  int bad = 0;
  int done = 0;
  if (aligned16(g) && (!WRITE || aligned16(out))) {
    for (; done + kStep <= len; done += kStep) {
      uint2 raw[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u)
        raw[u] = ld_nt(g + done + (u * kThreads + threadIdx.x) * kGroup);
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        uint16_t h[4];
        unpack_h4(raw[u], h);
        float4 f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          bad += h_nonfinite<GDT>(h[j]) ? 1 : 0;
          if (WRITE) set(f, j, h2f<GDT>(h[j]) / scale);
        }
        if (WRITE) st_nt(out + done + (u * kThreads + threadIdx.x) * kGroup, f);
      }
    }
  }
  for (int i = done + threadIdx.x; i < len; i += kThreads) {
    uint16_t h = g[i];
    bad += h_nonfinite<GDT>(h) ? 1 : 0;
    if (WRITE) out[i] = h2f<GDT>(h) / scale;
  }
  // workgroup reduction of the count, then one atomic per workgroup
  __shared__ int part[kThreads / 64];
  bad = wave_sum_int(bad);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = bad;
  __syncthreads();
  if (threadIdx.x == 0) {
    int s = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) s += part[w];
    // only workgroups that found a non-finite value touch the (pre-zeroed) count
    if (s) atomicAdd(nonfinite, s);
  }
}

// ---------------------------------------------------------- scale update --

__global__ void scale_update_kernel(mpx_scale_state* st, const int32_t* nonfinite) {
  mpx_scale_state s = *st;
  if (*nonfinite == 0) {
    s.counter += 1;
    if (s.counter == s.period) {
      s.scale = fminf(s.scale * s.factor, s.max_scale);
      s.counter = 0;
    }
  } else {
    s.scale = fmaxf(s.scale / s.factor, s.min_scale);
    s.counter = 0;
  }
  *st = s;
}

// ----------------------------------------------------------- masked AdamW --

struct AdamConsts {
  float b1, omb1, b2, omb2, lr, eps, wd;
  double beta1, beta2;  // for the bias corrections 1 - beta^t
};

// One element of AdamW, float32, in the order of the definition (no
// contraction into fused multiply-adds, so results match a plain float32
// evaluation of the same expression).
__device__ __forceinline__ void adamw_elem(float& p, float& m, float& v, float g,
                                           const AdamConsts& k, float bc1, float bc2) {
#pragma clang fp contract(off)
  m = k.b1 * m + k.omb1 * g;
  v = k.b2 * v + k.omb2 * (g * g);
  float mhat = m / bc1;
  float vhat = v / bc2;
  float upd = mhat / (sqrtf(vhat) + k.eps) + k.wd * p;
  p = p - k.lr * upd;
}

template <int GDT>
__device__ __forceinline__ float grad_value(const void* base, int i, float scale) {
  if constexpr (GDT == MPX_F32) {
    return reinterpret_cast<const float*>(base)[i];
  } else {
    return h2f<GDT>(reinterpret_cast<const uint16_t*>(base)[i]) / scale;
  }
}

// HDT: dtype of the half copy, or MPX_F32 for "no half copy".
template <int GDT, int HDT>
__global__ __launch_bounds__(kThreads) void adamw_kernel(
    const Chunk* __restrict__ chunks, void* const* __restrict__ p_ptrs,
    void* const* __restrict__ m_ptrs, void* const* __restrict__ v_ptrs,
    void* const* __restrict__ g_ptrs, void* const* __restrict__ h_ptrs, AdamConsts k,
    const int32_t* __restrict__ step, const mpx_scale_state* __restrict__ state,
    const int32_t* __restrict__ nonfinite) {
  if (*nonfinite != 0) return;  // skipped step: nothing is written (uniform)
  const int t = *step + 1;
  const float bc1 = (float)(1.0 - pow(k.beta1, (double)t));
  const float bc2 = (float)(1.0 - pow(k.beta2, (double)t));
  const float scale = state->scale;

  // two workgroups per chunk, each on one half (kAdamStep elements)
  const Chunk c = chunks[blockIdx.x >> 1];
  const int64_t start = c.start + (int64_t)(blockIdx.x & 1) * kAdamStep;
  float* p = reinterpret_cast<float*>(p_ptrs[c.tensor]) + start;
  float* m = reinterpret_cast<float*>(m_ptrs[c.tensor]) + start;
  float* v = reinterpret_cast<float*>(v_ptrs[c.tensor]) + start;
  constexpr int gsz = GDT == MPX_F32 ? 4 : 2;
  const char* g = reinterpret_cast<const char*>(g_ptrs[c.tensor]) + start * gsz;
  uint16_t* h = HDT != MPX_F32 ? reinterpret_cast<uint16_t*>(h_ptrs[c.tensor]) + start : nullptr;
  const int len = min(kAdamStep, c.len - (int)(blockIdx.x & 1) * kAdamStep);
  if (len <= 0) return;
  int done = 0;
  if (aligned16(p) && aligned16(m) && aligned16(v) && aligned16(g) &&
      (HDT == MPX_F32 || aligned16(h))) {
    for (; done + kAdamStep <= len; done += kAdamStep) {
      float4 pp[kAdamUnroll], mm[kAdamUnroll], vv[kAdamUnroll];
      float gg[kAdamUnroll][4];
#pragma unroll
      for (int u = 0; u < kAdamUnroll; ++u) {
        const int e = done + (u * kThreads + threadIdx.x) * kGroup;
        pp[u] = ld_nt(p + e);
        mm[u] = ld_nt(m + e);
        vv[u] = ld_nt(v + e);
        if constexpr (GDT == MPX_F32) {
          const float4 t4 = ld_nt(reinterpret_cast<const float*>(g) + e);
          gg[u][0] = t4.x; gg[u][1] = t4.y; gg[u][2] = t4.z; gg[u][3] = t4.w;
        } else {
          uint16_t hh[4];
          unpack_h4(ld_nt(reinterpret_cast<const uint16_t*>(g) + e), hh);
#pragma unroll
          for (int j = 0; j < 4; ++j) gg[u][j] = h2f<GDT>(hh[j]);
        }
      }
#pragma unroll
      for (int u = 0; u < kAdamUnroll; ++u) {
        const int e = done + (u * kThreads + threadIdx.x) * kGroup;
        float P[4], Mv[4], V[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          P[j] = get(pp[u], j);
          Mv[j] = get(mm[u], j);
          V[j] = get(vv[u], j);
          const float gj = GDT == MPX_F32 ? gg[u][j] : gg[u][j] / scale;
          adamw_elem(P[j], Mv[j], V[j], gj, k, bc1, bc2);
        }
        st_nt(p + e, make_float4(P[0], P[1], P[2], P[3]));
        st_nt(m + e, make_float4(Mv[0], Mv[1], Mv[2], Mv[3]));
        st_nt(v + e, make_float4(V[0], V[1], V[2], V[3]));
        if constexpr (HDT != MPX_F32) {
          uint16_t hh[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) hh[j] = f2h<HDT>(P[j]);
          st_nt(h + e, pack_h4(hh));
        }
      }
    }
  }
  for (int i = done + threadIdx.x; i < len; i += kThreads) {
    float pp = p[i], mm = m[i], vv = v[i];
    float gg = grad_value<GDT>(g, i, scale);
    adamw_elem(pp, mm, vv, gg, k, bc1, bc2);
    p[i] = pp;
    m[i] = mm;
    v[i] = vv;
    if constexpr (HDT != MPX_F32) h[i] = f2h<HDT>(pp);
  }
}

// Advances the applied-step count after the update (one thread; on a skipped
// step nothing changes).
__global__ void step_count_kernel(int32_t* step, const int32_t* nonfinite) {
  if (*nonfinite == 0) *step += 1;
}

__global__ void zero_i32_kernel(int32_t* p) { *p = 0; }

// ------------------------------------------------------------------ zero --

__global__ void zero_kernel(uint8_t* p, size_t n) {
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  size_t stride = (size_t)gridDim.x * blockDim.x;
  size_t n16 = n / 16;
  if ((reinterpret_cast<uintptr_t>(p) & 15u) == 0) {
    for (size_t j = i; j < n16; j += stride) reinterpret_cast<uint4*>(p)[j] = make_uint4(0, 0, 0, 0);
    for (size_t j = n16 * 16 + i; j < n; j += stride) p[j] = 0;
  } else {
    for (size_t j = i; j < n; j += stride) p[j] = 0;
  }
}

static bool same_shape(const mpx_tlist_s* a, const mpx_tlist_s* b) {
  return a->n == b->n && a->numels == b->numels;
}

}  // namespace mpx

using namespace mpx;

// =================================================================== ABI ==

extern "C" const char* mpx_last_error(void) { return g_err.c_str(); }

extern "C" int mpx_tlist_create(const void* const* ptrs, const int64_t* numels, int32_t n,
                                mpx_tlist* out) {
  clear_error();
  MPX_REQUIRE(out != nullptr, "out is NULL");
  MPX_REQUIRE(n >= 0, "negative tensor count");
  MPX_REQUIRE(n == 0 || (ptrs != nullptr && numels != nullptr), "ptrs/numels NULL");
  std::vector<Chunk> chunks;
  auto* t = new mpx_tlist_s();
  t->n = n;
  int64_t total = 0;
  for (int32_t i = 0; i < n; ++i) total += numels[i] > 0 ? numels[i] : 0;
  const int64_t chunk = chunk_len(total);
  for (int32_t i = 0; i < n; ++i) {
    if (numels[i] < 0 || (numels[i] > 0 && ptrs[i] == nullptr)) {
      delete t;
      set_error("mpx_tlist_create: bad tensor " + std::to_string(i));
      return MPX_ERR_INVALID;
    }
    t->ptrs.push_back(const_cast<void*>(ptrs[i]));
    t->numels.push_back(numels[i]);
    t->total += numels[i];
    for (int64_t s = 0; s < numels[i]; s += chunk) {
      int64_t len = numels[i] - s < chunk ? numels[i] - s : chunk;
      chunks.push_back(Chunk{i, (int32_t)len, s});
    }
  }
  t->nchunks = (int32_t)chunks.size();
  hipError_t e = hipSuccess;
  if (n > 0) e = hipMalloc(&t->d_ptrs, sizeof(void*) * n);
  if (e == hipSuccess && n > 0)
    e = hipMemcpy(t->d_ptrs, t->ptrs.data(), sizeof(void*) * n, hipMemcpyHostToDevice);
  if (e == hipSuccess && !chunks.empty()) e = hipMalloc(&t->d_chunks, sizeof(Chunk) * chunks.size());
  if (e == hipSuccess && !chunks.empty())
    e = hipMemcpy(t->d_chunks, chunks.data(), sizeof(Chunk) * chunks.size(), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    set_error(std::string("mpx_tlist_create: ") + hipGetErrorString(e));
    mpx_tlist_destroy(t);
    return MPX_ERR_HIP;
  }
  *out = t;
  return MPX_OK;
}

extern "C" int mpx_tlist_destroy(mpx_tlist t) {
  if (!t) return MPX_OK;
  if (t->d_ptrs) (void)hipFree(t->d_ptrs);
  if (t->d_chunks) (void)hipFree(t->d_chunks);
  delete t;
  return MPX_OK;
}

extern "C" int64_t mpx_tlist_numel(mpx_tlist t) { return t ? t->total : -1; }

extern "C" int mpx_cast_to_half(mpx_tlist src, mpx_tlist dst, mpx_dtype half, void* stream) {
  clear_error();
  MPX_REQUIRE(src && dst, "NULL list");
  MPX_REQUIRE(is_half(half), "half must be MPX_F16 or MPX_BF16");
  MPX_REQUIRE(same_shape(src, dst), "src and dst lists differ in shape");
  if (src->nchunks == 0) return MPX_OK;
  hipStream_t s = (hipStream_t)stream;
  if (half == MPX_F16)
    cast_kernel<MPX_F16><<<src->nchunks, kThreads, 0, s>>>(src->d_chunks, src->d_ptrs, dst->d_ptrs);
  else
    cast_kernel<MPX_BF16><<<src->nchunks, kThreads, 0, s>>>(src->d_chunks, src->d_ptrs, dst->d_ptrs);
  MPX_LAUNCHED();
  return MPX_OK;
}

extern "C" int mpx_cast_to_float(mpx_tlist src, mpx_tlist dst, mpx_dtype half, void* stream) {
  clear_error();
  MPX_REQUIRE(src && dst, "NULL list");
  MPX_REQUIRE(is_half(half), "half must be MPX_F16 or MPX_BF16");
  MPX_REQUIRE(same_shape(src, dst), "src and dst lists differ in shape");
  if (src->nchunks == 0) return MPX_OK;
  hipStream_t s = (hipStream_t)stream;
  if (half == MPX_F16)
    widen_kernel<MPX_F16><<<src->nchunks, kThreads, 0, s>>>(src->d_chunks, src->d_ptrs, dst->d_ptrs);
  else
    widen_kernel<MPX_BF16><<<src->nchunks, kThreads, 0, s>>>(src->d_chunks, src->d_ptrs, dst->d_ptrs);
  MPX_LAUNCHED();
  return MPX_OK;
}

extern "C" int mpx_unscale_check(mpx_tlist grads, mpx_dtype gdt, const mpx_scale_state* d_state,
                                 int32_t* d_nonfinite, mpx_tlist out_f32, void* stream) {
  clear_error();
  MPX_REQUIRE(grads && d_nonfinite, "NULL argument");
  MPX_REQUIRE(is_half(gdt), "gdt must be MPX_F16 or MPX_BF16");
  MPX_REQUIRE(!out_f32 || d_state, "d_state is required when out_f32 is given");
  MPX_REQUIRE(!out_f32 || same_shape(grads, out_f32), "out_f32 differs in shape from grads");
  hipStream_t s = (hipStream_t)stream;
  zero_i32_kernel<<<1, 1, 0, s>>>(d_nonfinite);
  MPX_LAUNCHED();
  if (grads->nchunks == 0) return MPX_OK;
  void* const* o = out_f32 ? out_f32->d_ptrs : nullptr;
  dim3 g(grads->nchunks), b(kThreads);
  if (gdt == MPX_F16) {
    if (out_f32)
      unscale_check_kernel<MPX_F16, true><<<g, b, 0, s>>>(grads->d_chunks, grads->d_ptrs, o, d_state, d_nonfinite);
    else
      unscale_check_kernel<MPX_F16, false><<<g, b, 0, s>>>(grads->d_chunks, grads->d_ptrs, o, d_state, d_nonfinite);
  } else {
    if (out_f32)
      unscale_check_kernel<MPX_BF16, true><<<g, b, 0, s>>>(grads->d_chunks, grads->d_ptrs, o, d_state, d_nonfinite);
    else
      unscale_check_kernel<MPX_BF16, false><<<g, b, 0, s>>>(grads->d_chunks, grads->d_ptrs, o, d_state, d_nonfinite);
  }
  MPX_LAUNCHED();
  return MPX_OK;
}

extern "C" int mpx_scale_update(mpx_scale_state* d_state, const int32_t* d_nonfinite, void* stream) {
  clear_error();
  MPX_REQUIRE(d_state && d_nonfinite, "NULL argument");
  scale_update_kernel<<<1, 1, 0, (hipStream_t)stream>>>(d_state, d_nonfinite);
  MPX_LAUNCHED();
  return MPX_OK;
}

template <int GDT, int HDT>
static void launch_adamw(mpx_tlist p, mpx_tlist m, mpx_tlist v, mpx_tlist g, mpx_tlist h,
                         const AdamConsts& k, int32_t* step, const mpx_scale_state* st,
                         const int32_t* nf, hipStream_t s) {
  adamw_kernel<GDT, HDT><<<2 * p->nchunks, kThreads, 0, s>>>(
      p->d_chunks, p->d_ptrs, m->d_ptrs, v->d_ptrs, g->d_ptrs, h ? h->d_ptrs : nullptr, k, step,
      st, nf);
  step_count_kernel<<<1, 1, 0, s>>>(step, nf);
}

extern "C" int mpx_adamw_masked(mpx_tlist p32, mpx_tlist m32, mpx_tlist v32, mpx_tlist grads,
                                mpx_dtype gdt, const mpx_adamw_hp* hp, int32_t* d_step,
                                const mpx_scale_state* d_state, const int32_t* d_nonfinite,
                                mpx_tlist half_copy, mpx_dtype half, void* stream) {
  clear_error();
  MPX_REQUIRE(p32 && m32 && v32 && grads && hp && d_step && d_state && d_nonfinite,
              "NULL argument");
  MPX_REQUIRE(gdt == MPX_F32 || is_half(gdt), "bad gradient dtype");
  MPX_REQUIRE(!half_copy || is_half(half), "half copy dtype must be MPX_F16 or MPX_BF16");
  MPX_REQUIRE(same_shape(p32, m32) && same_shape(p32, v32) && same_shape(p32, grads) &&
                  (!half_copy || same_shape(p32, half_copy)),
              "lists differ in shape");
  MPX_REQUIRE(hp->beta1 >= 0 && hp->beta1 < 1 && hp->beta2 >= 0 && hp->beta2 < 1,
              "betas must lie in [0, 1)");
  if (p32->nchunks == 0) return MPX_OK;
  AdamConsts k;
  k.b1 = (float)hp->beta1;
  k.omb1 = (float)(1.0 - hp->beta1);
  k.b2 = (float)hp->beta2;
  k.omb2 = (float)(1.0 - hp->beta2);
  k.lr = (float)hp->lr;
  k.eps = (float)hp->eps;
  k.wd = (float)hp->weight_decay;
  k.beta1 = hp->beta1;
  k.beta2 = hp->beta2;
  hipStream_t s = (hipStream_t)stream;
  const int hd = half_copy ? (int)half : (int)MPX_F32;
#define MPX_ADAMW_CASE(G, H)                                                             \
  if (gdt == G && hd == H) {                                                             \
    launch_adamw<G, H>(p32, m32, v32, grads, half_copy, k, d_step, d_state, d_nonfinite, s); \
    MPX_LAUNCHED();                                                                      \
    return MPX_OK;                                                                       \
  }
  MPX_ADAMW_CASE(MPX_F16, MPX_F16)
  MPX_ADAMW_CASE(MPX_F16, MPX_BF16)
  MPX_ADAMW_CASE(MPX_F16, MPX_F32)
  MPX_ADAMW_CASE(MPX_BF16, MPX_F16)
  MPX_ADAMW_CASE(MPX_BF16, MPX_BF16)
  MPX_ADAMW_CASE(MPX_BF16, MPX_F32)
  MPX_ADAMW_CASE(MPX_F32, MPX_F16)
  MPX_ADAMW_CASE(MPX_F32, MPX_BF16)
  MPX_ADAMW_CASE(MPX_F32, MPX_F32)
#undef MPX_ADAMW_CASE
  set_error("mpx_adamw_masked: unsupported dtype combination");
  return MPX_ERR_UNSUPPORTED;
}

extern "C" int mpx_zero(void* dst, size_t nbytes, void* stream) {
  clear_error();
  MPX_REQUIRE(dst || nbytes == 0, "NULL destination");
  if (nbytes == 0) return MPX_OK;
  size_t blocks = (nbytes / 16 + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 4096) blocks = 4096;
  zero_kernel<<<(unsigned)blocks, 256, 0, (hipStream_t)stream>>>(reinterpret_cast<uint8_t*>(dst), nbytes);
  MPX_LAUNCHED();
  return MPX_OK;
}
