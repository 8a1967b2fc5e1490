// Small memory-bound kernels of the forward: embedding gather, row RMSNorm,
// RoPE + KV-cache append for prefill rows, the second argmax pass and the
// device-side step state.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace wici {

namespace {
thread_local const LaunchTimer* g_launch_timer = nullptr;
}
void set_launch_timer(const LaunchTimer* t) { g_launch_timer = t; }
const LaunchTimer* launch_timer() { return g_launch_timer; }

// ---- embedding ------------------------------------------------------------------
// Q8 rows: codes (q + 128) and one half-precision scale per 32 elements (S).
__device__ __forceinline__ void load8(const uint8_t* p, float* o, const unsigned short* s) {
  const uint2 c = *reinterpret_cast<const uint2*>(p);
  const float d = (float)__builtin_bit_cast(_Float16, *s);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    o[j] = ((float)((c.x >> (8 * j)) & 0xffu) - 128.f) * d;
    o[4 + j] = ((float)((c.y >> (8 * j)) & 0xffu) - 128.f) * d;
  }
}

template <typename WT>
__global__ __launch_bounds__(256) void k_embed(const WT* __restrict__ E,
                                               const unsigned short* __restrict__ S, int d,
                                               const int32_t* __restrict__ tokens,
                                               const DecodeState* __restrict__ st,
                                               float* __restrict__ x) {
  const int t = blockIdx.x;
  const int tok = tokens ? tokens[t] : st->token;
  const size_t r = (size_t)(tok < 0 ? 0 : tok);
  const WT* row = E + r * d;
  for (int k = threadIdx.x * 8; k < d; k += 256 * 8) {
    float v[8];
    if constexpr (sizeof(WT) == 1) load8(row + k, v, S + r * (d / 32) + k / 32);
    else load8(row + k, v);
    if (tok < 0)
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = 0.f;
    float4* o = reinterpret_cast<float4*>(x + (size_t)t * d + k);
    o[0] = make_float4(v[0], v[1], v[2], v[3]);
    o[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
}

hipError_t launch_embed(int wt, const void* E, int V, int d, const int32_t* tokens, int T,
                        const void* state, float* x, hipStream_t st) {
  const DecodeState* s = static_cast<const DecodeState*>(state);
  switch (wt) {
    case W_BF16:
      launch_k(k_embed<bf16_t>, dim3(T), dim3(256), 0, st, kOnly, static_cast<const bf16_t*>(E),
               (const unsigned short*)nullptr, d, tokens, s, x);
      break;
    case W_F32:
      launch_k(k_embed<float>, dim3(T), dim3(256), 0, st, kOnly, static_cast<const float*>(E),
               (const unsigned short*)nullptr, d, tokens, s, x);
      break;
    case W_Q8: {
      const uint8_t* c = static_cast<const uint8_t*>(E);
      launch_k(k_embed<uint8_t>, dim3(T), dim3(256), 0, st, kOnly, c,
               reinterpret_cast<const unsigned short*>(c + q8_scale_offset(V, d)), d, tokens, s,
               x);
      break;
    }
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

__global__ void k_set_token(DecodeState* st, int token) {
  st->token = token;
  st->bad = 0;
}

__global__ void k_reset_state(DecodeState* st) {
  st->pos = 0;
  st->token = 0;
  st->bad = 0;
  st->fault = 0;
}

hipError_t launch_reset_state(void* state, hipStream_t st) {
  hipLaunchKernelGGL(k_reset_state, dim3(1), dim3(1), 0, st, static_cast<DecodeState*>(state));
  return hipGetLastError();
}

hipError_t launch_set_token(void* state, int token, hipStream_t st) {
  hipLaunchKernelGGL(k_set_token, dim3(1), dim3(1), 0, st, static_cast<DecodeState*>(state),
                     token);
  return hipGetLastError();
}

// Pages are handed out from the top of the pool down, so logical page i lives in
// physical page n_pages-1-i: any kernel that ignored the table would read the
// wrong page.
__global__ void k_init_block_table(int32_t* table, int n_pages) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n_pages) table[i] = n_pages - 1 - i;
}

__global__ void k_fill_i32(int32_t* p, int n, int v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

hipError_t launch_fill_i32(int32_t* p, int n, int v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_fill_i32, dim3((n + 255) / 256), dim3(256), 0, st, p, n, v);
  return hipGetLastError();
}

hipError_t launch_init_block_table(int32_t* table, int n_pages, hipStream_t st) {
  hipLaunchKernelGGL(k_init_block_table, dim3((n_pages + 255) / 256), dim3(256), 0, st, table,
                     n_pages);
  return hipGetLastError();
}

// ---- RMSNorm of T rows ------------------------------------------------------------
__global__ __launch_bounds__(256) void k_rmsnorm_rows(const float* __restrict__ x,
                                                      const float* __restrict__ g, float eps,
                                                      int d, ActBuf y) {
  __shared__ float red[4];
  const float* xr = x + (size_t)blockIdx.x * d;
  const size_t yr = (size_t)blockIdx.x * d;
  float ss = 0.f;
  for (int k = threadIdx.x * 4; k < d; k += 1024) {
    const float4 v = *reinterpret_cast<const float4*>(xr + k);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  const float r = 1.0f / sqrtf(block256_sum(ss, red) / (float)d + eps);
  for (int k = threadIdx.x * 4; k < d; k += 1024) {
    const float4 v = *reinterpret_cast<const float4*>(xr + k);
    const float4 w = *reinterpret_cast<const float4*>(g + k);
    store_act(y, yr + k + 0, v.x * r * w.x);
    store_act(y, yr + k + 1, v.y * r * w.y);
    store_act(y, yr + k + 2, v.z * r * w.z);
    store_act(y, yr + k + 3, v.w * r * w.w);
  }
}

// The same for rows of NV * 1024 values: the row and the gain are loaded at once
// and kept in registers (the loop form waits for each slice in turn, then reads
// the row again).  Same elements per thread and order of operations, so the
// results are bit-identical.
template <int NV>
__global__ __launch_bounds__(256) void k_rmsnorm_rows_reg(const float* __restrict__ x,
                                                          const float* __restrict__ g, float eps,
                                                          int d, ActBuf y) {
  __shared__ float red[4];
  const float4* xr = reinterpret_cast<const float4*>(x + (size_t)blockIdx.x * d);
  const size_t yr = (size_t)blockIdx.x * d;
  const int tid = threadIdx.x;
  float4 v[NV], w[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = xr[tid + 256 * i];
#pragma unroll
  for (int i = 0; i < NV; ++i) w[i] = reinterpret_cast<const float4*>(g)[tid + 256 * i];
  // the loop form's sum of squares as that kernel is compiled (y^2 rounded, then
  // x, z and w fused in), written out so that the compiler cannot fuse it
  // differently here: the same bits at every row length
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i)
    ss += __builtin_fmaf(v[i].w, v[i].w,
                         __builtin_fmaf(v[i].z, v[i].z, __builtin_fmaf(v[i].x, v[i].x, v[i].y * v[i].y)));
  const float r = 1.0f / sqrtf(block256_sum(ss, red) / (float)d + eps);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const size_t k = yr + 4 * (tid + 256 * i);
    store_act4(y, k, make_float4(v[i].x * r * w[i].x, v[i].y * r * w[i].y, v[i].z * r * w[i].z,
                                 v[i].w * r * w[i].w));
  }
}

hipError_t launch_rmsnorm_rows(const float* x, const float* gain, float eps, int T, int d,
                               const ActBuf& y, hipStream_t st) {
  if (d % 1024 == 0 && d / 1024 >= 1 && d / 1024 <= 8) {
    switch (d / 1024) {
#define WICI_RN(NV)                                                                              \
  case NV:                                                                                       \
    hipLaunchKernelGGL((k_rmsnorm_rows_reg<NV>), dim3(T), dim3(256), 0, st, x, gain, eps, d, y); \
    return hipGetLastError();
      WICI_RN(1) WICI_RN(2) WICI_RN(3) WICI_RN(4) WICI_RN(5) WICI_RN(6) WICI_RN(7) WICI_RN(8)
#undef WICI_RN
    }
  }
  hipLaunchKernelGGL(k_rmsnorm_rows, dim3(T), dim3(256), 0, st, x, gain, eps, d, y);
  return hipGetLastError();
}

// Residual add of split-K partial products, then (optionally) the row RMSNorm.
__global__ __launch_bounds__(256) void k_resid_sum_rmsnorm(float* __restrict__ x,
                                                           const float* __restrict__ P,
                                                           int nsplit, size_t p_split,
                                                           const float* __restrict__ g,
                                                           float eps, int d, ActBuf y) {
  __shared__ float red[4];
  float* xr = x + (size_t)blockIdx.x * d;
  const float* pr = P + (size_t)blockIdx.x * d;
  const size_t yr = (size_t)blockIdx.x * d;
  float ss = 0.f;
  for (int k = threadIdx.x * 4; k < d; k += 1024) {
    float4 v = *reinterpret_cast<const float4*>(xr + k);
    for (int s = 0; s < nsplit; ++s) {
      const float4 p = *reinterpret_cast<const float4*>(pr + s * p_split + k);
      v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
    }
    *reinterpret_cast<float4*>(xr + k) = v;
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  if (!g) return;
  const float r = 1.0f / sqrtf(block256_sum(ss, red) / (float)d + eps);
  for (int k = threadIdx.x * 4; k < d; k += 1024) {  // this thread's own values
    const float4 v = *reinterpret_cast<const float4*>(xr + k);
    const float4 w = *reinterpret_cast<const float4*>(g + k);
    store_act(y, yr + k + 0, v.x * r * w.x);
    store_act(y, yr + k + 1, v.y * r * w.y);
    store_act(y, yr + k + 2, v.z * r * w.z);
    store_act(y, yr + k + 3, v.w * r * w.w);
  }
}

// The same for rows of NV * 1024 values and NS partials: every load of the row
// (x, the partials, the gain) is issued at once and the row stays in registers for
// the norm (the loop form above waits for each partial in turn and reads x
// back).  Same elements per thread and the same order of additions, so the
// results are bit-identical.  8B at 1024 rows, four partials: 25.6 -> ~17 us.
template <int NS, int NV>
__global__ __launch_bounds__(256) void k_resid_sum_rmsnorm_reg(float* __restrict__ x,
                                                               const float* __restrict__ P,
                                                               size_t p_split,
                                                               const float* __restrict__ g,
                                                               float eps, int d, ActBuf y) {
  __shared__ float red[4];
  float4* xr = reinterpret_cast<float4*>(x + (size_t)blockIdx.x * d);
  const float4* pr = reinterpret_cast<const float4*>(P + (size_t)blockIdx.x * d);
  const size_t yr = (size_t)blockIdx.x * d;
  const int tid = threadIdx.x;
  float4 v[NV], p[NS][NV], w[NV];
#pragma unroll
  for (int i = 0; i < NV; ++i) v[i] = xr[tid + 256 * i];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int i = 0; i < NV; ++i) p[s][i] = pr[s * (p_split / 4) + tid + 256 * i];
  if (g) {
#pragma unroll
    for (int i = 0; i < NV; ++i) w[i] = reinterpret_cast<const float4*>(g)[tid + 256 * i];
  }
  float ss = 0.f;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      v[i].x += p[s][i].x; v[i].y += p[s][i].y; v[i].z += p[s][i].z; v[i].w += p[s][i].w;
    }
    xr[tid + 256 * i] = v[i];
    ss += v[i].x * v[i].x + v[i].y * v[i].y + v[i].z * v[i].z + v[i].w * v[i].w;
  }
  if (!g) return;
  const float r = 1.0f / sqrtf(block256_sum(ss, red) / (float)d + eps);
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const size_t k = yr + 4 * (tid + 256 * i);
    store_act4(y, k, make_float4(v[i].x * r * w[i].x, v[i].y * r * w[i].y, v[i].z * r * w[i].z,
                                 v[i].w * r * w[i].w));
  }
}

template <int NS>
static bool resid_sum_reg(float* x, const float* P, size_t p_split, const float* gain, float eps,
                          int T, int d, const ActBuf& y, hipStream_t st) {
  if (d % 1024 || p_split % 4) return false;
  switch (d / 1024) {
#define WICI_RS(NV)                                                                           \
  case NV:                                                                                    \
    hipLaunchKernelGGL((k_resid_sum_rmsnorm_reg<NS, NV>), dim3(T), dim3(256), 0, st, x, P, \
                       p_split, gain, eps, d, y);                                             \
    return true;
    WICI_RS(1) WICI_RS(2) WICI_RS(3) WICI_RS(4) WICI_RS(5) WICI_RS(6) WICI_RS(7) WICI_RS(8)
#undef WICI_RS
    default: return false;
  }
}

hipError_t launch_resid_sum_rmsnorm(float* x, const float* P, int nsplit, size_t p_split,
                                    const float* gain, float eps, int T, int d, const ActBuf& y,
                                    hipStream_t st) {
  if (nsplit < 1 || d % 4) return hipErrorInvalidValue;
  const bool reg = nsplit == 2   ? resid_sum_reg<2>(x, P, p_split, gain, eps, T, d, y, st)
                   : nsplit == 3 ? resid_sum_reg<3>(x, P, p_split, gain, eps, T, d, y, st)
                   : nsplit == 4 ? resid_sum_reg<4>(x, P, p_split, gain, eps, T, d, y, st)
                                 : false;
  if (!reg)
    hipLaunchKernelGGL(k_resid_sum_rmsnorm, dim3(T), dim3(256), 0, st, x, P, nsplit, p_split,
                       gain, eps, d, y);
  return hipGetLastError();
}

// ---- RoPE + KV append for prefill rows --------------------------------------------
// One block per row; thread j < hd/2 of a head rotates the pair (j, j + hd/2).
template <typename KT>
__global__ __launch_bounds__(256) void k_rope_append(float* __restrict__ qkv, int p0, int Hq,
                                                     const float* __restrict__ cos_t,
                                                     const float* __restrict__ sin_t,
                                                     KvLayout kv, const float* __restrict__ part,
                                                     int nsplit, size_t p_split) {
  const int t = blockIdx.x, pos = p0 + t;
  const int hd = kv.hd, half = hd >> 1, Hkv = kv.n_kv;
  const int width = (Hq + 2 * Hkv) * hd;
  float* row = qkv + (size_t)t * width;
  // element i of the row: the projection's output, or the sum of its K-range
  // partial products in range order
  const float* prow = part ? part + (size_t)t * width : row;
  auto val = [&](int i) {
    float v = prow[i];
    for (int s = 1; s < nsplit; ++s) v += prow[(size_t)s * p_split + i];
    return v;
  };
  const float* cr = cos_t + (size_t)pos * half;
  const float* sr = sin_t + (size_t)pos * half;
  KT* base = static_cast<KT*>(kv.base);
  const int phys = kv.table[pos / kv.page], slot = pos % kv.page;
  // rotate q heads (into qkv), k heads into the cache
  for (int i = threadIdx.x; i < (Hq + Hkv) * half; i += blockDim.x) {
    const int h = i / half, j = i % half;
    const float a = val(h * hd + j), b = val(h * hd + j + half), c = cr[j], s = sr[j];
    const float ra = a * c - b * s, rb = a * s + b * c;
    if (h < Hq) {
      row[h * hd + j] = ra;
      row[h * hd + j + half] = rb;
    } else {
      const int g = h - Hq;
      KT* dst = base + (((size_t)phys * 2 + 0) * Hkv + g) * kv.page * hd + (size_t)slot * hd;
      Elem<KT>::store(dst + j, ra);
      Elem<KT>::store(dst + j + half, rb);
    }
  }
  for (int i = threadIdx.x; i < Hkv * hd; i += blockDim.x) {
    const int g = i / hd, e = i % hd;
    KT* dst = base + (((size_t)phys * 2 + 1) * Hkv + g) * kv.page * hd + (size_t)slot * hd;
    Elem<KT>::store(dst + e, val((Hq + Hkv) * hd + i));
  }
}

// The same on 4-element slices (head dimension a multiple of 8), with every load
// of a thread's slices (both K-range partials, cos and sin) issued before any is
// used: the loop form above makes each of its ~14 iterations wait out its own
// loads.  Slices past the end load a clamped index and store nothing.  Same
// operations per element, so the results are bit-identical.
template <typename KT, int NP, int MAXI>
__global__ __launch_bounds__(256) void k_rope_append4(float* __restrict__ qkv, int p0, int Hq,
                                                      const float* __restrict__ cos_t,
                                                      const float* __restrict__ sin_t,
                                                      KvLayout kv, const float* __restrict__ part,
                                                      size_t p_split) {
  const int t = blockIdx.x, pos = p0 + t, tid = threadIdx.x;
  const int hd = kv.hd, half = hd >> 1, Hkv = kv.n_kv, q4 = half >> 2;
  const int width = (Hq + 2 * Hkv) * hd;
  float* row = qkv + (size_t)t * width;
  // the projection's row itself (rotated in place: every slice is read before
  // any is written, each by the thread that writes it) or its K-range partials
  const float* prow = part ? part + (size_t)t * width : row;
  auto ld4 = [&](int i) {  // elements i .. i + 3, the K-range partials summed in order
    float4 v = *reinterpret_cast<const float4*>(prow + i);
#pragma unroll
    for (int s = 1; s < NP; ++s) {
      const float4 w = *reinterpret_cast<const float4*>(prow + (size_t)s * p_split + i);
      v.x += w.x; v.y += w.y; v.z += w.z; v.w += w.w;
    }
    return v;
  };
  KT* base = static_cast<KT*>(kv.base);
  const int phys = kv.table[pos / kv.page], slot = pos % kv.page;
  const int nrot = (Hq + Hkv) * q4, nval = Hkv * hd / 4;  // slices
  float4 a[MAXI], b[MAXI], c[MAXI], sn[MAXI], v[MAXI];
#pragma unroll
  for (int k = 0; k < MAXI; ++k) {
    const int i = min(tid + 256 * k, nrot - 1), h = i / q4, j = 4 * (i % q4);
    a[k] = ld4(h * hd + j);
    b[k] = ld4(h * hd + j + half);
    c[k] = *reinterpret_cast<const float4*>(cos_t + (size_t)pos * half + j);
    sn[k] = *reinterpret_cast<const float4*>(sin_t + (size_t)pos * half + j);
    v[k] = ld4((Hq + Hkv) * hd + 4 * min(tid + 256 * k, nval - 1));
  }
  auto put = [&](KT* dst, float4 x) {
    if constexpr (sizeof(KT) == 4) {
      *reinterpret_cast<float4*>(dst) = x;
    } else {
      const uint2 u = make_uint2((uint32_t)f32_to_bf16(x.x) | ((uint32_t)f32_to_bf16(x.y) << 16),
                                 (uint32_t)f32_to_bf16(x.z) | ((uint32_t)f32_to_bf16(x.w) << 16));
      *reinterpret_cast<uint2*>(dst) = u;
    }
  };
#pragma unroll
  for (int k = 0; k < MAXI; ++k) {
    const int i = tid + 256 * k;
    if (i < nrot) {
      const int h = i / q4, j = 4 * (i % q4);
      float4 ra, rb;
      ra.x = a[k].x * c[k].x - b[k].x * sn[k].x; rb.x = a[k].x * sn[k].x + b[k].x * c[k].x;
      ra.y = a[k].y * c[k].y - b[k].y * sn[k].y; rb.y = a[k].y * sn[k].y + b[k].y * c[k].y;
      ra.z = a[k].z * c[k].z - b[k].z * sn[k].z; rb.z = a[k].z * sn[k].z + b[k].z * c[k].z;
      ra.w = a[k].w * c[k].w - b[k].w * sn[k].w; rb.w = a[k].w * sn[k].w + b[k].w * c[k].w;
      if (h < Hq) {
        *reinterpret_cast<float4*>(row + h * hd + j) = ra;
        *reinterpret_cast<float4*>(row + h * hd + j + half) = rb;
      } else {
        KT* dst = base + (((size_t)phys * 2 + 0) * Hkv + (h - Hq)) * kv.page * hd + (size_t)slot * hd;
        put(dst + j, ra);
        put(dst + j + half, rb);
      }
    }
    if (i < nval) {
      const int g = (4 * i) / hd, e = (4 * i) % hd;
      KT* dst = base + (((size_t)phys * 2 + 1) * Hkv + g) * kv.page * hd + (size_t)slot * hd;
      put(dst + e, v[k]);
    }
  }
}

template <typename KT>
static bool rope_append4(float* qkv, int T, int p0, int Hq, const float* cos_t,
                         const float* sin_t, KvLayout kv, hipStream_t st, const float* part,
                         int nsplit, size_t p_split) {
  constexpr int MAXI = 4;
  const int hd = kv.hd;
  if (hd % 8 || p_split % 4 || (Hq + kv.n_kv) * (hd / 8) > 256 * MAXI ||
      kv.n_kv * hd / 4 > 256 * MAXI)
    return false;
  switch (part ? nsplit : 1) {
    case 1:
      hipLaunchKernelGGL((k_rope_append4<KT, 1, MAXI>), dim3(T), dim3(256), 0, st, qkv, p0, Hq,
                         cos_t, sin_t, kv, (const float*)nullptr, p_split);
      return true;
    case 2:
      hipLaunchKernelGGL((k_rope_append4<KT, 2, MAXI>), dim3(T), dim3(256), 0, st, qkv, p0, Hq,
                         cos_t, sin_t, kv, part, p_split);
      return true;
    case 3:
      hipLaunchKernelGGL((k_rope_append4<KT, 3, MAXI>), dim3(T), dim3(256), 0, st, qkv, p0, Hq,
                         cos_t, sin_t, kv, part, p_split);
      return true;
    case 4:
      hipLaunchKernelGGL((k_rope_append4<KT, 4, MAXI>), dim3(T), dim3(256), 0, st, qkv, p0, Hq,
                         cos_t, sin_t, kv, part, p_split);
      return true;
    default:
      return false;
  }
}

hipError_t launch_rope_append(bool kv_bf16, float* qkv, int T, int p0, int Hq,
                              const float* cos_t, const float* sin_t, KvLayout kv,
                              hipStream_t st, const float* part, int nsplit, size_t p_split) {
  if (nsplit < 1 || (nsplit > 1 && !part)) return hipErrorInvalidValue;
  if (nsplit == 1) part = nullptr;
  if (kv_bf16 ? rope_append4<bf16_t>(qkv, T, p0, Hq, cos_t, sin_t, kv, st, part, nsplit, p_split)
              : rope_append4<float>(qkv, T, p0, Hq, cos_t, sin_t, kv, st, part, nsplit, p_split))
    return hipGetLastError();
  if (kv_bf16)
    hipLaunchKernelGGL(k_rope_append<bf16_t>, dim3(T), dim3(256), 0, st, qkv, p0, Hq, cos_t,
                       sin_t, kv, part, nsplit, p_split);
  else
    hipLaunchKernelGGL(k_rope_append<float>, dim3(T), dim3(256), 0, st, qkv, p0, Hq, cos_t,
                       sin_t, kv, part, nsplit, p_split);
  return hipGetLastError();
}

// ---- plain streaming read (the bandwidth ceiling the decode GEMVs are held to) ----------
// Workgroup b of G reads the 16 KiB blocks b, b + G, b + 2G, ... of the buffer:
// four non-temporal 16-byte loads per lane per block, all issued before any is
// used.  The XOR of every loaded word keeps the loads from being dropped; one
// word per thread is written (never read).
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(256) void k_stream_read(const u32x4* __restrict__ p, size_t blocks,
                                                     unsigned* __restrict__ sink) {
  unsigned acc = 0;
  for (size_t b = blockIdx.x; b < blocks; b += gridDim.x) {
    const u32x4* q = p + b * 1024 + threadIdx.x;
    const u32x4 v0 = __builtin_nontemporal_load(q);
    const u32x4 v1 = __builtin_nontemporal_load(q + 256);
    const u32x4 v2 = __builtin_nontemporal_load(q + 512);
    const u32x4 v3 = __builtin_nontemporal_load(q + 768);
    const u32x4 x = v0 ^ v1 ^ v2 ^ v3;
    acc ^= x.x ^ x.y ^ x.z ^ x.w;
  }
  sink[(size_t)blockIdx.x * 256 + threadIdx.x] = acc;
}

hipError_t launch_stream_read(const void* buf, size_t bytes, int grid, unsigned* sink,
                              hipStream_t st) {
  if (!buf || !sink || grid < 1 || bytes < 16384 || bytes % 16384) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_stream_read, dim3(grid), dim3(256), 0, st,
                     static_cast<const u32x4*>(buf), bytes / 16384, sink);
  return hipGetLastError();
}

// out[0] = XOR of in[0 .. n): one workgroup.  Every 32-bit word of a streamed
// buffer is XORed into exactly one thread's sink word, so the XOR of a read's
// sink is the XOR of the whole buffer, whatever the grid.
__global__ __launch_bounds__(256) void k_xor_reduce(const unsigned* __restrict__ in, int n,
                                                    unsigned* __restrict__ out) {
  __shared__ unsigned red[256];
  unsigned a = 0;
  for (int i = threadIdx.x; i < n; i += 256) a ^= in[i];
  red[threadIdx.x] = a;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) red[threadIdx.x] ^= red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = red[0];
}

hipError_t launch_xor_reduce(const unsigned* in, int n, unsigned* out, hipStream_t st) {
  if (!in || !out || n < 0) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_xor_reduce, dim3(1), dim3(256), 0, st, in, n, out);
  return hipGetLastError();
}

// ---- argmax, second pass -------------------------------------------------------------
// One 256-thread workgroup.  The state it updates is read first, alongside the
// partials, so its load latency is not added after the reduction.
__global__ __launch_bounds__(256) void k_argmax_final(const ArgmaxPart* __restrict__ part,
                                                       int n, DecodeState* st,
                                                       int32_t* __restrict__ hist, int advance,
                                                       int set_pos, DecodeState* mirror) {
  __shared__ float sv[4];
  __shared__ int si[4];
  __shared__ int sbad[4];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  DecodeState cur{};
  if (tid == 0) cur = *st;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  int bad = 0;
  for (int i = tid; i < n; i += 256) {
    const ArgmaxPart p = part[i];
    if (p.i < 0) bad = 1;
    else if (am_better(p.v, p.i, bv, bi)) { bv = p.v; bi = p.i; }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = __shfl_xor(bv, m);
    const int oi = __shfl_xor(bi, m);
    if (am_better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    bad |= __shfl_xor(bad, m);
  }
  if (lane == 0) { sv[w] = bv; si[w] = bi; sbad[w] = bad; }
  __syncthreads();
  if (tid == 0) {
    for (int k = 1; k < 4; ++k) {
      if (am_better(sv[k], si[k], bv, bi)) { bv = sv[k]; bi = si[k]; }
      bad |= sbad[k];
    }
    if (set_pos < 0 && cur.bad) return;  // an earlier step of this run failed
    const int pos = set_pos >= 0 ? set_pos : cur.pos + advance;
    const int tok = bad ? -1 : bi;
    st->bad = bad;
    st->token = tok;
    st->pos = pos;
    if (pos >= 1) hist[pos - 1] = tok;
    if (mirror) {  // pinned host copy; `done` last, after a system-scope fence
      mirror->bad = bad;
      mirror->token = tok;
      mirror->pos = pos;
      mirror->fault = cur.fault;
      __threadfence_system();
      mirror->done = 1;
    }
  }
}

hipError_t launch_argmax_final(const ArgmaxPart* part, int n, void* state, int32_t* hist,
                               int advance, int set_pos, void* host_mirror, hipStream_t st) {
  launch_k(k_argmax_final, dim3(1), dim3(256), 0, st, kOnly, part, n,
           static_cast<DecodeState*>(state), hist, advance, set_pos,
           static_cast<DecodeState*>(host_mirror));
  return hipGetLastError();
}

}  // namespace wici
