// Weight-streaming GEMV for the batch-1 decode step (y = W x).
//
// Decode is bound by HBM bandwidth: every weight byte is read once per token
// and used for one multiply-add.  On MI355X the DRAM side streams fastest when
// the whole chip reads one sliding, contiguous window of memory with a modest
// number of non-temporal 16-byte loads in flight per lane (measured: ~7.2 TB/s
// with one 256-thread workgroup per CU and eight loads per lane, against
// 5.4-6.5 TB/s for more workgroups or scattered row streams).  The kernel is
// shaped after that:
//  - a persistent grid (one or two workgroups per CU); wavefront w of the grid
//    owns row groups w, w + W, w + 2W, ... (W wavefronts in all), so at any time
//    the chip streams a contiguous band of rows;
//  - a row group is ROWS complete rows (two for a gate/up pair of the SwiGLU
//    epilogue) read with 64 lanes x 16 B = 1 KiB coalesced loads, in batches of
//    U sweeps of 512 elements; the next batch is issued before the current one
//    is consumed (double buffering), so loads never stop at row boundaries;
//  - the first batch is issued before the prologue, which stages x * gain in
//    LDS; an RMS-normalised input gets its 1/rms factor applied to the finished
//    row sums (W (x g r) = r W (x g)), so one barrier publishes the vector;
//  - row sums are reduced with DPP row operations; after the prologue no
//    wavefront ever waits for another.
#include "common.h"
#include "kernels.h"

namespace wici {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
template <typename WT> struct Vec8;   // 8 weights
template <> struct Vec8<bf16_t> { u32x4 a; };
template <> struct Vec8<float> { u32x4 a, b; };

// Weights are read exactly once per step: non-temporal loads keep them from
// displacing the small vectors that are reused from the caches.
__device__ __forceinline__ void ld(Vec8<bf16_t>& v, const bf16_t* p) {
  v.a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void ld(Vec8<float>& v, const float* p) {
  v.a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  v.b = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p) + 1);
}
__device__ __forceinline__ void zero(Vec8<bf16_t>& v) { v.a = u32x4{0, 0, 0, 0}; }
__device__ __forceinline__ void zero(Vec8<float>& v) { v.a = u32x4{0, 0, 0, 0}; v.b = v.a; }
__device__ __forceinline__ float dot8(const Vec8<bf16_t>& v, const float* x) {
  const float4 xa = *reinterpret_cast<const float4*>(x);
  const float4 xb = *reinterpret_cast<const float4*>(x + 4);
  return __uint_as_float(v.a.x << 16) * xa.x + __uint_as_float(v.a.x & 0xffff0000u) * xa.y +
         __uint_as_float(v.a.y << 16) * xa.z + __uint_as_float(v.a.y & 0xffff0000u) * xa.w +
         __uint_as_float(v.a.z << 16) * xb.x + __uint_as_float(v.a.z & 0xffff0000u) * xb.y +
         __uint_as_float(v.a.w << 16) * xb.z + __uint_as_float(v.a.w & 0xffff0000u) * xb.w;
}
__device__ __forceinline__ float dot8(const Vec8<float>& v, const float* x) {
  const float4 xa = *reinterpret_cast<const float4*>(x);
  const float4 xb = *reinterpret_cast<const float4*>(x + 4);
  return __uint_as_float(v.a.x) * xa.x + __uint_as_float(v.a.y) * xa.y +
         __uint_as_float(v.a.z) * xa.z + __uint_as_float(v.a.w) * xa.w +
         __uint_as_float(v.b.x) * xb.x + __uint_as_float(v.b.y) * xb.y +
         __uint_as_float(v.b.z) * xb.z + __uint_as_float(v.b.w) * xb.w;
}

// Batch b of a wavefront = (row group, first sweep); nsb batches per group.
template <typename WT, int ROWS, int U>
struct Batch {
  Vec8<WT> w[ROWS][U];
};

template <typename WT, int EPI, bool NORM, int ROWS, int U>
__global__ __launch_bounds__(256) void k_gemv(const WT* __restrict__ W, int N, int K,
                                              const float* __restrict__ x,
                                              const float* __restrict__ gain, float eps,
                                              float* __restrict__ y,
                                              ArgmaxPart* __restrict__ part) {
  static_assert(EPI != GEMV_SWIGLU || ROWS % 2 == 0, "SwiGLU needs whole gate/up pairs");
  extern __shared__ float xs[];  // K floats
  __shared__ float red[4];
  __shared__ float am_v[4];
  __shared__ int am_i[4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int nsweep = (K + 511) >> 9;          // 512-element sweeps per row
  const int nsb = (nsweep + U - 1) / U;       // batches per row group
  const int ngroups = (N + ROWS - 1) / ROWS;
  const int wid = blockIdx.x * 4 + wave, nw = gridDim.x * 4;
  const int my_groups = wid < ngroups ? (ngroups - 1 - wid) / nw + 1 : 0;
  const int nbatch = my_groups * nsb;

  // issue batch b into buf (rows past N and lanes past K read nothing)
  auto issue = [&](Batch<WT, ROWS, U>& buf, int b) {
    const int gi = b / nsb, s0 = (b - gi * nsb) * U;
    const int r0 = (wid + gi * nw) * ROWS;
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
      const WT* wr = W + (size_t)min(r0 + r, N - 1) * K + lane * 8;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int k = (s0 + u) * 512 + lane * 8;
        if (r0 + r < N && k < K) ld(buf.w[r][u], wr + (s0 + u) * 512);
        else zero(buf.w[r][u]);
      }
    }
  };

  Batch<WT, ROWS, U> b0, b1;
  if (nbatch > 0) issue(b0, 0);

  // ---- stage x * gain in LDS, sum of squares for the norm ---------------------------
  float ss = 0.f;
  {
    constexpr int SU = 4;
    for (int k0 = tid * 4; k0 < K; k0 += 1024 * SU) {
      float4 v[SU];
#pragma unroll
      for (int u = 0; u < SU; ++u)
        if (k0 + u * 1024 < K) v[u] = *reinterpret_cast<const float4*>(x + k0 + u * 1024);
#pragma unroll
      for (int u = 0; u < SU; ++u) {
        const int k = k0 + u * 1024;
        if (k < K) {
          float4 t = v[u];
          if (NORM) {
            ss += t.x * t.x + t.y * t.y + t.z * t.z + t.w * t.w;
            const float4 g = *reinterpret_cast<const float4*>(gain + k);
            t.x *= g.x; t.y *= g.y; t.z *= g.z; t.w *= g.w;
          }
          *reinterpret_cast<float4*>(xs + k) = t;
        }
      }
    }
  }
  if (NORM) {
    ss = wave_sum(ss);
    if (lane == 0) red[wave] = ss;
  }
  __syncthreads();
  const float rnorm = NORM ? 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)K + eps)
                           : 1.0f;

  float acc[ROWS];
#pragma unroll
  for (int r = 0; r < ROWS; ++r) acc[r] = 0.f;
  float best_v = -INFINITY;
  int best_i = 0x7fffffff;
  bool bad = false;

  auto consume = [&](const Batch<WT, ROWS, U>& buf, int b) {
    const int gi = b / nsb, sb = b - gi * nsb, s0 = sb * U;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = (s0 + u) * 512 + lane * 8;
      if (k < K) {
        const float* xk = xs + k;
#pragma unroll
        for (int r = 0; r < ROWS; ++r) acc[r] += dot8(buf.w[r][u], xk);
      }
    }
    if (sb == nsb - 1) {  // row group complete
      const int r0 = (wid + gi * nw) * ROWS;
#pragma unroll
      for (int r = 0; r < ROWS; ++r) acc[r] = wave_sum(acc[r]) * rnorm;
      if (EPI == GEMV_SWIGLU) {
#pragma unroll
        for (int r = 0; r < ROWS; r += 2)
          if (lane == r && r0 + r + 1 < N) y[(r0 + r) >> 1] = silu(acc[r]) * acc[r + 1];
      } else {
#pragma unroll
        for (int r = 0; r < ROWS; ++r) {
          if (lane == r && r0 + r < N) {
            if (EPI == GEMV_RESID) y[r0 + r] += acc[r];
            else y[r0 + r] = acc[r];
          }
          if (EPI == GEMV_ARGMAX && r0 + r < N) {
            // NaN never compares better; a non-finite logit is flagged separately
            if (am_better(acc[r], r0 + r, best_v, best_i)) { best_v = acc[r]; best_i = r0 + r; }
            bad |= !isfinite(acc[r]);
          }
        }
      }
#pragma unroll
      for (int r = 0; r < ROWS; ++r) acc[r] = 0.f;
    }
  };

  // double-buffered stream of batches: issue b+1, consume b
  for (int b = 0; b < nbatch; b += 2) {
    if (b + 1 < nbatch) issue(b1, b + 1);
    consume(b0, b);
    if (b + 1 < nbatch) {
      if (b + 2 < nbatch) issue(b0, b + 2);
      consume(b1, b + 1);
    }
  }

  if (EPI == GEMV_ARGMAX) {
    // a non-finite logit marks the partial with index -1
    if (lane == 0) { am_v[wave] = best_v; am_i[wave] = bad ? -1 : best_i; }
    __syncthreads();
    if (tid == 0) {
      float bv = am_v[0]; int bi = am_i[0];
      bool b = bi < 0;
      for (int w = 1; w < 4; ++w) {
        b |= am_i[w] < 0;
        if (am_better(am_v[w], am_i[w], bv, bi)) { bv = am_v[w]; bi = am_i[w]; }
      }
      part[blockIdx.x].v = bv;
      part[blockIdx.x].i = b ? -1 : bi;
    }
  }
}

// Launch shape: ROWS rows per group, U sweeps per batch, `grid` workgroups.
template <typename WT, int EPI, int ROWS, int U>
hipError_t launch_gemv_cfg(const WT* W, int N, int K, const float* x, const float* gain,
                           float eps, float* y, ArgmaxPart* part, int grid, hipStream_t st) {
  const size_t lds = (size_t)K * sizeof(float);
#define WICI_GEMV_NORM(NR)                                                                   \
  do {                                                                                       \
    if (lds > 65536)                                                                         \
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemv<WT, EPI, NR, ROWS, U>), \
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);       \
    hipLaunchKernelGGL((k_gemv<WT, EPI, NR, ROWS, U>), dim3(grid), dim3(256), lds, st, W, N, K, \
                       x, gain, eps, y, part);                                               \
  } while (0)
  if (gain) WICI_GEMV_NORM(true);
  else WICI_GEMV_NORM(false);
#undef WICI_GEMV_NORM
  return hipGetLastError();
}

// Launch shape per matrix: two rows per group, 4 sweeps (2 KiB of bf16 per row)
// per batch, two workgroups per CU; one workgroup per CU when the staged vector
// is too large for two.  (From a sweep of group rows {1,2,4}, sweeps per batch
// {2,4,8} and 256..1024 workgroups over the decode matrices of the 8B shape.)
struct GemvShape { int grid; };

static GemvShape gemv_shape(int N, int K) {
  GemvShape s{(size_t)K * 4 > 80 * 1024 ? 256 : 512};
  const int need = ((N + 1) / 2 + 3) / 4;  // workgroups for one group per wavefront
  if (need < s.grid) s.grid = need < 1 ? 1 : need;
  return s;
}

int gemv_argmax_blocks(int N) { return gemv_shape(N, 0).grid; }

template <typename WT, int EPI>
static hipError_t gemv_dispatch(const GemvShape& s, const WT* W, int N, int K, const float* x,
                                const float* gain, float eps, float* y, ArgmaxPart* part,
                                hipStream_t st) {
  // the same bytes per batch for both weight types
  if (sizeof(WT) == 2)
    return launch_gemv_cfg<WT, EPI, 2, 4>(W, N, K, x, gain, eps, y, part, s.grid, st);
  return launch_gemv_cfg<WT, EPI, 2, 2>(W, N, K, x, gain, eps, y, part, s.grid, st);
}

template <typename WT>
static hipError_t gemv_t(int epi, const WT* W, int N, int K, const float* x, const float* gain,
                         float eps, float* y, ArgmaxPart* part, hipStream_t st) {
  const GemvShape s = gemv_shape(N, K);
  switch (epi) {
    case GEMV_STORE: return gemv_dispatch<WT, GEMV_STORE>(s, W, N, K, x, gain, eps, y, part, st);
    case GEMV_RESID: return gemv_dispatch<WT, GEMV_RESID>(s, W, N, K, x, gain, eps, y, part, st);
    case GEMV_SWIGLU: return gemv_dispatch<WT, GEMV_SWIGLU>(s, W, N, K, x, gain, eps, y, part, st);
    case GEMV_ARGMAX: return gemv_dispatch<WT, GEMV_ARGMAX>(s, W, N, K, x, gain, eps, y, part, st);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemv(bool w_bf16, int epi, const void* W, int N, int K, const float* x,
                       const float* norm_gain, float eps, float* y, ArgmaxPart* part,
                       int* nblocks, hipStream_t st) {
  if (nblocks) *nblocks = gemv_shape(N, K).grid;
  if (w_bf16)
    return gemv_t<bf16_t>(epi, static_cast<const bf16_t*>(W), N, K, x, norm_gain, eps, y, part, st);
  return gemv_t<float>(epi, static_cast<const float*>(W), N, K, x, norm_gain, eps, y, part, st);
}

}  // namespace wici
