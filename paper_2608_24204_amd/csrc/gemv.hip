// Weight-streaming GEMV for the batch-1 decode step (y = W x).
//
// Decode is bound by HBM bandwidth: every weight byte is read once per token
// and used for one multiply-add.  The kernel therefore only has to keep enough
// 16-byte loads in flight on every CU and waste none of the bytes:
//  - a persistent grid of 256-thread workgroups; each workgroup first stages the
//    fp32 input vector in LDS (optionally RMS-normalised and scaled by the norm
//    gain, the sum of squares being recomputed per workgroup so no extra launch
//    or grid-wide reduction is needed);
//  - each wavefront owns complete rows, two at a time (a gate/up pair for the
//    SwiGLU epilogue), and streams them with 64 lanes x 16 B = 1 KiB fully
//    coalesced loads, unrolled so that up to 16 loads per lane are in flight;
//  - a row's 64 partial sums are reduced with cross-lane shuffles; there are no
//    barriers after the staging step, so wavefronts never wait for each other.
#include "common.h"
#include "kernels.h"

namespace wici {

template <typename WT, int EPI, bool NORM>
__global__ __launch_bounds__(256) void k_gemv(const WT* __restrict__ W, int N, int K,
                                              const float* __restrict__ x,
                                              const float* __restrict__ gain, float eps,
                                              float* __restrict__ y,
                                              ArgmaxPart* __restrict__ part) {
  extern __shared__ float xs[];  // K floats
  __shared__ float red[4];
  __shared__ float am_v[4];
  __shared__ int am_i[4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;

  // ---- stage x (optionally normalised) in LDS --------------------------------
  float ss = 0.f;
  for (int k = tid * 4; k < K; k += 1024) {
    float4 v = *reinterpret_cast<const float4*>(x + k);
    *reinterpret_cast<float4*>(xs + k) = v;
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  if (NORM) {
    const float tot = block256_sum(ss, red);
    const float r = 1.0f / sqrtf(tot / (float)K + eps);
    for (int k = tid * 4; k < K; k += 1024) {
      float4 v = *reinterpret_cast<float4*>(xs + k);
      float4 g = *reinterpret_cast<const float4*>(gain + k);
      v.x = v.x * r * g.x; v.y = v.y * r * g.y; v.z = v.z * r * g.z; v.w = v.w * r * g.w;
      *reinterpret_cast<float4*>(xs + k) = v;
    }
  }
  __syncthreads();

  // ---- stream row pairs --------------------------------------------------------
  const int npairs = (N + 1) >> 1;
  const int nwaves = gridDim.x * 4;
  const int nfull = K >> 9;               // full 512-element sweeps of the wave
  const bool tail = (nfull << 9) + lane * 8 < K;
  float best_v = -INFINITY;
  int best_i = 0x7fffffff;
  bool bad = false;

  for (int p = blockIdx.x * 4 + wave; p < npairs; p += nwaves) {
    const int r0 = 2 * p;
    const bool has1 = r0 + 1 < N;
    const WT* w0 = W + (size_t)r0 * K + lane * 8;
    const WT* w1 = has1 ? w0 + K : w0;
    const float* xl = xs + lane * 8;
    float a0 = 0.f, a1 = 0.f;
#pragma unroll 8
    for (int it = 0; it < nfull; ++it) {
      float u[8], v[8];
      load8(w0 + it * 512, u);
      load8(w1 + it * 512, v);
      const float4 xa = *reinterpret_cast<const float4*>(xl + it * 512);
      const float4 xb = *reinterpret_cast<const float4*>(xl + it * 512 + 4);
      a0 += u[0] * xa.x + u[1] * xa.y + u[2] * xa.z + u[3] * xa.w +
            u[4] * xb.x + u[5] * xb.y + u[6] * xb.z + u[7] * xb.w;
      a1 += v[0] * xa.x + v[1] * xa.y + v[2] * xa.z + v[3] * xa.w +
            v[4] * xb.x + v[5] * xb.y + v[6] * xb.z + v[7] * xb.w;
    }
    if (tail) {
      float u[8], v[8];
      load8(w0 + nfull * 512, u);
      load8(w1 + nfull * 512, v);
      const float* xt = xl + nfull * 512;
#pragma unroll
      for (int e = 0; e < 8; ++e) { a0 += u[e] * xt[e]; a1 += v[e] * xt[e]; }
    }
    a0 = wave_sum(a0);
    a1 = wave_sum(a1);
    if (EPI == GEMV_SWIGLU) {
      if (lane == 0) y[p] = silu(a0) * a1;
    } else if (EPI == GEMV_RESID) {
      if (lane == 0) y[r0] += a0;
      if (lane == 1 && has1) y[r0 + 1] += a1;
    } else {
      if (lane == 0) y[r0] = a0;
      if (lane == 1 && has1) y[r0 + 1] = a1;
      if (EPI == GEMV_ARGMAX) {
        // NaN never compares better; the final pass detects non-finite logits
        if (am_better(a0, r0, best_v, best_i)) { best_v = a0; best_i = r0; }
        if (has1 && am_better(a1, r0 + 1, best_v, best_i)) { best_v = a1; best_i = r0 + 1; }
        bad |= !isfinite(a0) || (has1 && !isfinite(a1));
      }
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

static int gemv_grid(int N) {
  const int npairs = (N + 1) / 2;
  int g = (npairs + 3) / 4;  // one pair per wavefront
  if (g > 1024) g = 1024;
  if (g < 1) g = 1;
  return g;
}

int gemv_argmax_blocks(int N) { return gemv_grid(N); }

template <typename WT>
static hipError_t gemv_t(int epi, const WT* W, int N, int K, const float* x,
                         const float* gain, float eps, float* y, ArgmaxPart* part,
                         hipStream_t st) {
  const int g = gemv_grid(N);
  const size_t lds = (size_t)K * sizeof(float);
  const bool nrm = gain != nullptr;
#define WICI_GEMV(E, NR)                                                                  \
  do {                                                                                    \
    if (lds > 65536)                                                                      \
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&k_gemv<WT, E, NR>),        \
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);    \
    hipLaunchKernelGGL((k_gemv<WT, E, NR>), dim3(g), dim3(256), lds, st, W, N, K, x, gain, \
                       eps, y, part);                                                     \
  } while (0)
  switch (epi) {
    case GEMV_STORE: if (nrm) WICI_GEMV(GEMV_STORE, true); else WICI_GEMV(GEMV_STORE, false); break;
    case GEMV_RESID: if (nrm) WICI_GEMV(GEMV_RESID, true); else WICI_GEMV(GEMV_RESID, false); break;
    case GEMV_SWIGLU: if (nrm) WICI_GEMV(GEMV_SWIGLU, true); else WICI_GEMV(GEMV_SWIGLU, false); break;
    case GEMV_ARGMAX: if (nrm) WICI_GEMV(GEMV_ARGMAX, true); else WICI_GEMV(GEMV_ARGMAX, false); break;
    default: return hipErrorInvalidValue;
  }
#undef WICI_GEMV
  return hipGetLastError();
}

hipError_t launch_gemv(bool w_bf16, int epi, const void* W, int N, int K, const float* x,
                       const float* norm_gain, float eps, float* y, ArgmaxPart* part,
                       int* nblocks, hipStream_t st) {
  if (nblocks) *nblocks = gemv_grid(N);
  if (w_bf16)
    return gemv_t<bf16_t>(epi, static_cast<const bf16_t*>(W), N, K, x, norm_gain, eps, y, part, st);
  return gemv_t<float>(epi, static_cast<const float*>(W), N, K, x, norm_gain, eps, y, part, st);
}

}  // namespace wici
