// Prefill projections: C[M, N] = A[M, K] x W[N, K]^T with fused epilogues.
//
// A holds fp32 activations (one row per prompt position), W the bf16 weights in
// their [out, in] layout, so both operands are contiguous along K, which is the
// layout the gfx950 bf16 matrix cores consume (8 consecutive K values per lane).
//
// MFMA kernel: 128x128 output tile per 256-thread block (2x2 wavefronts of
// 64x64, each a 4x4 grid of v_mfma_f32_16x16x32_bf16 tiles), K steps of 32
// staged through LDS with the next step's global loads issued before the
// current step's matrix ops.  The fp32 activations are converted to bf16 while
// being staged; in the split mode each value a is stored as hi = bf16(a) and
// lo = bf16(a - hi) and both are multiplied with the (exact) bf16 weights, which
// keeps the product accurate to about 2^-16 relative instead of 2^-8.
//
// Vector kernel: plain fp32 64x64 tiles, for fp32 weights.
#include "common.h"
#include "kernels.h"

namespace wici {

template <int EPI>
__device__ __forceinline__ void epi_store(float* C, int ldc, int M, int N, int m, int n,
                                          float v, float other) {
  if (m >= M || n >= N) return;
  if (EPI == GEMV_STORE) C[(size_t)m * ldc + n] = v;
  else if (EPI == GEMV_RESID) C[(size_t)m * ldc + n] += v;
  else if (EPI == GEMV_SWIGLU) {
    if (!(n & 1)) C[(size_t)m * ldc + (n >> 1)] = silu(v) * other;
  }
}

// --------------------------------------------------------------------- MFMA
template <bool SPLIT, int EPI>
__global__ __launch_bounds__(256) void k_gemm_mfma(const float* __restrict__ A, int lda,
                                                   const bf16_t* __restrict__ W, int M, int N,
                                                   int K, float* __restrict__ C, int ldc) {
  constexpr int BM = 128, BN = 128, BK = 32, LDK = BK + 8;
  __shared__ __attribute__((aligned(16))) bf16_t As[BM][LDK];
  __shared__ __attribute__((aligned(16))) bf16_t Al[SPLIT ? BM : 1][LDK];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[BN][LDK];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int wm = wave >> 1, wn = wave & 1;

  const int lrow = tid >> 1, lk = (tid & 1) * 16;
  const bool a_ok = m0 + lrow < M, w_ok = n0 + lrow < N;
  const float* Ap = A + (size_t)(a_ok ? m0 + lrow : 0) * lda + lk;
  const bf16_t* Wp = W + (size_t)(w_ok ? n0 + lrow : 0) * K + lk;

  float4 ra[4];
  uint4 rw[2];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      ra[i] = a_ok ? *reinterpret_cast<const float4*>(Ap + k0 + 4 * i) : make_float4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      rw[i] = w_ok ? *reinterpret_cast<const uint4*>(Wp + k0 + 8 * i) : make_uint4(0, 0, 0, 0);
  };
  auto sstore = [&]() {
    const float* f = reinterpret_cast<const float*>(ra);
    uint32_t hi[8], lo[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const bf16_t h0 = f32_to_bf16(f[2 * i]), h1 = f32_to_bf16(f[2 * i + 1]);
      hi[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
      if (SPLIT) {
        const bf16_t l0 = f32_to_bf16(f[2 * i] - bf16_to_f32(h0));
        const bf16_t l1 = f32_to_bf16(f[2 * i + 1] - bf16_to_f32(h1));
        lo[i] = (uint32_t)l0 | ((uint32_t)l1 << 16);
      }
    }
    *reinterpret_cast<uint4*>(&As[lrow][lk]) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
    *reinterpret_cast<uint4*>(&As[lrow][lk + 8]) = make_uint4(hi[4], hi[5], hi[6], hi[7]);
    if (SPLIT) {
      *reinterpret_cast<uint4*>(&Al[lrow][lk]) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
      *reinterpret_cast<uint4*>(&Al[lrow][lk + 8]) = make_uint4(lo[4], lo[5], lo[6], lo[7]);
    }
    *reinterpret_cast<uint4*>(&Bs[lrow][lk]) = rw[0];
    *reinterpret_cast<uint4*>(&Bs[lrow][lk + 8]) = rw[1];
  };

  floatx4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  const int fr = lane & 15, fk = (lane >> 4) * 8;
  gload(0);
  for (int k0 = 0; k0 < K; k0 += BK) {
    __syncthreads();
    sstore();
    __syncthreads();
    if (k0 + BK < K) gload(k0 + BK);
    bf16x8_t af[4], al[4], bfr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      af[i] = *reinterpret_cast<const bf16x8_t*>(&As[wm * 64 + i * 16 + fr][fk]);
      if (SPLIT) al[i] = *reinterpret_cast<const bf16x8_t*>(&Al[wm * 64 + i * 16 + fr][fk]);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
      bfr[j] = *reinterpret_cast<const bf16x8_t*>(&Bs[wn * 64 + j * 16 + fr][fk]);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        if (SPLIT)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[i], bfr[j], acc[i][j], 0, 0, 0);
      }
  }

  // lane holds rows 4*(lane/16)+r and column lane%16 of each 16x16 tile
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm * 64 + i * 16 + (lane >> 4) * 4 + r;
        const int n = n0 + wn * 64 + j * 16 + (lane & 15);
        const float v = acc[i][j][r];
        const float o = EPI == GEMV_SWIGLU ? __shfl_xor(v, 1) : 0.f;
        epi_store<EPI>(C, ldc, M, N, m, n, v, o);
      }
}

// ------------------------------------------------------------------- vector fp32
template <typename WT, int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ A, int lda,
                                                  const WT* __restrict__ W, int M, int N, int K,
                                                  float* __restrict__ C, int ldc) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float As[BK][BM + 4];
  __shared__ float Ws[BK][BN + 4];
  const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  const int lr = tid >> 2, lk = (tid & 3) * 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += BK) {
    const int am = m0 + lr, wn = n0 + lr;
    float4 a = am < M ? *reinterpret_cast<const float4*>(A + (size_t)am * lda + k0 + lk)
                      : make_float4(0, 0, 0, 0);
    float w[4];
    if (wn < N) {
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = Elem<WT>::load(W + (size_t)wn * K + k0 + lk + e);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) w[e] = 0.f;
    }
    __syncthreads();
    As[lk + 0][lr] = a.x; As[lk + 1][lr] = a.y; As[lk + 2][lr] = a.z; As[lk + 3][lr] = a.w;
#pragma unroll
    for (int e = 0; e < 4; ++e) Ws[lk + e][lr] = w[e];
    __syncthreads();
#pragma unroll
    for (int k = 0; k < BK; ++k) {
      float av[4], wv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) { av[i] = As[k][ty * 4 + i]; wv[i] = Ws[k][tx * 4 + i]; }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += av[i] * wv[j];
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
      epi_store<EPI>(C, ldc, M, N, m, n, acc[i][j], (j & 1) ? 0.f : acc[i][j + 1 < 4 ? j + 1 : j]);
    }
}

template <bool SPLIT>
static hipError_t gemm_mfma_t(int epi, const float* A, int lda, const bf16_t* W, int M, int N,
                              int K, float* C, int ldc, hipStream_t st) {
  dim3 grid((N + 127) / 128, (M + 127) / 128);
  switch (epi) {
    case GEMV_STORE:
      hipLaunchKernelGGL((k_gemm_mfma<SPLIT, GEMV_STORE>), grid, dim3(256), 0, st, A, lda, W, M, N, K, C, ldc);
      break;
    case GEMV_RESID:
      hipLaunchKernelGGL((k_gemm_mfma<SPLIT, GEMV_RESID>), grid, dim3(256), 0, st, A, lda, W, M, N, K, C, ldc);
      break;
    case GEMV_SWIGLU:
      hipLaunchKernelGGL((k_gemm_mfma<SPLIT, GEMV_SWIGLU>), grid, dim3(256), 0, st, A, lda, W, M, N, K, C, ldc);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename WT>
static hipError_t gemm_f32_t(int epi, const float* A, int lda, const WT* W, int M, int N, int K,
                             float* C, int ldc, hipStream_t st) {
  dim3 grid((N + 63) / 64, (M + 63) / 64);
  switch (epi) {
    case GEMV_STORE:
      hipLaunchKernelGGL((k_gemm_f32<WT, GEMV_STORE>), grid, dim3(256), 0, st, A, lda, W, M, N, K, C, ldc);
      break;
    case GEMV_RESID:
      hipLaunchKernelGGL((k_gemm_f32<WT, GEMV_RESID>), grid, dim3(256), 0, st, A, lda, W, M, N, K, C, ldc);
      break;
    case GEMV_SWIGLU:
      hipLaunchKernelGGL((k_gemm_f32<WT, GEMV_SWIGLU>), grid, dim3(256), 0, st, A, lda, W, M, N, K, C, ldc);
      break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(int mode, bool w_bf16, int epi, const float* A, int lda, const void* W,
                       int M, int N, int K, float* C, int ldc, hipStream_t st) {
  if (mode == 0 || mode == 1) {
    if (!w_bf16) return hipErrorInvalidValue;
    const bf16_t* Wb = static_cast<const bf16_t*>(W);
    return mode == 0 ? gemm_mfma_t<true>(epi, A, lda, Wb, M, N, K, C, ldc, st)
                     : gemm_mfma_t<false>(epi, A, lda, Wb, M, N, K, C, ldc, st);
  }
  if (w_bf16)
    return gemm_f32_t<bf16_t>(epi, A, lda, static_cast<const bf16_t*>(W), M, N, K, C, ldc, st);
  return gemm_f32_t<float>(epi, A, lda, static_cast<const float*>(W), M, N, K, C, ldc, st);
}

}  // namespace wici
