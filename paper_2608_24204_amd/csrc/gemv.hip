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
//    U sweeps of 512 elements; the next batch is in flight while the current
//    one is consumed (double buffering), so loads never stop at row boundaries.
//
// Vector-memory completions are counted in issue order, and the compiler can
// only wait for "all but the last n" when n is the same on every path.  So
// every load is unconditional (addresses clamped into the matrix; lanes past
// the row end are loaded but never used), finished rows go to LDS rather than
// to global memory, and the loop is peeled so that its two issues are
// unconditional: consuming a batch then waits for that batch alone, with the
// next one still in flight.  The prologue issues all loads of x (and the norm
// gain, and the residual values this wavefront will update) first, then the
// first weight batch, and waits for x alone; an RMS-normalised input gets its
// 1/rms factor applied to the finished row sums (W (x g r) = r W (x g)), so
// one barrier publishes the staged vector.  Row sums are reduced with DPP row
// operations; each wavefront writes its rows at the end.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace wici {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
// The weights one lane takes per sweep: 8 bf16, 8 fp32 (two loads) or 16 Q8 codes.
template <typename WT> struct Vec8;
template <> struct Vec8<bf16_t> { u32x4 a; };
template <> struct Vec8<float> { u32x4 a, b; };
template <> struct Vec8<uint8_t> { u32x4 a; };
template <typename WT> struct LaneElems { static constexpr int n = 8; };
template <> struct LaneElems<uint8_t> { static constexpr int n = 16; };

// Weights are read exactly once per step: non-temporal loads keep them from
// displacing the small vectors that are reused from the caches.
__device__ __forceinline__ void ld(Vec8<bf16_t>& v, const bf16_t* p) {
  v.a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
}
__device__ __forceinline__ void ld(Vec8<float>& v, const float* p) {
  v.a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  v.b = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p) + 1);
}
__device__ __forceinline__ void ld(Vec8<uint8_t>& v, const uint8_t* p) {
  v.a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
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

// 16 codes (q + 128 in bytes) times 16 x values, as sum(c x); the caller
// subtracts 128 sum(x) (precomputed per 16-element chunk) and applies the scale.
__device__ __forceinline__ float dot16(const Vec8<uint8_t>& v, const float* x) {
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float4 xv = *reinterpret_cast<const float4*>(x + 4 * w);
    const unsigned c = v.a[w];
    s += (float)(c & 0xffu) * xv.x + (float)((c >> 8) & 0xffu) * xv.y +
         (float)((c >> 16) & 0xffu) * xv.z + (float)(c >> 24) * xv.w;
  }
  return s;
}

// Batch b of a wavefront = (row group, first sweep); nsb batches per group.  Q8
// batches also carry each lane's block scale per row and sweep.
template <typename WT, int ROWS, int U>
struct Batch {
  Vec8<WT> w[ROWS][U];
  float sc[ROWS][U];
};
__device__ __forceinline__ float half_to_f32(unsigned short h) {
  return (float)__builtin_bit_cast(_Float16, h);
}

// Rounds of x staging: each round is 8 float4 per thread (8192 floats per
// workgroup), all issued before the first weight batch.
constexpr int kMaxGemvK = 32768;

template <typename WT, int EPI, bool NORM, int ROWS, int U, int XR>
__global__ __launch_bounds__(256) void k_gemv(const WT* __restrict__ W, int N, int K,
                                              const float* __restrict__ x,
                                              const float* __restrict__ gain, float eps,
                                              float* __restrict__ y,
                                              ArgmaxPart* __restrict__ part, int max_out,
                                              QkvRope rope,
                                              const unsigned short* __restrict__ S) {
  static_assert(EPI != GEMV_SWIGLU || ROWS % 2 == 0, "SwiGLU needs whole gate/up pairs");
  static_assert(EPI != GEMV_QKV || ROWS == 2, "QKV row groups are RoPE pairs");
  constexpr int OPG = EPI == GEMV_SWIGLU ? ROWS / 2 : ROWS;  // outputs per row group
  constexpr bool Q8 = sizeof(WT) == 1;
  constexpr int EPL = LaneElems<WT>::n, SW = 64 * EPL;      // elements per lane / sweep
  extern __shared__ float smem[];
  float* xs = smem;                          // K floats: x * gain
  float* xsum = smem + K;                    // Q8: sum of each 16 elements of xs
  float* ys = smem + K + (Q8 ? K / 16 : 0);  // [4 wavefronts][max_out] finished outputs
  __shared__ float red[4];
  __shared__ float am_v[4];
  __shared__ int am_i[4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int nsweep = (K + SW - 1) / SW;       // sweeps per row
  const int nsb = (nsweep + U - 1) / U;       // batches per row group
  const int ngroups = (N + ROWS - 1) / ROWS;
  const int wid = blockIdx.x * 4 + wave, nw = gridDim.x * 4;
  const int my_groups = wid < ngroups ? (ngroups - 1 - wid) / nw + 1 : 0;
  const int nbatch = my_groups * nsb;
  const int nout = my_groups * OPG;
  const int nf4 = K >> 2;
  // global row (or SwiGLU output) index of this wavefront's output j
  auto out_row = [&](int j) {
    const int gi = j / OPG, o = j - gi * OPG;
    return EPI == GEMV_SWIGLU ? (wid + gi * nw) * OPG + o : (wid + gi * nw) * ROWS + o;
  };
  const int n_rows_out = EPI == GEMV_SWIGLU ? N / 2 : N;

  // matrix row of member r of row group g: consecutive rows, or for QKV the RoPE
  // pair (j, j + hd/2) of head g / (hd/2)
  const int half = rope.kv.hd >> 1;
  auto grow = [&](int g, int r) {
    if (EPI == GEMV_QKV) {
      const int hh = g / half;
      return hh * 2 * half + (g - hh * half) + r * half;
    }
    return g * ROWS + r;
  };

  // issue batch b into buf: always ROWS x U loads (row and column clamped)
  auto issue = [&](Batch<WT, ROWS, U>& buf, int b) {
    const int gi = b / nsb, s0 = (b - gi * nsb) * U;
    const int g = wid + gi * nw;
#pragma unroll
    for (int r = 0; r < ROWS; ++r) {
      const WT* wr = W + (size_t)min(grow(g, r), N - 1) * K;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int k = min((s0 + u) * SW + lane * EPL, K - EPL);
        ld(buf.w[r][u], wr + k);
        if (Q8)
          buf.sc[r][u] = half_to_f32(S[(size_t)min(grow(g, r), N - 1) * (K / 32) + k / 32]);
      }
    }
  };

  // ---- prologue: x, gain and residual loads, then the first weight batch ----------
  float4 xv[XR][8], xg[NORM ? XR : 1][8];
#pragma unroll
  for (int r = 0; r < XR; ++r)
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int f = min(r * 2048 + u * 256 + tid, nf4 - 1);
      xv[r][u] = reinterpret_cast<const float4*>(x)[f];
      if (NORM) xg[NORM ? r : 0][u] = reinterpret_cast<const float4*>(gain)[f];
    }
  float yres = 0.f;
  if (EPI == GEMV_RESID) yres = y[min(out_row(lane), n_rows_out - 1)];
  Batch<WT, ROWS, U> b0, b1;
  issue(b0, 0);
  // QKV: the position, its KV page, and this lane's rotation (group `lane`)
  int pos = 0, phys = 0;
  float rc = 0.f, rs = 0.f;
  if (EPI == GEMV_QKV) {
    pos = static_cast<const DecodeState*>(rope.state)->pos;
    phys = rope.kv.table[pos / rope.kv.page];
    const int g = min(wid + lane * nw, ngroups - 1);
    const int j = g - (g / half) * half;
    rc = rope.cos_t[(size_t)pos * half + j];
    rs = rope.sin_t[(size_t)pos * half + j];
  }

  float ss = 0.f;
#pragma unroll
  for (int r = 0; r < XR; ++r)
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int f = r * 2048 + u * 256 + tid;
      if (f < nf4) {
        float4 t = xv[r][u];
        if (NORM) {
          const float4 g = xg[NORM ? r : 0][u];
          ss += t.x * t.x + t.y * t.y + t.z * t.z + t.w * t.w;
          t.x *= g.x; t.y *= g.y; t.z *= g.z; t.w *= g.w;
        }
        reinterpret_cast<float4*>(xs)[f] = t;
      }
    }
  if (NORM) {
    ss = wave_sum(ss);
    if (lane == 0) red[wave] = ss;
  }
  __syncthreads();
  if (Q8) {  // block sums of the staged vector for the code offset
    for (int c = tid; c < K / 16; c += 256) {
      float t = 0.f;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float4 v = reinterpret_cast<const float4*>(xs)[c * 4 + w];
        t += (v.x + v.y) + (v.z + v.w);
      }
      xsum[c] = t;
    }
    __syncthreads();
  }
  const float rnorm = NORM ? 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)K + eps)
                           : 1.0f;

  float acc[ROWS];
#pragma unroll
  for (int r = 0; r < ROWS; ++r) acc[r] = 0.f;
  float* yw = ys + wave * max_out;

  auto consume = [&](const Batch<WT, ROWS, U>& buf, int b) {
    const int gi = b / nsb, sb = b - gi * nsb, s0 = sb * U;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int k = (s0 + u) * SW + lane * EPL;
      if (k < K) {
        const float* xk = xs + k;
        if constexpr (Q8) {
          const float off = 128.f * xsum[k / 16];
#pragma unroll
          for (int r = 0; r < ROWS; ++r) acc[r] += buf.sc[r][u] * (dot16(buf.w[r][u], xk) - off);
        } else {
#pragma unroll
          for (int r = 0; r < ROWS; ++r) acc[r] += dot8(buf.w[r][u], xk);
        }
      }
    }
    if (sb == nsb - 1) {  // row group complete
#pragma unroll
      for (int r = 0; r < ROWS; ++r) acc[r] = wave_sum(acc[r]) * rnorm;
      if (lane == 0) {
        if (EPI == GEMV_SWIGLU) {
#pragma unroll
          for (int r = 0; r < ROWS; r += 2) yw[gi * OPG + r / 2] = silu(acc[r]) * acc[r + 1];
        } else {
#pragma unroll
          for (int r = 0; r < ROWS; ++r) yw[gi * OPG + r] = acc[r];
        }
      }
#pragma unroll
      for (int r = 0; r < ROWS; ++r) acc[r] = 0.f;
    }
  };

  // ---- double-buffered stream of batches (steady state: unconditional issues) -----
  int b = 0;
  for (; b + 2 < nbatch; b += 2) {
    issue(b1, b + 1);
    consume(b0, b);
    issue(b0, b + 2);
    consume(b1, b + 1);
  }
  if (b + 1 < nbatch) {
    issue(b1, b + 1);
    consume(b0, b);
    consume(b1, b + 1);
  } else if (b < nbatch) {
    consume(b0, b);
  }

  // ---- outputs of this wavefront (its own LDS slots: no barrier needed) -----------
  if (EPI == GEMV_QKV) {
    const KvLayout& kv = rope.kv;
    const int slot = pos % kv.page;
    for (int gi = lane; gi < my_groups; gi += 64) {
      const int g = wid + gi * nw, hh = g / half, j = g - hh * half;
      const float a = yw[2 * gi], b = yw[2 * gi + 1];
      const float c = gi < 64 ? rc : rope.cos_t[(size_t)pos * half + j];
      const float sn = gi < 64 ? rs : rope.sin_t[(size_t)pos * half + j];
      if (hh < rope.n_q) {
        y[(size_t)hh * 2 * half + j] = (a * c - b * sn) * rope.q_scale;
        y[(size_t)hh * 2 * half + j + half] = (a * sn + b * c) * rope.q_scale;
      } else {
        const int which = hh < rope.n_q + kv.n_kv ? 0 : 1;  // key or value head
        const int h = hh - rope.n_q - which * kv.n_kv;
        const float va = which ? a : a * c - b * sn, vb = which ? b : a * sn + b * c;
        const size_t off =
            ((((size_t)phys * 2 + which) * kv.n_kv + h) * kv.page + slot) * kv.hd + j;
        if (rope.kv_bf16) {
          bf16_t* d = static_cast<bf16_t*>(kv.base) + off;
          d[0] = f32_to_bf16(va);
          d[half] = f32_to_bf16(vb);
        } else {
          float* d = static_cast<float*>(kv.base) + off;
          d[0] = va;
          d[half] = vb;
        }
      }
    }
    return;
  }
  float best_v = -INFINITY;
  int best_i = 0x7fffffff;
  bool bad = false;
  for (int j = lane; j < nout; j += 64) {
    const int row = out_row(j);
    const float v = yw[j];
    if (row < n_rows_out) {
      if (EPI == GEMV_RESID) y[row] = (j < 64 ? yres : y[row]) + v;
      else y[row] = v;
      if (EPI == GEMV_ARGMAX) {
        // NaN never compares better; a non-finite logit is flagged separately
        if (am_better(v, row, best_v, best_i)) { best_v = v; best_i = row; }
        bad |= !isfinite(v);
      }
    }
  }
  if (EPI == GEMV_ARGMAX) {
    // (value, lowest index) over the workgroup; a non-finite logit marks the
    // partial with index -1
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const float ov = __shfl_xor(best_v, m);
      const int oi = __shfl_xor(best_i, m);
      if (am_better(ov, oi, best_v, best_i)) { best_v = ov; best_i = oi; }
      bad |= __shfl_xor((int)bad, m) != 0;
    }
    if (lane == 0) { am_v[wave] = best_v; am_i[wave] = bad ? -1 : best_i; }
    __syncthreads();
    if (tid == 0) {
      float bv = am_v[0]; int bi = am_i[0];
      bool bb = bi < 0;
      for (int w = 1; w < 4; ++w) {
        bb |= am_i[w] < 0;
        if (am_better(am_v[w], am_i[w], bv, bi)) { bv = am_v[w]; bi = am_i[w]; }
      }
      part[blockIdx.x].v = bv;
      part[blockIdx.x].i = bb ? -1 : bi;
    }
  }
}

// Launch shape: ROWS rows per group, U sweeps per batch, `grid` workgroups.
template <typename WT, int EPI, int ROWS, int U>
hipError_t launch_gemv_cfg(const WT* W, int N, int K, const float* x, const float* gain,
                           float eps, float* y, ArgmaxPart* part, int grid, hipStream_t st,
                           const QkvRope* rope = nullptr) {
  if (K < 8 || K % 8 || K > kMaxGemvK || N < 1 || grid < 1) return hipErrorInvalidValue;
  QkvRope rp{};
  rp.kv.hd = 2;  // unused outside GEMV_QKV (keeps the pair arithmetic defined)
  if (EPI == GEMV_QKV) {
    if (!rope || rope->kv.hd < 2 || rope->kv.hd % 2 || N != (rope->n_q + 2 * rope->kv.n_kv) * rope->kv.hd)
      return hipErrorInvalidValue;
    rp = *rope;
  }
  constexpr int OPG = EPI == GEMV_SWIGLU ? ROWS / 2 : ROWS;
  const int ngroups = (N + ROWS - 1) / ROWS, nw = grid * 4;
  const int max_out = (ngroups + nw - 1) / nw * OPG;
  constexpr bool Q8 = sizeof(WT) == 1;
  if (Q8 && K % 32) return hipErrorInvalidValue;
  const size_t lds = ((size_t)K + (Q8 ? K / 16 : 0) + 4 * (size_t)max_out) * sizeof(float);
  const unsigned short* S =
      Q8 ? reinterpret_cast<const unsigned short*>(reinterpret_cast<const char*>(W) +
                                                   q8_scale_offset(N, K))
         : nullptr;
  const int xr = K <= 8192 ? 1 : K <= 16384 ? 2 : 4;
#define WICI_GEMV_GO(NR, XR)                                                                 \
  do {                                                                                       \
    auto fn = &k_gemv<WT, EPI, NR, ROWS, U, XR>;                                             \
    if (lds > 65536)                                                                         \
      (void)hipFuncSetAttribute(reinterpret_cast<const void*>(fn),                           \
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);       \
    launch_k(fn, dim3(grid), dim3(256), lds, st, kOnly, W, N, K, x, gain, eps, y, part,      \
             max_out, rp, S);                                                                \
  } while (0)
#define WICI_GEMV_XR(NR)                   \
  do {                                     \
    if (xr == 1) WICI_GEMV_GO(NR, 1);      \
    else if (xr == 2) WICI_GEMV_GO(NR, 2); \
    else WICI_GEMV_GO(NR, 4);              \
  } while (0)
  if (gain) WICI_GEMV_XR(true);
  else WICI_GEMV_XR(false);
#undef WICI_GEMV_XR
#undef WICI_GEMV_GO
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
                                hipStream_t st, const QkvRope* rope) {
  // 16-byte loads per lane: 4 sweeps per batch for bf16 (2 KiB per row), 2 for
  // fp32 (two loads per sweep) and for Q8 (2 KiB of codes per row, plus the
  // scales; measured faster than 4 on every 8B matrix, by 0.3-1.3 us)
  if (sizeof(WT) == 2)
    return launch_gemv_cfg<WT, EPI, 2, 4>(W, N, K, x, gain, eps, y, part, s.grid, st, rope);
  return launch_gemv_cfg<WT, EPI, 2, 2>(W, N, K, x, gain, eps, y, part, s.grid, st, rope);
}

template <typename WT>
static hipError_t gemv_t(int epi, const WT* W, int N, int K, const float* x, const float* gain,
                         float eps, float* y, ArgmaxPart* part, hipStream_t st,
                         const QkvRope* rope) {
  const GemvShape s = gemv_shape(N, K);
#define WICI_GEMV_EPI(E) \
  case E: return gemv_dispatch<WT, E>(s, W, N, K, x, gain, eps, y, part, st, rope)
  switch (epi) {
    WICI_GEMV_EPI(GEMV_STORE);
    WICI_GEMV_EPI(GEMV_RESID);
    WICI_GEMV_EPI(GEMV_SWIGLU);
    WICI_GEMV_EPI(GEMV_ARGMAX);
    WICI_GEMV_EPI(GEMV_QKV);
    default: return hipErrorInvalidValue;
  }
#undef WICI_GEMV_EPI
}

hipError_t launch_gemv(int wt, int epi, const void* W, int N, int K, const float* x,
                       const float* norm_gain, float eps, float* y, ArgmaxPart* part,
                       int* nblocks, hipStream_t st, const QkvRope* rope) {
  if (nblocks) *nblocks = gemv_shape(N, K).grid;
  switch (wt) {
    case W_BF16:
      return gemv_t<bf16_t>(epi, static_cast<const bf16_t*>(W), N, K, x, norm_gain, eps, y, part,
                            st, rope);
    case W_F32:
      return gemv_t<float>(epi, static_cast<const float*>(W), N, K, x, norm_gain, eps, y, part,
                           st, rope);
    case W_Q8:
      return gemv_t<uint8_t>(epi, static_cast<const uint8_t*>(W), N, K, x, norm_gain, eps, y,
                             part, st, rope);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace wici
