// Weight-streaming GEMV for the batch-1 decode step (y = W x).
//
// Decode is bound by HBM bandwidth: every weight byte is read once per token
// and used for one multiply-add.  On MI355X the DRAM side streams fastest when
// the whole chip reads one sliding, contiguous window of memory, each workgroup
// reading a contiguous block of it with a few 16-byte non-temporal loads in
// flight per lane (measured: ~7.3 TB/s with two or three 256-thread workgroups
// per CU and four loads per lane, against 5.4-6.5 TB/s for scattered row
// streams).  The kernel is shaped after that:
//  - a row group is R consecutive rows (two rows of one RoPE pair for the QKV
//    epilogue) and belongs to one workgroup: workgroup b owns groups b, b + G,
//    b + 2G, ... (G workgroups), so at any time the chip streams a band of G
//    groups and each workgroup a contiguous piece of it;
//  - all 256 lanes of the workgroup read every row of the group together: lane
//    t takes the EPL elements at t*EPL + j*256*EPL of the row (unit j), so one
//    unit of a row is 4 KiB (bf16) read by one coalesced instruction per
//    wavefront, and lane t always meets the same J slices of x: they are loaded
//    (times the norm gain) into registers once, with no LDS staging and no
//    barrier before the stream starts;
//  - a group's R x J loads are issued together and consumed together; two or
//    three workgroups per CU keep enough of them in flight (measured faster
//    than double buffering within a wavefront, which puts too many bytes in
//    flight chip-wide);
//  - each wavefront reduces its share of a group's row sums (DPP row
//    operations) and parks it in LDS; the four shares of every row are added at
//    the end, where the epilogue (residual add, SwiGLU, RoPE + KV append,
//    argmax partial) runs once per row.  An RMS-normalised input gets its
//    1/rms factor applied there (W (x g r) = r W (x g)).
//
// Every load is unconditional (addresses clamped into the matrix and the
// vector; lanes past the row end are loaded but never used).  The prologue
// issues the loads of x (and the norm gain, and the residual values this
// workgroup will update) and then the first group's weights, so they share one
// memory round trip.
#include "common.h"
#include "kernels.h"
#include "launch.h"

#include <algorithm>

namespace wici {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
// The weights one lane takes per unit: 8 bf16, 8 fp32 (two loads) or 16 Q8 codes.
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
__device__ __forceinline__ float half_to_f32(unsigned short h) {
  return (float)__builtin_bit_cast(_Float16, h);
}

constexpr int kMaxGemvK = 32768;

// Register forms of the dot products (x slices live in registers).
__device__ __forceinline__ float dot8r(const Vec8<bf16_t>& v, const float (&x)[8]) {
  return __uint_as_float(v.a.x << 16) * x[0] + __uint_as_float(v.a.x & 0xffff0000u) * x[1] +
         __uint_as_float(v.a.y << 16) * x[2] + __uint_as_float(v.a.y & 0xffff0000u) * x[3] +
         __uint_as_float(v.a.z << 16) * x[4] + __uint_as_float(v.a.z & 0xffff0000u) * x[5] +
         __uint_as_float(v.a.w << 16) * x[6] + __uint_as_float(v.a.w & 0xffff0000u) * x[7];
}
__device__ __forceinline__ float dot8r(const Vec8<float>& v, const float (&x)[8]) {
  return __uint_as_float(v.a.x) * x[0] + __uint_as_float(v.a.y) * x[1] +
         __uint_as_float(v.a.z) * x[2] + __uint_as_float(v.a.w) * x[3] +
         __uint_as_float(v.b.x) * x[4] + __uint_as_float(v.b.y) * x[5] +
         __uint_as_float(v.b.z) * x[6] + __uint_as_float(v.b.w) * x[7];
}
// 16 codes (q + 128) times 16 x values, as sum(c x); the caller subtracts
// 128 sum(x) and applies the block scale.
__device__ __forceinline__ float dot16r(const Vec8<uint8_t>& v, const float (&x)[16]) {
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const unsigned c = v.a[w];
    s += (float)(c & 0xffu) * x[4 * w] + (float)((c >> 8) & 0xffu) * x[4 * w + 1] +
         (float)((c >> 16) & 0xffu) * x[4 * w + 2] + (float)(c >> 24) * x[4 * w + 3];
  }
  return s;
}

// Rows per group for J units per row: 4-8 loads per lane per group, R even for
// SwiGLU (gate/up pairs), R = 2 for QKV (RoPE pairs).
// (Q8 rows of up to 4096 codes are one unit: 8 rows per group, 4 for SwiGLU,
// which double-buffers instead; measured on the 8B matrices.)
__host__ __device__ constexpr int gemv_rows(int epi, int J, bool q8 = false) {
  return epi == GEMV_QKV ? 2
         : epi == GEMV_SWIGLU ? (J == 1 ? 4 : 2)
         : (J == 1 ? (q8 ? 8 : 4) : J <= 4 ? 2 : 1);
}

template <typename WT, int EPI, int J, bool DB, bool EMB>
__global__ __launch_bounds__(256) void k_gemv(const WT* __restrict__ W, int N, int K,
                                              const float* __restrict__ x,
                                              const float* __restrict__ gain, float eps,
                                              float* __restrict__ y,
                                              ArgmaxPart* __restrict__ part, int max_rows,
                                              QkvRope rope,
                                              const unsigned short* __restrict__ S) {
  constexpr int R = gemv_rows(EPI, J, sizeof(WT) == 1);
  constexpr bool NORM = EPI != GEMV_RESID;   // the residual GEMVs take x as is
  // EMB (first layer's QKV projection, bf16 weights): x is the embedding row of
  // the state's token, gathered here; workgroup 0 also stores it as the residual
  // stream x (which the caller passes as `x`)
  static_assert(!EMB || (EPI == GEMV_QKV && sizeof(WT) == 2), "embedding gather: bf16 QKV only");
  constexpr bool Q8 = sizeof(WT) == 1;
  constexpr int EPL = LaneElems<WT>::n, SPAN = 256 * EPL, NF4 = EPL / 4;
  extern __shared__ float ps[];  // [4 wavefronts][max_rows] row-sum shares
  __shared__ float red[4];
  __shared__ float am_v[4];
  __shared__ int am_i[4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int G = gridDim.x, blk = blockIdx.x;
  const int ngroups = EPI == GEMV_QKV ? N / 2 : (N + R - 1) / R;
  const int my_groups = blk < ngroups ? (ngroups - 1 - blk) / G + 1 : 0;
  const int nrows = my_groups * R;  // this workgroup's rows, group by group
  // matrix row of member r of row group g: consecutive rows, or for QKV the RoPE
  // pair (j, j + hd/2) of head g / (hd/2)
  const int half = rope.kv.hd >> 1;
  auto grow = [&](int g, int r) {
    if (EPI == GEMV_QKV) {
      const int hh = g / half;
      return hh * 2 * half + (g - hh * half) + r * half;
    }
    return g * R + r;
  };
  auto lrow = [&](int i) {  // matrix row of local row i
    const int gi = i / R;
    return grow(blk + gi * G, i - gi * R);
  };
  auto kofs = [&](int j) { return min(tid * EPL + j * SPAN, K - EPL); };

  // ---- prologue: x, gain and residual loads, then the first group's weights -----
  // (EMB: the token first, the gain, the weights, then the token's embedding row)
  int etok = 0;
  if constexpr (EMB) etok = static_cast<const DecodeState*>(rope.state)->token;
  float4 xv[J][NF4], xg[NORM ? J : 1][NF4];
#pragma unroll
  for (int j = 0; j < J; ++j)
#pragma unroll
    for (int q = 0; q < NF4; ++q) {
      const int f = (kofs(j) >> 2) + q;
      if (!EMB) xv[j][q] = reinterpret_cast<const float4*>(x)[f];
      if (NORM) xg[NORM ? j : 0][q] = reinterpret_cast<const float4*>(gain)[f];
    }
  float yres = 0.f;  // residual of local row tid
  if (EPI == GEMV_RESID) yres = y[min(lrow(min(tid, max(nrows - 1, 0))), N - 1)];
  typedef Vec8<WT> WBuf[R][J];
  typedef float SBuf[R][J];
  WBuf w0, w1;
  SBuf sc0, sc1;
  // always R x J loads (rows and columns clamped)
  auto load_group = [&](WBuf& w, SBuf& sc, int g) {
#pragma unroll
    for (int r = 0; r < R; ++r) {
      const int row = min(grow(g, r), N - 1);
      const WT* wr = W + (size_t)row * K;
#pragma unroll
      for (int j = 0; j < J; ++j) {
        const int k = kofs(j);
        ld(w[r][j], wr + k);
        if (Q8) sc[r][j] = half_to_f32(S[(size_t)row * (K / 32) + k / 32]);
      }
    }
  };
  load_group(w0, sc0, blk);
  int pos = 0, phys = 0;  // QKV: the position and its KV page
  if (EPI == GEMV_QKV) {
    pos = static_cast<const DecodeState*>(rope.state)->pos;
    phys = rope.kv.table[pos / rope.kv.page];
  }
  if constexpr (EMB) {
    // a negative token (left by a failed step) reads as a zero row
    const bf16_t* er = static_cast<const bf16_t*>(rope.embed) + (size_t)max(etok, 0) * K;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(er + kofs(j));
      const bool z = etok < 0;
      xv[j][0] = make_float4(z ? 0.f : __uint_as_float(v.x << 16), z ? 0.f : __uint_as_float(v.x & 0xffff0000u),
                             z ? 0.f : __uint_as_float(v.y << 16), z ? 0.f : __uint_as_float(v.y & 0xffff0000u));
      xv[j][1] = make_float4(z ? 0.f : __uint_as_float(v.z << 16), z ? 0.f : __uint_as_float(v.z & 0xffff0000u),
                             z ? 0.f : __uint_as_float(v.w << 16), z ? 0.f : __uint_as_float(v.w & 0xffff0000u));
      if (blk == 0 && tid * EPL + j * SPAN < K) {
        float4* xo = reinterpret_cast<float4*>(const_cast<float*>(x) + kofs(j));
        xo[0] = xv[j][0];
        xo[1] = xv[j][1];
      }
    }
  }

  // x slices of this lane (times the gain; zero past the row end), their sum of
  // squares and, for Q8, 128 times their sum (the code offset)
  float xs[J][EPL];
  float xo[J];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const bool ok = tid * EPL + j * SPAN < K;
    xo[j] = 0.f;
#pragma unroll
    for (int q = 0; q < NF4; ++q) {
      float4 t = xv[j][q];
      if (NORM) {
        ss += ok ? t.x * t.x + t.y * t.y + t.z * t.z + t.w * t.w : 0.f;
        const float4 g = xg[NORM ? j : 0][q];
        t.x *= g.x; t.y *= g.y; t.z *= g.z; t.w *= g.w;
      }
      xs[j][4 * q + 0] = ok ? t.x : 0.f;
      xs[j][4 * q + 1] = ok ? t.y : 0.f;
      xs[j][4 * q + 2] = ok ? t.z : 0.f;
      xs[j][4 * q + 3] = ok ? t.w : 0.f;
    }
    if (Q8) {
#pragma unroll
      for (int e = 0; e < EPL; ++e) xo[j] += xs[j][e];
      xo[j] *= 128.f;
    }
  }
  // QKV: the rotation of this thread's pair (local group tid), used at the end
  float rc = 0.f, rs = 0.f;
  if (EPI == GEMV_QKV) {
    const int g = min(blk + min(tid, max(my_groups - 1, 0)) * G, ngroups - 1);
    const int j = g - (g / half) * half;
    rc = rope.cos_t[(size_t)pos * half + j];
    rs = rope.sin_t[(size_t)pos * half + j];
  }

  // ---- the workgroup's row groups ---------------------------------------------------
  auto use = [&](const WBuf& w, const SBuf& sc, int gi) {
    float acc[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      acc[r] = 0.f;
#pragma unroll
      for (int j = 0; j < J; ++j) {
        if constexpr (Q8) acc[r] += sc[r][j] * (dot16r(w[r][j], xs[j]) - xo[j]);
        else acc[r] += dot8r(w[r][j], xs[j]);
      }
      acc[r] = wave_sum(acc[r]);
    }
    if (lane == 0) {
#pragma unroll
      for (int r = 0; r < R; ++r) ps[wave * max_rows + gi * R + r] = acc[r];
    }
  };
  if constexpr (DB) {
    // double buffered, peeled so that both issues of the steady state are
    // unconditional: consuming a group waits for that group's loads alone
    int gi = 0;
    for (; gi + 2 < my_groups; gi += 2) {
      load_group(w1, sc1, blk + (gi + 1) * G);
      use(w0, sc0, gi);
      load_group(w0, sc0, blk + (gi + 2) * G);
      use(w1, sc1, gi + 1);
    }
    if (gi + 1 < my_groups) {
      load_group(w1, sc1, blk + (gi + 1) * G);
      use(w0, sc0, gi);
      use(w1, sc1, gi + 1);
    } else {
      use(w0, sc0, gi);
    }
  } else {
    for (int gi = 0;;) {
      use(w0, sc0, gi);
      if (++gi >= my_groups) break;
      load_group(w0, sc0, blk + gi * G);
    }
  }
  if (NORM) {
    ss = wave_sum(ss);
    if (lane == 0) red[wave] = ss;
  }
  __syncthreads();
  const float rnorm = NORM ? 1.0f / sqrtf((red[0] + red[1] + red[2] + red[3]) / (float)K + eps)
                           : 1.0f;
  auto rowsum = [&](int i) {
    return (ps[i] + ps[max_rows + i] + ps[2 * max_rows + i] + ps[3 * max_rows + i]) * rnorm;
  };

  // ---- epilogue: one thread per row (per RoPE pair for QKV) -------------------------
  if (EPI == GEMV_QKV) {
    const KvLayout& kv = rope.kv;
    const int slot = pos % kv.page;
    for (int p = tid; p < my_groups; p += 256) {
      const int g = blk + p * G, hh = g / half, j = g - hh * half;
      const float a = rowsum(2 * p), b = rowsum(2 * p + 1);
      const float c = p < 256 ? rc : rope.cos_t[(size_t)pos * half + j];
      const float sn = p < 256 ? rs : rope.sin_t[(size_t)pos * half + j];
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
  for (int i = tid; i < nrows; i += 256) {
    const int row = lrow(i);
    const float v = rowsum(i);
    if (EPI == GEMV_SWIGLU) {
      // rows (2m, 2m + 1) of the packed matrix are (gate_m, up_m); R is even
      if ((i & 1) == 0 && row + 1 < N) y[row / 2] = silu(v) * rowsum(i + 1);
    } else if (row < N) {
      if (EPI == GEMV_RESID) y[row] = (i < 256 ? yres : y[row]) + v;
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
      for (int w2 = 1; w2 < 4; ++w2) {
        bb |= am_i[w2] < 0;
        if (am_better(am_v[w2], am_i[w2], bv, bi)) { bv = am_v[w2]; bi = am_i[w2]; }
      }
      part[blk].v = bv;
      part[blk].i = bb ? -1 : bi;
    }
  }
}

// Launch shape: J = ceil(K / (256 EPL)) units per row, rounded up to an
// instantiated count (1-8, 10, 12, 14, 16; fp32 and Q8 up to 8); two workgroups
// per CU; a workgroup with at most 8 groups (16 for Q8) double-buffers them
// when the two buffers fit the registers (its groups' round trips would otherwise follow one
// another), one with more groups streams them one at a time (double buffering
// there puts too many bytes in flight) — except bf16 rows of three units
// (K = 4097..6144, the 32B shape's K = 5120), which stream at ~4.4 TB/s single
// buffered and ~6.8 double buffered whatever the group count (gate/up 127 ->
// 83 us, LM head 344 -> 229 us at 512 workgroups).  (From sweeps of 256..1536
// workgroups and single or double buffering over the decode matrices of the 8B
// and 32B shapes.)
struct GemvCfg {
  int J, grid, max_rows;
  bool db;  // double-buffered groups (few groups per workgroup)
  size_t lds;
};

static int gemv_units(int wt, int K) {
  const int epl = wt == W_Q8 ? 16 : 8;
  const int n = (K + 256 * epl - 1) / (256 * epl);
  if (n <= 8) return n;
  if (wt != W_BF16) return 0;  // beyond the fp32 / Q8 register budget
  return n <= 10 ? 10 : n <= 12 ? 12 : n <= 14 ? 14 : n <= 16 ? 16 : 0;
}

static GemvCfg gemv_cfg(int wt, int epi, int N, int K) {
  GemvCfg c{};
  c.J = gemv_units(wt, K);
  const int R = gemv_rows(epi, c.J, wt == W_Q8);
  const int ngroups = epi == GEMV_QKV ? N / 2 : (N + R - 1) / R;
  // bf16 long-row residual products (K >= 7 x 2048: the FFN down projection) on
  // 256 double-buffered workgroups: 3.6% faster than 512 in the 8B decode step
  // (sweep of 256-1024 workgroups, single and double buffering)
  const bool long_resid = wt == W_BF16 && epi == GEMV_RESID && c.J >= 7;
  const int g = long_resid ? 256 : 512;
  c.grid = std::max(1, std::min(g, ngroups));
  c.max_rows = (ngroups + c.grid - 1) / c.grid * R;
  c.db = c.max_rows / R <= (wt == W_Q8 ? 16 : long_resid ? 16 : 8) ||
         (wt == W_BF16 && c.J == 3);
  c.lds = (size_t)4 * c.max_rows * sizeof(float);
  return c;
}

template <typename WT, int EPI, int J, bool DB, bool EMB>
static hipError_t gemv_go(const GemvCfg& cf, const WT* W, int N, int K, const float* x,
                          const float* gain, float eps, float* y, ArgmaxPart* part,
                          int* nblocks, hipStream_t st, const QkvRope& rp) {
  if constexpr ((sizeof(WT) != 2 && J > 8) || (EMB && (EPI != GEMV_QKV || sizeof(WT) != 2))) {
    return hipErrorInvalidValue;
  } else {
    constexpr bool Q8 = sizeof(WT) == 1;
    const unsigned short* S =
        Q8 ? reinterpret_cast<const unsigned short*>(reinterpret_cast<const char*>(W) +
                                                     q8_scale_offset(N, K))
           : nullptr;
    // a grid larger than what is resident at once would leave a tail of late
    // workgroups: clamp it to the kernel's occupancy (queried once per kernel)
    static const int resident = [] {
      int dev = 0, cus = 0, per_cu = 0;
      if (hipGetDevice(&dev) != hipSuccess ||
          hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
          hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, k_gemv<WT, EPI, J, DB, EMB>, 256, 4096) !=
              hipSuccess)
        return 0;
      return cus * per_cu;
    }();
    (void)hipGetLastError();
    GemvCfg c = cf;
    if (resident > 0 && c.grid > resident) {
      const int R = gemv_rows(EPI, J, sizeof(WT) == 1);
      const int ngroups = EPI == GEMV_QKV ? N / 2 : (N + R - 1) / R;
      c.grid = resident;
      c.max_rows = (ngroups + c.grid - 1) / c.grid * R;
      c.lds = (size_t)4 * c.max_rows * sizeof(float);
    }
    if (nblocks) *nblocks = c.grid;
    launch_k(k_gemv<WT, EPI, J, DB, EMB>, dim3(c.grid), dim3(256), c.lds, st, kOnly, W, N, K, x, gain,
             eps, y, part, c.max_rows, rp, S);
    return hipGetLastError();
  }
}

template <typename WT, int EPI, bool EMB = false>
static hipError_t gemv_dispatch(const GemvCfg& cf, const WT* W, int N, int K, const float* x,
                                const float* gain, float eps, float* y, ArgmaxPart* part,
                                int* nblocks, hipStream_t st, const QkvRope& rp) {
  // double buffering for up to 8 units per row (4 for Q8, whose units are twice
  // as wide in x; beyond that two groups' loads do not fit the registers)
  constexpr int kDbMaxJ = sizeof(WT) == 1 ? 4 : 8;
#define WICI_J(JJ)                                                                    \
  case JJ:                                                                            \
    return cf.db && JJ <= kDbMaxJ                                                     \
               ? gemv_go<WT, EPI, JJ, (JJ <= kDbMaxJ), EMB>(cf, W, N, K, x, gain, eps, y, part, nblocks, st, rp) \
               : gemv_go<WT, EPI, JJ, false, EMB>(cf, W, N, K, x, gain, eps, y, part, nblocks, st, rp)
  switch (cf.J) {
    WICI_J(1); WICI_J(2); WICI_J(3); WICI_J(4); WICI_J(5); WICI_J(6); WICI_J(7); WICI_J(8);
    WICI_J(10); WICI_J(12); WICI_J(14); WICI_J(16);
    default: return hipErrorInvalidValue;
  }
#undef WICI_J
}

template <typename WT>
static hipError_t gemv_t(int epi, const WT* W, int N, int K, const float* x, const float* gain,
                         float eps, float* y, ArgmaxPart* part, int* nblocks, hipStream_t st,
                         const QkvRope* rope) {
  constexpr int wt = sizeof(WT) == 1 ? W_Q8 : sizeof(WT) == 2 ? W_BF16 : W_F32;
  if (K < 8 || K % 8 || K > kMaxGemvK || N < 1 || (wt == W_Q8 && K % 32) ||
      gemv_units(wt, K) == 0)
    return hipErrorInvalidValue;
  // the residual GEMVs take x as is, every other epilogue an RMS-normalised x
  if ((epi == GEMV_RESID) != (gain == nullptr)) return hipErrorInvalidValue;
  QkvRope rp{};
  rp.kv.hd = 2;  // unused outside GEMV_QKV (keeps the pair arithmetic defined)
  if (epi == GEMV_QKV) {
    if (!rope || rope->kv.hd < 2 || rope->kv.hd % 2 ||
        N != (rope->n_q + 2 * rope->kv.n_kv) * rope->kv.hd)
      return hipErrorInvalidValue;
    rp = *rope;
  }
  if (epi == GEMV_SWIGLU && N % 2) return hipErrorInvalidValue;
  const GemvCfg cf = gemv_cfg(wt, epi, N, K);
  if (epi == GEMV_QKV && rp.embed) {
    if constexpr (wt == W_BF16)
      return gemv_dispatch<WT, GEMV_QKV, true>(cf, W, N, K, x, gain, eps, y, part, nblocks, st, rp);
    else
      return hipErrorInvalidValue;
  }
#define WICI_GEMV_EPI(E) \
  case E: return gemv_dispatch<WT, E>(cf, W, N, K, x, gain, eps, y, part, nblocks, st, rp)
  switch (epi) {
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
  switch (wt) {
    case W_BF16:
      return gemv_t<bf16_t>(epi, static_cast<const bf16_t*>(W), N, K, x, norm_gain, eps, y, part,
                            nblocks, st, rope);
    case W_F32:
      return gemv_t<float>(epi, static_cast<const float*>(W), N, K, x, norm_gain, eps, y, part,
                           nblocks, st, rope);
    case W_Q8:
      return gemv_t<uint8_t>(epi, static_cast<const uint8_t*>(W), N, K, x, norm_gain, eps, y,
                             part, nblocks, st, rope);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace wici
