// Prefill projections: C[M, N] = A[M, K] x W[N, K]^T with fused epilogues.
//
// A holds activations (one row per prompt position), W the bf16 weights in their
// [out, in] layout, so both operands are contiguous along K, which is the layout
// the gfx950 matrix cores consume (8 consecutive K values per lane).
//
// MFMA kernel.  A arrives as NT bf16 planes whose sum is the fp32 activation
// (see ActBuf); the weights are exact bf16, so the kernel accumulates the NT
// products A_p W^T with v_mfma_f32_16x16x32_bf16 and the result carries the
// activation's precision, not bf16's.  Tiling:
//  - a block of WM x WN wavefronts owns a (64 WM) x (64 WN) output tile, each
//    wavefront a 64 x 64 sub-tile (4 x 4 matrix-core tiles, 64 accumulator
//    registers);
//  - both operands are staged through LDS in 32-deep K steps, double-buffered
//    (64-byte rows with the 16-byte chunks XOR-swizzled by row, so that neither
//    the stores nor the fragment reads hit the same bank twice); the next
//    step's global loads are in flight while the current step's matrix ops run,
//    one barrier a step;
//  - tiles are numbered A-tile-row-major and dealt to the 8 XCDs in contiguous
//    ranges (workgroups are dispatched round-robin over XCDs), so the blocks
//    resident on one XCD share an A row-tile through that XCD's L2.
// Two variants: bf16 weights go straight from global memory into LDS (k_gemm_dma);
// 8-bit weights pass through registers, where their codes become bf16 values
// (k_gemm_mfma).
//
// Vector kernel: plain fp32 64x64 tiles, for fp32 weights / fp32 activations.
#include "common.h"
#include "kernels.h"

#include <algorithm>

namespace wici {

// ------------------------------------------------------------------ epilogue
// The value of the lane's neighbour across bit 0 of the lane index: in a matrix-core
// result tile lane l holds column l % 16, so this is the SwiGLU partner (gate 2i,
// up 2i + 1).  A DPP quad permutation [1, 0, 3, 2] (a register move, where a
// shuffle goes through the LDS permute unit).
__device__ __forceinline__ float pair_swap(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
}

template <int EPI>
__device__ __forceinline__ void epi_out(float* C, int ldc, const ActBuf& H, int ldh, int M,
                                        int N, int m, int n, float v, float other) {
  if (m >= M || n >= N) return;
  if (EPI == GEMV_STORE) C[(size_t)m * ldc + n] = v;
  else if (EPI == GEMV_RESID) C[(size_t)m * ldc + n] += v;
  else if (EPI == GEMV_SWIGLU) {
    if (!(n & 1)) store_act(H, (size_t)m * ldh + (n >> 1), silu(v) * other);
  }
}

// --------------------------------------------------------------------- MFMA
constexpr int kBK = 32;   // K per step (one v_mfma_f32_16x16x32_bf16 depth)
constexpr int kLDK = 32;  // LDS row (bf16 elements): 64 bytes, four 16-byte chunks

// LDS position (bf16 elements) of 16-byte chunk `chunk` of tile row `row`: the chunk
// index is XOR-ed with bits 2-3 of the row.  Sixteen lanes that store together
// (4 consecutive rows x 4 chunks, as loaded from global memory) then cover four
// disjoint 64-byte bank ranges, and sixteen lanes that read a fragment (16 rows,
// one chunk) cover all 64 banks once: neither access conflicts.
__device__ __forceinline__ int lds_swz(int row) { return (row >> 2) & 3; }
__device__ __forceinline__ int lds_chunk(int row, int chunk) {
  return row * kLDK + 8 * (chunk ^ lds_swz(row));
}

// Q8 weights: a step of 32 along K is one quantisation block, so the codes go
// through the matrix cores exactly (an integer in [-127, 127] is a bf16 value),
// the NT products of a step are summed in a fresh accumulator, and that sum is
// multiplied by the column's block scale and added: one scale multiply per
// step and output, the products staying exact.
template <int NT, int WM, int WN, int EPI, bool Q8>
__global__ __launch_bounds__(64 * WM * WN) void k_gemm_mfma(
    const bf16_t* __restrict__ A, size_t a_plane, int lda, const void* __restrict__ Wv, int M,
    int N, int K, int ks, float* __restrict__ C, size_t c_split, int ldc, ActBuf H, int ldh,
    const unsigned short* __restrict__ S) {
  constexpr int BM = 64 * WM, BN = 64 * WN, NTH = 64 * WM * WN;
  constexpr int A_CHUNKS = NT * BM * (kBK / 8);  // 16-byte chunks per step
  constexpr int W_CHUNKS = BN * (Q8 ? kBK / 16 : kBK / 8);
  constexpr int WCPR = Q8 ? 2 : 4;               // weight chunks per row and step
  const bf16_t* W = static_cast<const bf16_t*>(Wv);
  const uint8_t* Wq = static_cast<const uint8_t*>(Wv);
  constexpr int A_PER = (A_CHUNKS + NTH - 1) / NTH;
  constexpr int W_PER = (W_CHUNKS + NTH - 1) / NTH;
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];
  bf16_t* As = smem;                            // [2][NT][BM][kLDK]
  bf16_t* Bs = smem + 2 * NT * BM * kLDK;       // [2][BN][kLDK]

  // ---- tile of this block (A-row-major tile order, contiguous ranges per XCD) ----
  const int n_mt = (M + BM - 1) / BM, n_nt = (N + BN - 1) / BN, T = n_mt * n_nt;
  const int per_xcd = (T + 7) / 8;
  const int t = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
  if (t >= T) return;
  const int m0 = (t / n_nt) * BM, n0 = (t % n_nt) * BN;
  // split K: block row y of the grid takes K range [y ks, (y + 1) ks) and writes
  // its own output (c_split elements further on)
  const int kbeg = blockIdx.y * ks;
  C += blockIdx.y * c_split;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave / WN, wn = wave % WN;

  uint4 ra[A_PER], rw[W_PER];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
      const int c = tid + i * NTH;
      if (c < A_CHUNKS) {
        const int p = c / (BM * 4), row = (c / 4) % BM, part = c % 4;
        const int m = m0 + row;
        ra[i] = m < M ? *reinterpret_cast<const uint4*>(A + p * a_plane + (size_t)m * lda + kbeg + k0 + part * 8)
                      : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int i = 0; i < W_PER; ++i) {
      const int c = tid + i * NTH;
      if (c < W_CHUNKS) {
        const int row = c / WCPR, part = c % WCPR, n = n0 + row;
        if (Q8)
          rw[i] = n < N ? *reinterpret_cast<const uint4*>(Wq + (size_t)n * K + kbeg + k0 + part * 16)
                        : make_uint4(0x80808080u, 0x80808080u, 0x80808080u, 0x80808080u);
        else
          rw[i] = n < N ? *reinterpret_cast<const uint4*>(W + (size_t)n * K + kbeg + k0 + part * 8)
                        : make_uint4(0, 0, 0, 0);
      }
    }
  };
  // Q8: the block scales of this lane's four output columns for step kt, loaded
  // one step ahead together with that step's tiles
  const int fr = lane & 15, fk = (lane >> 4) * 8;
  unsigned short scq[4];
  float scn[4];
  auto sload = [&](int kt) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = min(n0 + wn * 64 + j * 16 + fr, N - 1);
      scq[j] = S[(size_t)n * (K / 32) + kbeg / 32 + kt];
    }
  };
  auto sfix = [&]() {
#pragma unroll
    for (int j = 0; j < 4; ++j) scn[j] = (float)__builtin_bit_cast(_Float16, scq[j]);
  };
  auto sstore = [&](int s) {
#pragma unroll
    for (int i = 0; i < A_PER; ++i) {
      const int c = tid + i * NTH;
      if (c < A_CHUNKS) {
        const int p = c / (BM * 4), row = (c / 4) % BM, part = c % 4;
        *reinterpret_cast<uint4*>(As + ((size_t)s * NT + p) * BM * kLDK + lds_chunk(row, part)) = ra[i];
      }
    }
#pragma unroll
    for (int i = 0; i < W_PER; ++i) {
      const int c = tid + i * NTH;
      if (c < W_CHUNKS) {
        const int row = c / WCPR, part = c % WCPR;
        if (Q8) {
          // 16 codes -> 16 bf16 values (code - 128, exact)
          unsigned o[8];
          const unsigned wv[4] = {rw[i].x, rw[i].y, rw[i].z, rw[i].w};
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const unsigned w = wv[e / 2], sh = 16 * (e & 1);
            const float lo = (float)((w >> sh) & 0xffu) - 128.f;
            const float hi = (float)((w >> (sh + 8)) & 0xffu) - 128.f;
            o[e] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xffff0000u);
          }
          bf16_t* bt = Bs + (size_t)s * BN * kLDK;
          *reinterpret_cast<uint4*>(bt + lds_chunk(row, 2 * part)) = make_uint4(o[0], o[1], o[2], o[3]);
          *reinterpret_cast<uint4*>(bt + lds_chunk(row, 2 * part + 1)) = make_uint4(o[4], o[5], o[6], o[7]);
        } else {
          *reinterpret_cast<uint4*>(Bs + (size_t)s * BN * kLDK + lds_chunk(row, part)) = rw[i];
        }
      }
    }
  };

  floatx4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};

  const int KT = ks / kBK;
  if (Q8) sload(0);
  gload(0);
  sstore(0);
  if (Q8) sfix();
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int s = kt & 1;
    if (kt + 1 < KT) {
      if (Q8) sload(kt + 1);
      gload((kt + 1) * kBK);
    }
    bf16x8_t bfr[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      bfr[j] = *reinterpret_cast<const bf16x8_t*>(Bs + (size_t)s * BN * kLDK +
                                                  lds_chunk(wn * 64 + j * 16 + fr, fk / 8));
    if constexpr (Q8) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        floatx4_t part[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) part[j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int p = 0; p < NT; ++p) {
          const bf16x8_t af = *reinterpret_cast<const bf16x8_t*>(
              As + ((size_t)s * NT + p) * BM * kLDK + lds_chunk(wm * 64 + i * 16 + fr, fk / 8));
#pragma unroll
          for (int j = 0; j < 4; ++j)
            part[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bfr[j], part[j], 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[i][j][r] += part[j][r] * scn[j];
      }
    } else {
#pragma unroll
      for (int p = 0; p < NT; ++p) {
        bf16x8_t af[4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
          af[i] = *reinterpret_cast<const bf16x8_t*>(
              As + ((size_t)s * NT + p) * BM * kLDK + lds_chunk(wm * 64 + i * 16 + fr, fk / 8));
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
      }
    }
    if (kt + 1 < KT) {
      sstore(s ^ 1);
      if (Q8) sfix();
    }
    __syncthreads();
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
        const float o = EPI == GEMV_SWIGLU ? pair_swap(v) : 0.f;
        epi_out<EPI>(C, ldc, H, ldh, M, N, m, n, v, o);
      }
}

// --------------------------------------------------------- MFMA, direct to LDS
// bf16 weights: a K step's tiles go from global memory straight into LDS
// (global_load_lds_dwordx4: each lane's 16 bytes land at the wavefront's LDS
// base + 16 x lane, so the row swizzle is applied by choosing which chunk each
// lane fetches) through a ring of STG stages, STG - 1 steps' loads in flight while
// one is multiplied, with no registers held for them and no register-to-LDS copy.
// The waits are explicit (this step's loads counted down, then a bare barrier): a
// __syncthreads would wait for every load in flight.  Rows past M or N fetch the
// last row (their outputs are dropped).  Four wavefronts in a 2 x 2 grid, each
// owning 64 rows x 64 WNT columns: a 128 x 128 WNT block.
//
// The loop is bound by LDS traffic, not by the matrix cores: per K step a
// wavefront reads NT x 4 activation fragments and 4 WNT weight fragments
// (16 bytes a lane each) for NT x 16 WNT products, and the stage fills write
// (NT + WNT) x 8 KB per workgroup.  Wider wavefront tiles (WNT = 2) re-read
// each activation fragment for twice the columns, which cuts the bytes per
// product by a third or more when the activation has two or three terms.
// Two stages keep two workgroups per CU (2 x 80 KB at NT = 3, WNT = 2).
constexpr int kDmaStages = 2;

__device__ __forceinline__ void dma16(const bf16_t* g, bf16_t* lds_wave) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)lds_wave, 16, 0, 0);
}
// s_waitcnt with vmcnt <= VM, lgkmcnt 0, expcnt unconstrained (gfx9 encoding)
template <int VM>
__device__ __forceinline__ void wait_vm_lgkm() {
  static_assert(VM >= 0 && VM < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((VM & 15) | ((VM >> 4) << 14) | (7 << 4));
}

template <int NT, int EPI, int STG = kDmaStages, int WNT = 1, bool NMAJ = false>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WNT == 2 ? 2 : 1))) void k_gemm_dma(const bf16_t* __restrict__ A, size_t a_plane,
                                                  int lda, const bf16_t* __restrict__ W, int M,
                                                  int N, int K, int ks, float* __restrict__ C,
                                                  size_t c_split, int ldc, ActBuf H, int ldh) {
  constexpr int BM = 128, BN = 128 * WNT, FN = 4 * WNT;  // FN: 16-column tiles per wavefront
  constexpr int TILE = 128 * kLDK;            // bf16 elements of one 128-row tile of a step
  constexpr int STAGE = (NT + WNT) * TILE;    // NT activation planes, then WNT weight tiles
  constexpr int PER_LANE = (NT + WNT) * 2;    // 16-byte units per lane per stage
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];

  const int n_mt = (M + BM - 1) / BM, n_nt = (N + BN - 1) / BN;
  int m0, n0;
  if (NMAJ) {
    // each XCD owns a contiguous range of weight column tiles for every row tile,
    // the row tiles of one column tile on consecutive workgroups (so the blocks
    // resident on an XCD share weight tiles through its L2)
    const int nper = (n_nt + 7) / 8, loc = blockIdx.x / 8;
    const int nt_i = (blockIdx.x % 8) * nper + loc / n_mt;
    if (nt_i >= n_nt || loc >= nper * n_mt) return;
    m0 = (loc % n_mt) * BM;
    n0 = nt_i * BN;
  } else {
    const int T = n_mt * n_nt, per_xcd = (T + 7) / 8;
    const int t = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (t >= T) return;
    m0 = (t / n_nt) * BM;
    n0 = (t % n_nt) * BN;
  }
  const int kbeg = blockIdx.y * ks;
  C += blockIdx.y * c_split;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;

  // unit u = (i * 4 + wave) * 64 + lane of a stage holds (128-row tile u / 512,
  // row (u % 512) / 4, LDS chunk u % 4), i.e. the row's global chunk
  // (u % 4) ^ lds_swz(row); tiles 0..NT-1 are the activation planes, NT.. the weights
  const bf16_t* src[PER_LANE];
#pragma unroll
  for (int i = 0; i < PER_LANE; ++i) {
    const int u = (i * 4 + wave) * 64 + lane, mat = u >> 9, r = (u & 511) >> 2;
    const int c = (u & 3) ^ lds_swz(r);
    if (mat < NT)
      src[i] = A + mat * a_plane + (size_t)min(m0 + r, M - 1) * lda + kbeg + c * 8;
    else
      src[i] = W + (size_t)min(n0 + (mat - NT) * 128 + r, N - 1) * K + kbeg + c * 8;
  }
  auto issue = [&](int stage, int kt) {
    bf16_t* sb = smem + stage * STAGE;
#pragma unroll
    for (int i = 0; i < PER_LANE; ++i) dma16(src[i] + kt * kBK, sb + (i * 4 + wave) * 512);
  };

  floatx4_t acc[4][FN];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  const int fr = lane & 15, fk = (lane >> 4) * 8;

  static_assert(STG >= 2 && STG <= 4, "stage ring of 2-4");
  const int KT = ks / kBK;
#pragma unroll
  for (int s = 0; s < STG - 1; ++s)
    if (s < KT) issue(s, s);
  for (int kt = 0; kt < KT; ++kt) {
    // this step's units have landed (the next steps' may still be in flight) and
    // every wavefront is done reading the stage that is refilled next
    const int ahead = min(STG - 2, KT - 1 - kt);  // later steps already issued
    if (ahead >= 2) wait_vm_lgkm<2 * PER_LANE>();
    else if (ahead == 1) wait_vm_lgkm<PER_LANE>();
    else wait_vm_lgkm<0>();
    __builtin_amdgcn_s_barrier();
    if (kt + STG - 1 < KT) issue((kt + STG - 1) % STG, kt + STG - 1);
    const bf16_t* sb = smem + (kt % STG) * STAGE;
    // weight fragments: wavefront column block wn covers weight rows
    // [64 WNT wn, 64 WNT (wn + 1)) of the block, i.e. of tile (64 WNT wn + 16 j) / 128
    bf16x8_t bfr[FN];
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const int row = wn * 64 * WNT + j * 16 + fr;
      bfr[j] = *reinterpret_cast<const bf16x8_t*>(sb + (NT + row / 128) * TILE +
                                                  lds_chunk(row % 128, fk / 8));
    }
#pragma unroll
    for (int p = 0; p < NT; ++p) {
      bf16x8_t af[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t*>(sb + p * TILE +
                                                   lds_chunk(wm * 64 + i * 16 + fr, fk / 8));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
  }

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm * 64 + i * 16 + (lane >> 4) * 4 + r;
        const int n = n0 + wn * 64 * WNT + j * 16 + (lane & 15);
        const float v = acc[i][j][r];
        const float o = EPI == GEMV_SWIGLU ? pair_swap(v) : 0.f;
        epi_out<EPI>(C, ldc, H, ldh, M, N, m, n, v, o);
      }
}

// ------------------------------------------------------------ skinny (M <= 32)
// For a handful of rows (a batched decode step: one row per sequence) the product
// is bound by streaming W, like the decode GEMV, not by the matrix cores.  A
// workgroup owns 16 TN columns (weight rows) and all M (<= 16 TM) rows; its four
// wavefronts split K and add their partial tiles through LDS at the end.  A
// wavefront loads its weight fragments straight from memory into the operand
// registers of v_mfma_f32_16x16x32_bf16 (lane l: row n0 + 16 j + l % 16, eight
// consecutive K at 8 (l / 16)), two K steps per batch, double-buffered, every
// load unconditional (rows clamped; rows of A past M are clamped too and their
// outputs dropped), so a batch's wait leaves the next batch in flight.  The
// activation fragments (NT bf16 planes, TM row tiles) come from L2.
template <int NT, int TM, int TN>
struct SkinnyBatch {
  static constexpr int D = 2;  // K steps per batch
  bf16x8_t w[D][TN];
  bf16x8_t a[D][NT][TM];
};

template <int NT, int TM, int TN, int EPI>
__global__ __launch_bounds__(256) void k_gemm_skinny(const bf16_t* __restrict__ A,
                                                     size_t a_plane, int lda,
                                                     const bf16_t* __restrict__ W, int M, int N,
                                                     int K, float* __restrict__ C, int ldc,
                                                     ActBuf H, int ldh) {
  using Bt = SkinnyBatch<NT, TM, TN>;
  constexpr int D = Bt::D;
  __shared__ floatx4_t red[4][TM][TN][64];
  const int n0 = blockIdx.x * 16 * TN;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int fr = lane & 15, fk = (lane >> 4) * 8;
  const int KT = K / kBK;
  const int kt0 = wave * KT / 4, kt1 = (wave + 1) * KT / 4, nst = kt1 - kt0;
  const int nb = (nst + D - 1) / D;  // batches of this wavefront
  const bf16_t* wrow[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) wrow[j] = W + (size_t)min(n0 + j * 16 + fr, N - 1) * K + fk;
  const bf16_t* arow[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) arow[i] = A + (size_t)min(i * 16 + fr, M - 1) * lda + fk;

  auto issue = [&](Bt& buf, int b) {
#pragma unroll
    for (int d = 0; d < D; ++d) {
      const int k = min(kt0 + b * D + d, KT - 1) * kBK;
#pragma unroll
      for (int j = 0; j < TN; ++j)
        buf.w[d][j] = __builtin_nontemporal_load(reinterpret_cast<const bf16x8_t*>(wrow[j] + k));
#pragma unroll
      for (int p = 0; p < NT; ++p)
#pragma unroll
        for (int i = 0; i < TM; ++i)
          buf.a[d][p][i] = *reinterpret_cast<const bf16x8_t*>(arow[i] + p * a_plane + k);
    }
  };
  floatx4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const Bt& buf, int b) {
#pragma unroll
    for (int d = 0; d < D; ++d)
      if (b * D + d < nst) {
#pragma unroll
        for (int p = 0; p < NT; ++p)
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(buf.a[d][p][i], buf.w[d][j],
                                                                  acc[i][j], 0, 0, 0);
      }
  };
  Bt b0, b1;
  issue(b0, 0);
  int b = 0;
  for (; b + 2 < nb; b += 2) {
    issue(b1, b + 1);
    compute(b0, b);
    issue(b0, b + 2);
    compute(b1, b + 1);
  }
  if (b + 1 < nb) {
    issue(b1, b + 1);
    compute(b0, b);
    compute(b1, b + 1);
  } else if (b < nb) {
    compute(b0, b);
  }

  // sum the four K ranges, then the epilogue (lane: rows 16 i + 4 (l / 16) + r,
  // column l % 16 of tile j)
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) red[wave][i][j][lane] = acc[i][j];
  __syncthreads();
  for (int t = wave; t < TM * TN; t += 4) {
    const int i = t / TN, j = t % TN;
    floatx4_t v = red[0][i][j][lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const floatx4_t u = red[w][i][j][lane];
      v[0] += u[0]; v[1] += u[1]; v[2] += u[2]; v[3] += u[3];
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = i * 16 + (lane >> 4) * 4 + r, n = n0 + j * 16 + (lane & 15);
      const float o = EPI == GEMV_SWIGLU ? pair_swap(v[r]) : 0.f;
      epi_out<EPI>(C, ldc, H, ldh, M, N, m, n, v[r], o);
    }
  }
}

// ------------------------------------------------- few rows, staged through LDS
// The same product for at most 32 rows, bf16 weights, K a multiple of 128: a
// workgroup owns 64 weight rows (16 per wavefront) and walks its K range in
// 128-deep slices through a ring of kRowsStages LDS stages, the weight slice
// (64 rows x 256 bytes) and the activation slice (NT planes x 16 TM rows x 256
// bytes) fetched by global_load_lds_dwordx4 in whole 128-byte lines, sixteen
// lanes to a row.  (Fragment-shaped loads straight into registers touch sixteen
// rows per instruction, 64 bytes each, and stream no faster than ~4.9 TB/s.)
// The 16-byte chunks of a row are XOR-swizzled by the row's low bits, so a
// fragment read (sixteen rows, one chunk) covers all 64 banks once.
//
// Products with few weight rows are split along K over grid slots: the splits
// of a 64-row tile occupy workgroup indices of one residue mod 8, so they run on
// one XCD (dispatch deals workgroups to the XCDs in turn) and exchange their
// partials through its L2, as the decode attention merge does: each split
// stores its accumulators, waits for the L2 to acknowledge them, records its
// XCD and takes a ticket from the tile's counter; the last one drops its CU's
// L1, adds the partials in split order (so the sum does not depend on timing),
// applies the epilogue and resets the counter.  A split that ran elsewhere
// sets *fault.
constexpr int kRowsKC = 128;     // K per LDS stage
constexpr int kRowsStages = 3;   // two slices in flight while one is multiplied
static_assert(kRowsStages >= 2 && kRowsStages <= 4, "stage ring of 2-4");
constexpr int kRowsSyncLine = 64;  // ints per tile: counter at 0, XCD records from 32
constexpr int kRowsMaxTiles = kGemmRowsSyncInts / kRowsSyncLine;  // tiles that can be split

template <int NT, int TM, int EPI>
__global__ __launch_bounds__(256) void k_gemm_rows(const bf16_t* __restrict__ A, size_t a_plane,
                                                   int lda, const bf16_t* __restrict__ W, int M,
                                                   int N, int K, int nsplit, int ks,
                                                   float* __restrict__ C, int ldc, ActBuf H,
                                                   int ldh, floatx4_t* __restrict__ part,
                                                   int* __restrict__ sync,
                                                   int* __restrict__ fault, int drill) {
  constexpr int CH = kRowsKC / 8;                 // 16-byte chunks per row of a slice
  constexpr int WUNITS = 64 * CH;                 // weight units (16 bytes) per slice
  constexpr int XUNITS = NT * 16 * TM * CH;       // activation units per slice
  constexpr int PL = (WUNITS + XUNITS) / 256;     // units per lane per slice
  constexpr int STAGE = (WUNITS + XUNITS) * 8;    // bf16 elements per stage
  static_assert((WUNITS + XUNITS) % 256 == 0, "whole instructions per slice");
  extern __shared__ __attribute__((aligned(16))) bf16_t smem[];

  const int T = (N + 63) / 64;
  const int loc = blockIdx.x / 8;
  const int t = blockIdx.x % 8 + 8 * (loc / nsplit), split = loc % nsplit;
  if (t >= T) return;
  const int n0 = t * 64, kbeg = split * ks;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;

  // unit u = (i * 4 + wave) * 64 + lane of a stage: weight row u / CH for u <
  // WUNITS, else activation plane / row; its LDS chunk u % CH holds the row's
  // global chunk (u % CH) ^ (row & (CH - 1))
  const bf16_t* src[PL];
#pragma unroll
  for (int i = 0; i < PL; ++i) {
    const int u = (i * 4 + wave) * 64 + lane;
    if (u < WUNITS) {
      const int r = u / CH, c = (u % CH) ^ (r & (CH - 1));
      src[i] = W + (size_t)min(n0 + r, N - 1) * K + kbeg + c * 8;
    } else {
      const int v = u - WUNITS, p = v / (16 * TM * CH), r = (v / CH) % (16 * TM);
      const int c = (v % CH) ^ (r & (CH - 1));
      src[i] = A + p * a_plane + (size_t)min(r, M - 1) * lda + kbeg + c * 8;
    }
  }
  // Each workgroup starts its walk at its own slice and wraps around: in lockstep
  // every workgroup would read the same K offset of rows 8 KB apart, which
  // crowds a few HBM channels.  Offsets of 7 slices between the workgroups of
  // an XCD and 4 between XCDs measured best (a bare stream of the 8B gate/up
  // weights: 5.2 -> 6.0 TB/s; offsets of 1 slice: 4.2).
  const int KT = ks / kRowsKC;
  const int rot = ((blockIdx.x / 8) * 7 + (blockIdx.x % 8) * 4) % KT;
  auto issue = [&](int stage, int kt) {
    bf16_t* sb = smem + stage * STAGE;
    const int kk = kt + rot < KT ? kt + rot : kt + rot - KT;
#pragma unroll
    for (int i = 0; i < PL; ++i) dma16(src[i] + kk * kRowsKC, sb + (i * 4 + wave) * 512);
  };

  floatx4_t acc[TM];
#pragma unroll
  for (int i = 0; i < TM; ++i) acc[i] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  const int fr = lane & 15, g = lane >> 4;
#pragma unroll
  for (int s = 0; s < kRowsStages - 1; ++s)
    if (s < KT) issue(s, s);
  for (int kt = 0; kt < KT; ++kt) {
    const int ahead = min(kRowsStages - 2, KT - 1 - kt);  // later slices already issued
    if (ahead >= 2) wait_vm_lgkm<2 * PL>();
    else if (ahead == 1) wait_vm_lgkm<PL>();
    else wait_vm_lgkm<0>();
    __builtin_amdgcn_s_barrier();
    if (kt + kRowsStages - 1 < KT) issue((kt + kRowsStages - 1) % kRowsStages, kt + kRowsStages - 1);
    const bf16_t* sb = smem + (kt % kRowsStages) * STAGE;
    const bf16_t* xb = sb + WUNITS * 8;
#pragma unroll
    for (int st = 0; st < kRowsKC / kBK; ++st) {
      const int c = 4 * st + g;  // this lane's chunk of the 32-deep step
      const int wr = wave * 16 + fr;
      const bf16x8_t wf = *reinterpret_cast<const bf16x8_t*>(sb + (wr * CH + (c ^ (wr & (CH - 1)))) * 8);
#pragma unroll
      for (int p = 0; p < NT; ++p)
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int xr = i * 16 + fr;
          const bf16x8_t xf = *reinterpret_cast<const bf16x8_t*>(
              xb + ((p * 16 * TM + xr) * CH + (c ^ (xr & (CH - 1)))) * 8);
          acc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xf, wf, acc[i], 0, 0, 0);
        }
    }
  }

  if (nsplit > 1) {
    __shared__ int s_last;
    floatx4_t* slab = part + ((size_t)(t * nsplit + split) * 4 * TM + wave * TM) * 64;
#pragma unroll
    for (int i = 0; i < TM; ++i) slab[i * 64 + lane] = acc[i];
    const int me = xcc_id();
    int* line = sync + (size_t)t * kRowsSyncLine;
    if (tid == 0) line[32 + split] = me;
    // this thread's stores have reached the L2 (the empty asm keeps the compiler
    // from moving memory operations across the wait)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0);
    asm volatile("" ::: "memory");
    __syncthreads();
    if (tid == 0) {
      const int old = __hip_atomic_fetch_add(line, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
      s_last = old == nsplit - 1;
      if (old == nsplit - 1)  // reset for the next launch
        __hip_atomic_exchange(line, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
    __syncthreads();
    if (!s_last) return;
    // drop this CU's L1 (it may hold lines of the partials from before their
    // stores); the loads below also bypass it (sc0)
    asm volatile("buffer_inv sc0" ::: "memory");
    const __amdgpu_buffer_rsrc_t rp =
        rsrc(part + (size_t)t * nsplit * 4 * TM * 64, (size_t)nsplit * 4 * TM * 64 * 16);
    const __amdgpu_buffer_rsrc_t rs = rsrc(line, kRowsSyncLine * 4);
    if (wave == 0 && lane < nsplit) {
      const int xo = __builtin_amdgcn_raw_buffer_load_b32(rs, (32 + lane) * 4, 0, 1);
      if (xo != me || drill) *fault = 1;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      floatx4_t sum = floatx4_t{0.f, 0.f, 0.f, 0.f};
      for (int sp = 0; sp < nsplit; ++sp) {
        const u32x4_t v = load_l2(rp, (int)((((size_t)sp * 4 * TM + wave * TM + i) * 64 + lane) * 16));
        sum[0] += __uint_as_float(v.x); sum[1] += __uint_as_float(v.y);
        sum[2] += __uint_as_float(v.z); sum[3] += __uint_as_float(v.w);
      }
      acc[i] = sum;
    }
  }
  // epilogue (lane: rows 16 i + 4 g + r, column n0 + 16 wave + fr)
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int m = i * 16 + 4 * g + r, n = n0 + wave * 16 + fr;
      const float v = acc[i][r];
      const float o = EPI == GEMV_SWIGLU ? pair_swap(v) : 0.f;
      epi_out<EPI>(C, ldc, H, ldh, M, N, m, n, v, o);
    }
}

// ------------------------------------------------------------------- vector fp32
template <typename WT, int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ A, int lda,
                                                  const WT* __restrict__ W, int M, int N, int K,
                                                  float* __restrict__ C, int ldc, ActBuf H,
                                                  int ldh, const unsigned short* __restrict__ S) {
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
      if constexpr (sizeof(WT) == 1) {  // Q8: (code - 128) * block scale
        const float d = (float)__builtin_bit_cast(_Float16, S[(size_t)wn * (K / 32) + (k0 + lk) / 32]);
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = ((float)W[(size_t)wn * K + k0 + lk + e] - 128.f) * d;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) w[e] = Elem<WT>::load(W + (size_t)wn * K + k0 + lk + e);
      }
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
      epi_out<EPI>(C, ldc, H, ldh, M, N, m, n, acc[i][j], (j & 1) ? 0.f : acc[i][j | 1]);
    }
}

// ------------------------------------------------------------------- launchers
template <int NT, int WM, int WN, int EPI, bool Q8>
static hipError_t gemm_mfma_launch(const ActBuf& A, int lda, const void* W, int M, int N, int K,
                                   float* C, int ldc, const ActBuf& H, int ldh, hipStream_t st,
                                   int nsplit = 1, size_t c_split = 0) {
  constexpr int BM = 64 * WM, BN = 64 * WN;
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  const int grid = (tiles + 7) / 8 * 8;
  const size_t lds = (size_t)2 * (NT * BM + BN) * kLDK * sizeof(bf16_t);
  const unsigned short* S =
      Q8 ? reinterpret_cast<const unsigned short*>(static_cast<const char*>(W) +
                                                   q8_scale_offset(N, K))
         : nullptr;
  auto fn = &k_gemm_mfma<NT, WM, WN, EPI, Q8>;
  if (lds > 65536)
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  hipLaunchKernelGGL(fn, dim3(grid, nsplit), dim3(64 * WM * WN), lds, st, A.planes,
                     A.plane_stride, lda, W, M, N, K, K / nsplit, C, c_split, ldc, H, ldh, S);
  return hipGetLastError();
}

template <int NT, int EPI, int STG = kDmaStages, int WNT = 1, bool NMAJ = false>
static hipError_t gemm_dma_launch(const ActBuf& A, int lda, const void* W, int M, int N, int K,
                                  float* C, int ldc, const ActBuf& H, int ldh, hipStream_t st,
                                  int nsplit = 1, size_t c_split = 0) {
  const int n_mt = (M + 127) / 128, n_nt = (N + 128 * WNT - 1) / (128 * WNT);
  const int grid = NMAJ ? 8 * ((n_nt + 7) / 8) * n_mt : (n_mt * n_nt + 7) / 8 * 8;
  const size_t lds = (size_t)STG * (NT + WNT) * 128 * kLDK * sizeof(bf16_t);
  auto fn = &k_gemm_dma<NT, EPI, STG, WNT, NMAJ>;
  if (lds > 65536)
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  hipLaunchKernelGGL(fn, dim3(grid, nsplit), dim3(256), lds, st, A.planes, A.plane_stride, lda,
                     static_cast<const bf16_t*>(W), M, N, K, K / nsplit, C, c_split, ldc, H, ldh);
  return hipGetLastError();
}

// Block shape 128 x 128 (four waves of 64 x 64).  Measured on the projection
// shapes of 1B-32B models at 1-2K rows, it beats 256 x 128 blocks by 14-35%: the
// smaller block keeps two workgroups resident per CU, which hides the global-load
// latency of the next K slice better than the halved weight re-reads save.
// bf16 weights from 1024 rows on: 64 x 128 wavefront tiles (128 x 256 blocks),
// each XCD owning a range of weight column tiles.  Measured with two or three
// activation terms: 8B gate/up 539 -> 504 us at 1024 rows, 32B gate/up 3202 ->
// 2050 and QKV 528 -> 426 us at 2048 rows; below 1024 rows the halved block
// count loses (1B QKV at 512 rows 56 -> 87 us, 128-row chunk tails 1.3-1.6x).
constexpr int kWideRows = 1024;

template <int NT, int EPI>
static hipError_t gemm_dma_pick(const ActBuf& A, int lda, const void* W, int M, int N, int K,
                                float* C, int ldc, const ActBuf& H, int ldh, hipStream_t st,
                                int nsplit = 1, size_t c_split = 0) {
  if (M >= kWideRows)
    return gemm_dma_launch<NT, EPI, kDmaStages, 2, true>(A, lda, W, M, N, K, C, ldc, H, ldh, st,
                                                         nsplit, c_split);
  return gemm_dma_launch<NT, EPI>(A, lda, W, M, N, K, C, ldc, H, ldh, st, nsplit, c_split);
}

template <int EPI, bool Q8>
static hipError_t gemm_mfma(const ActBuf& A, int lda, const void* W, int M, int N, int K,
                            float* C, int ldc, const ActBuf& H, int ldh, hipStream_t st) {
  if (!Q8) {
    switch (A.nt) {
      case 1: return gemm_dma_pick<1, EPI>(A, lda, W, M, N, K, C, ldc, H, ldh, st);
      case 2: return gemm_dma_pick<2, EPI>(A, lda, W, M, N, K, C, ldc, H, ldh, st);
      case 3: return gemm_dma_pick<3, EPI>(A, lda, W, M, N, K, C, ldc, H, ldh, st);
      default: return hipErrorInvalidValue;
    }
  }
  switch (A.nt) {
    case 1: return gemm_mfma_launch<1, 2, 2, EPI, Q8>(A, lda, W, M, N, K, C, ldc, H, ldh, st);
    case 2: return gemm_mfma_launch<2, 2, 2, EPI, Q8>(A, lda, W, M, N, K, C, ldc, H, ldh, st);
    case 3: return gemm_mfma_launch<3, 2, 2, EPI, Q8>(A, lda, W, M, N, K, C, ldc, H, ldh, st);
    default: return hipErrorInvalidValue;
  }
}

template <int NT, int TM, int TN, int EPI>
static hipError_t gemm_skinny_launch(const ActBuf& A, int lda, const void* W, int M, int N, int K,
                                     float* C, int ldc, const ActBuf& H, int ldh, hipStream_t st) {
  const int grid = (N + 16 * TN - 1) / (16 * TN);
  hipLaunchKernelGGL((k_gemm_skinny<NT, TM, TN, EPI>), dim3(grid), dim3(256), 0, st, A.planes,
                     A.plane_stride, lda, static_cast<const bf16_t*>(W), M, N, K, C, ldc, H, ldh);
  return hipGetLastError();
}

// Columns per workgroup: as many as still leave >= 512 workgroups (2 per CU).
template <int NT, int TM, int EPI>
static hipError_t gemm_skinny_tn(const ActBuf& A, int lda, const void* W, int M, int N, int K,
                                 float* C, int ldc, const ActBuf& H, int ldh, hipStream_t st) {
  if (N >= 64 * 512)
    return gemm_skinny_launch<NT, TM, 4, EPI>(A, lda, W, M, N, K, C, ldc, H, ldh, st);
  if (N >= 32 * 512)
    return gemm_skinny_launch<NT, TM, 2, EPI>(A, lda, W, M, N, K, C, ldc, H, ldh, st);
  return gemm_skinny_launch<NT, TM, 1, EPI>(A, lda, W, M, N, K, C, ldc, H, ldh, st);
}

template <int EPI>
static hipError_t gemm_skinny(const ActBuf& A, int lda, const void* W, int M, int N, int K,
                              float* C, int ldc, const ActBuf& H, int ldh, hipStream_t st) {
#define WICI_SKT(NT_)                                                                         \
  return M <= 16 ? gemm_skinny_tn<NT_, 1, EPI>(A, lda, W, M, N, K, C, ldc, H, ldh, st)        \
                 : gemm_skinny_tn<NT_, 2, EPI>(A, lda, W, M, N, K, C, ldc, H, ldh, st)
  switch (A.nt) {
    case 1: WICI_SKT(1);
    case 2: WICI_SKT(2);
    case 3: WICI_SKT(3);
    default: return hipErrorInvalidValue;
  }
#undef WICI_SKT
}

template <int NT, int TM, int EPI>
static hipError_t gemm_rows_launch(const ActBuf& A, int lda, const void* W, int M, int N, int K,
                                   int nsplit, float* C, int ldc, const ActBuf& H, int ldh,
                                   float* part, int* sync, int* fault, hipStream_t st,
                                   int drill = 0) {
  const int T = (N + 63) / 64;
  const int grid = 8 * ((T + 7) / 8) * nsplit;
  const size_t lds = (size_t)kRowsStages * (64 + NT * 16 * TM) * kRowsKC * sizeof(bf16_t);
  auto fn = &k_gemm_rows<NT, TM, EPI>;
  if (lds >= 65536)
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(fn),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  hipLaunchKernelGGL(fn, dim3(grid), dim3(256), lds, st, A.planes, A.plane_stride, lda,
                     static_cast<const bf16_t*>(W), M, N, K, nsplit, K / nsplit, C, ldc, H, ldh,
                     reinterpret_cast<floatx4_t*>(part), sync, fault, drill);
  return hipGetLastError();
}

template <typename WT, int EPI>
static hipError_t gemm_f32(const ActBuf& A, int lda, const WT* W, int M, int N, int K, float* C,
                           int ldc, const ActBuf& H, int ldh, hipStream_t st) {
  dim3 grid((N + 63) / 64, (M + 63) / 64);
  const unsigned short* S =
      sizeof(WT) == 1 ? reinterpret_cast<const unsigned short*>(
                            reinterpret_cast<const char*>(W) + q8_scale_offset(N, K))
                      : nullptr;
  hipLaunchKernelGGL((k_gemm_f32<WT, EPI>), grid, dim3(256), 0, st, A.f32, lda, W, M, N, K, C,
                     ldc, H, ldh, S);
  return hipGetLastError();
}

// Split K for products with too few output tiles to fill the chip: as many
// splits as still leave at most two blocks per CU (512), each at least 256 deep.
// (Blocks of 128 x 256 for bf16 weights from kWideRows rows on, else 128 x 128.)
int gemm_split_count(int wt, int nt, int M, int N, int K, int max_split) {
  if (nt < 1 || M <= 32 || (wt != W_BF16 && wt != W_Q8)) return 1;
  const int bn = wt == W_BF16 && M >= kWideRows ? 256 : 128;
  const int tiles = ((M + 127) / 128) * ((N + bn - 1) / bn);
  int n = std::max(1, std::min(max_split, 512 / std::max(tiles, 1)));
  while (n > 1 && (K % (kBK * n) || K / n < 256)) --n;
  return n;
}

template <int NT>
static hipError_t gemm_split_nt(int wt, const ActBuf& A, int lda, const void* W, int M, int N,
                                int K, int nsplit, float* P, size_t p_split, hipStream_t st) {
  const ActBuf none{};
  if (wt == W_Q8)
    return gemm_mfma_launch<NT, 2, 2, GEMV_STORE, true>(A, lda, W, M, N, K, P, N, none, 0, st,
                                                         nsplit, p_split);
  // the residual products (O, down: few output columns, split K) from 1024 rows
  // on: 8B down 274 -> 235 us, O 70 -> 66 us (the wider tile halves the
  // activation fragment reads per product; the placement lets the row tiles of
  // one weight tile share it in the XCD's L2)
  return gemm_dma_pick<NT, GEMV_STORE>(A, lda, W, M, N, K, P, N, none, 0, st, nsplit, p_split);
}

hipError_t launch_gemm_split(int wt, const ActBuf& A, int lda, const void* W, int M, int N, int K,
                             int nsplit, float* P, size_t p_split, hipStream_t st) {
  if (nsplit < 1 || K % (kBK * nsplit) || M <= 32 || (wt != W_BF16 && wt != W_Q8))
    return hipErrorInvalidValue;
  switch (A.nt) {
    case 1: return gemm_split_nt<1>(wt, A, lda, W, M, N, K, nsplit, P, p_split, st);
    case 2: return gemm_split_nt<2>(wt, A, lda, W, M, N, K, nsplit, P, p_split, st);
    case 3: return gemm_split_nt<3>(wt, A, lda, W, M, N, K, nsplit, P, p_split, st);
    default: return hipErrorInvalidValue;
  }
}

// Splits along K for the few-rows kernel: the fewest (up to 16) that give at
// least 192 workgroups with whole 128-deep slices, as far as the partials fit
// `part_floats` and the tiles the sync lines.  (Measured at 16 rows on the 8B
// shapes: QKV 2 splits 13.7 us, 4 17.3; O 4 splits 10.6 us, 8 12.1; down 4
// splits 25.5 us, 7 28.6: more, shorter workgroups pay more in pipeline fill
// and in the sum.)
int gemm_rows_splits(int M, int N, int K, size_t part_floats) {
  const int T = (N + 63) / 64, TM = M <= 16 ? 1 : 2;
  if (T > kRowsMaxTiles) return 1;
  int best = 1;
  for (int s = 2; s <= 16 && T * best < 192; ++s) {
    if (K % (s * kRowsKC)) continue;
    if ((size_t)T * s * 4 * TM * 64 * 4 > part_floats) break;
    best = s;
  }
  return best;
}

hipError_t launch_gemm_rows(int wt, int epi, const ActBuf& A, int lda, const void* W, int M,
                            int N, int K, float* C, int ldc, const ActBuf& H, int ldh,
                            float* part, size_t part_floats, int* sync, int* fault,
                            hipStream_t st, bool drill) {
  if (wt != W_BF16 || A.nt < 1 || A.nt > 3 || M < 1 || M > 32 || K % kRowsKC)
    return launch_gemm(wt, epi, A, lda, W, M, N, K, C, ldc, H, ldh, st);
  const int nsplit = part && sync && fault ? gemm_rows_splits(M, N, K, part_floats) : 1;
#define WICI_RW(NT_, TM_, E) \
  gemm_rows_launch<NT_, TM_, E>(A, lda, W, M, N, K, nsplit, C, ldc, H, ldh, part, sync, fault, st, \
                                drill)
#define WICI_RW_NT(E)                                                        \
  switch (A.nt) {                                                            \
    case 1: return M <= 16 ? WICI_RW(1, 1, E) : WICI_RW(1, 2, E);            \
    case 2: return M <= 16 ? WICI_RW(2, 1, E) : WICI_RW(2, 2, E);            \
    default: return M <= 16 ? WICI_RW(3, 1, E) : WICI_RW(3, 2, E);           \
  }
  switch (epi) {
    case GEMV_STORE: WICI_RW_NT(GEMV_STORE)
    case GEMV_RESID: WICI_RW_NT(GEMV_RESID)
    case GEMV_SWIGLU: WICI_RW_NT(GEMV_SWIGLU)
    default: return hipErrorInvalidValue;
  }
#undef WICI_RW_NT
#undef WICI_RW
}

hipError_t launch_gemm(int wt, int epi, const ActBuf& A, int lda, const void* W, int M, int N,
                       int K, float* C, int ldc, const ActBuf& H, int ldh, hipStream_t st) {
  if (K % kBK) return hipErrorInvalidValue;
#define WICI_EPI(CALL)                                      \
  switch (epi) {                                            \
    case GEMV_STORE: return CALL(GEMV_STORE);               \
    case GEMV_RESID: return CALL(GEMV_RESID);               \
    case GEMV_SWIGLU: return CALL(GEMV_SWIGLU);             \
    default: return hipErrorInvalidValue;                   \
  }
  if (A.nt == 0) {
#define WICI_F32(E) gemm_f32<WT_, E>(A, lda, static_cast<const WT_*>(W), M, N, K, C, ldc, H, ldh, st)
    if (wt == W_BF16) { using WT_ = bf16_t; WICI_EPI(WICI_F32) }
    if (wt == W_F32) { using WT_ = float; WICI_EPI(WICI_F32) }
    if (wt == W_Q8) { using WT_ = uint8_t; WICI_EPI(WICI_F32) }
#undef WICI_F32
    return hipErrorInvalidValue;
  }
#define WICI_SK(E) gemm_skinny<E>(A, lda, W, M, N, K, C, ldc, H, ldh, st)
  if (wt == W_BF16 && M <= 32) { WICI_EPI(WICI_SK) }
#undef WICI_SK
#define WICI_MF(E) gemm_mfma<E, Q8_>(A, lda, W, M, N, K, C, ldc, H, ldh, st)
  if (wt == W_BF16) { constexpr bool Q8_ = false; WICI_EPI(WICI_MF) }
  if (wt == W_Q8) { constexpr bool Q8_ = true; WICI_EPI(WICI_MF) }
#undef WICI_MF
#undef WICI_EPI
  return hipErrorInvalidValue;
}

}  // namespace wici
