// Decode attention pieces shared by the attention launcher and the QKV
// projection that can run it in the same launch (included by attention.hip and
// gemv.hip only).
#pragma once
#include "common.h"
#include "kernels.h"

namespace wici {

constexpr int kChunk = 64;       // positions per decode split (at most one per lane of a wave:
                                 // the softmax statistics take one position per lane)

typedef short short4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));

// Merge of a KV head's splits in the last of its split blocks to finish (the
// batch-1 launch of k_attn_decode_mfma with FUSE, at most kFuseMaxSplits splits).
// Every split of head g runs on the same XCD, so the blocks exchange their
// partials through that XCD's L2 alone: each block's stores are acknowledged by
// the L2 (a wait for all of them) before it takes a ticket from the head's
// counter, an atomic performed in the same L2.  The block drawing the last
// ticket drops its CU's L1 (another workgroup on the CU may hold an older copy
// of a line), reads the partials from the L2 and merges them:
// out[h, d] = sum_s e^(m_s - M) o_s[d] / sum_s e^(m_s - M) l_s.  It then resets
// the counter for the next launch.  The placement is checked, not assumed: each
// block records the XCD it ran on (the hardware's XCC id) and the merging block
// compares them with its own; a mismatch sets fz.state->fault, which the step
// reports as an error.
constexpr int kFuseMaxSplits = 32;
constexpr int kFuseLine = 64;   // ints per head of the counter and XCD arrays (256 bytes)

template <int HD, int G>
__device__ __forceinline__ void attn_merge_in_last_split(const AttnFuse& fz, int g, int split,
                                                         int nsplit, int n,
                                                         const float* part_o,
                                                         const float* part_ml, int span = 1) {
  constexpr int COLS = G * HD / 4;      // float4 columns of the group's output
  constexpr int P = 256 / COLS;         // threads per column (>= 2)
  constexpr int PER = kFuseMaxSplits / P;
  __shared__ int s_last;
  __shared__ float s_w[G][kFuseMaxSplits];
  __shared__ float4 s_red[P][COLS];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int active = (n + kChunk * span - 1) / (kChunk * span);  // splits holding positions
  const int me = xcc_id();
  if (tid == 0) fz.xcc[g * kFuseLine + split] = me;
  // this thread's stores have reached the L2 (the empty asm keeps the compiler
  // from moving memory operations across the wait)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0);
  asm volatile("" ::: "memory");
  __syncthreads();
  if (tid == 0) {
    const int old = __hip_atomic_fetch_add(fz.cnt + g * kFuseLine, 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_WORKGROUP);
    s_last = old == active - 1;
    if (old == active - 1)  // reset for the next launch (an atomic, like every access to it)
      __hip_atomic_exchange(fz.cnt + g * kFuseLine, 0, __ATOMIC_RELAXED,
                            __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  __syncthreads();
  if (!s_last) return;
  // drop this CU's L1: another workgroup on the CU may have read a line of the
  // statistics (lines are shared between groups) before this group's splits
  // wrote it; the loads below also carry sc0, which alone does not force a miss
  asm volatile("buffer_inv sc0" ::: "memory");

  // the group's partials: column c of splits p, p + P, ... (clamped, all issued at once)
  const int c = tid % COLS, p = tid / COLS;
  const int hl = c / (HD / 4), d4 = c % (HD / 4);
  const int hh = g * G + hl;
  const __amdgpu_buffer_rsrc_t ro = rsrc(part_o, (size_t)fz.n_heads * nsplit * HD * 4);
  const __amdgpu_buffer_rsrc_t rm = rsrc(part_ml, (size_t)fz.n_heads * nsplit * 2 * 4);
  const __amdgpu_buffer_rsrc_t rx = rsrc(fz.xcc, (size_t)fz.n_kv * kFuseLine * 4);
  u32x4_t pv[PER];
  if (p < P) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int sp = min(p + P * k, active - 1);
      pv[k] = load_l2(ro, (int)((((size_t)hh * nsplit + sp) * HD + 4 * d4) * 4));
    }
  }
  // statistics: one wavefront per head, lane = split
  for (int h = wave; h < G; h += (int)(blockDim.x >> 6)) {
    const int hq = g * G + h, sp = min(lane, active - 1);
    const size_t f = ((size_t)hq * nsplit + sp) * 2;   // float index of (m, l)
    const u32x4_t st2 = load_l2(rm, (int)((f & ~(size_t)3) * 4));
    const u32x4_t xv = load_l2(rx, (g * kFuseLine + (sp & ~3)) * 4);
    // both loads in one round trip (the compiler would otherwise issue the XCD
    // record's load only inside the branch that tests it, after the reductions)
    asm volatile("" ::"v"(st2.x), "v"(xv.x));
    const bool odd = (f & 3) != 0;
    const float mv = __uint_as_float(odd ? st2.z : st2.x), lv = __uint_as_float(odd ? st2.w : st2.y);
    const int xo = (int)(xv[sp & 3]);
    const bool on = lane < active;
    const float M = wave_max(on ? mv : -INFINITY);
    const float e = on ? __expf(mv - M) : 0.f;
    const float L = wave_sum(e * (on ? lv : 0.f));
    if (on) s_w[h][lane] = e / L;
    if (on && (xo != me || fz.drill)) static_cast<DecodeState*>(fz.state)->fault = 1;
  }
  __syncthreads();
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  if (p < P) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int sp = p + P * k;
      if (sp < active) {
        const float w = s_w[hl][sp];
        acc.x += w * __uint_as_float(pv[k].x);
        acc.y += w * __uint_as_float(pv[k].y);
        acc.z += w * __uint_as_float(pv[k].z);
        acc.w += w * __uint_as_float(pv[k].w);
      }
    }
    s_red[p][c] = acc;
  }
  __syncthreads();
  if (tid < COLS) {
    float4 o = s_red[0][tid];
#pragma unroll
    for (int q = 1; q < P; ++q) {
      const float4 t = s_red[q][tid];
      o.x += t.x; o.y += t.y; o.z += t.z; o.w += t.w;
    }
    reinterpret_cast<float4*>(fz.out)[(size_t)g * COLS + tid] = o;
  }
}

// One decode split on the matrix cores, for a bf16 cache: positions
// [64 split, 64 split + 64) of KV head g, all G query heads (see the comment
// above k_attn_decode_mfma).  Writes the split's unnormalised output and
// (max, sum) statistics into part_o / part_ml ([Hq][nsplit] order) and returns
// the context length n = pos + 1, or 0 when the split lies past the context
// (nothing is written then).  Called by whole 256-thread workgroups.
//
// With ROPE (the batched step), q_in is the sequence's raw projection row
// (query heads, key heads, value heads) and this launch does the work of the
// RoPE + append kernel it replaces: every split rotates its query at the
// position (and scales it by rope.q_scale), and the split holding the position
// rotates that position's key, rounds key and value to the cache type, uses
// them for its own scores and stores them in the cache.  A lane's dimensions
// 32 s + 8 (l / 16) + e hold both members of each RoPE pair (j, j + HD / 2):
// steps s and s + DS / 2.

template <int HD, int G, bool ROPE = false>
__device__ __forceinline__ int attn_split_mfma(const float* __restrict__ q_in, const KvLayout& kv,
                                               const DecodeState* __restrict__ st,
                                               float* __restrict__ part_o,
                                               float* __restrict__ part_ml, int g, int split,
                                               int nsplit, RopeIn rope = RopeIn{}) {
  constexpr int DS = HD / 32;  // 32-deep steps of S^T
  constexpr int DT = HD / 16;  // 16-wide output tiles of P V
  constexpr int VP = 16 + 4;   // LDS row of one dimension's 16 positions (8-byte aligned reads)
  __shared__ bf16_t vt[4][HD][VP];
  __shared__ float wm[4][G], wl[4][G];
  __shared__ float wo[4][G][HD];

  const int Hkv = kv.n_kv;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int start = split * kChunk;
  const int ps = __ffs(kv.page) - 1;
  const bf16_t* base = static_cast<const bf16_t*>(kv.base);
  const size_t head_stride = (size_t)kv.page * HD;

  // this lane's page, its query slice (head r16) and the position.  The compiler
  // tests the position (the exit below) before it issues the page and query
  // loads, so those follow in a round trip of their own; a fence that keeps them
  // ahead of the test (two round trips instead of three) measured slower.
  const int jl = start + 16 * wave + r16;  // this lane's key/value position
  const int jc = min(jl, kv.max_pos - 1);
  const int phys = kv.table[jc >> ps];
  float qv[DS][8];
  {
    const float* qr = q_in + ((size_t)g * G + min(r16, G - 1)) * HD + 8 * g4;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const float4 a = *reinterpret_cast<const float4*>(qr + 32 * s);
      const float4 b = *reinterpret_cast<const float4*>(qr + 32 * s + 4);
      qv[s][0] = a.x; qv[s][1] = a.y; qv[s][2] = a.z; qv[s][3] = a.w;
      qv[s][4] = b.x; qv[s][5] = b.y; qv[s][6] = b.z; qv[s][7] = b.w;
    }
  }
  const int n = st->pos + 1;
  if (start >= n) return 0;

  // then the keys and values of this lane's position
  const bf16_t* pk = base + (((size_t)phys * 2 + 0) * Hkv + g) * head_stride +
                     (size_t)(jc & (kv.page - 1)) * HD + 8 * g4;
  const bf16_t* pv = pk + (size_t)Hkv * head_stride;
  bf16x8_t kf[DS];
  uint4 vr[DS];
#pragma unroll
  for (int s = 0; s < DS; ++s) {
    kf[s] = *reinterpret_cast<const bf16x8_t*>(pk + 32 * s);
    vr[s] = *reinterpret_cast<const uint4*>(pv + 32 * s);
  }
  if constexpr (ROPE) {
    constexpr int H2 = DS / 2;  // steps holding the first member of a pair
    const int pos = n - 1;
    const float* cr = rope.cos + (size_t)pos * (HD / 2) + 8 * g4;
    const float* sr = rope.sin + (size_t)pos * (HD / 2) + 8 * g4;
    // the query, rotated and scaled
#pragma unroll
    for (int s = 0; s < H2; ++s)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float a = qv[s][e], bb = qv[s + H2][e], c = cr[32 * s + e], sn = sr[32 * s + e];
        const float ra = a * c - bb * sn, rb = a * sn + bb * c;
        qv[s][e] = ra * rope.q_scale;
        qv[s + H2][e] = rb * rope.q_scale;
      }
    // the new position's key (rotated) and value, from the projection row
    if (jl == pos) {
      const float* kr = q_in + ((size_t)Hkv * G + g) * HD + 8 * g4;
      const float* vrow = q_in + ((size_t)Hkv * G + Hkv + g) * HD + 8 * g4;
#pragma unroll
      for (int s = 0; s < H2; ++s)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float a = kr[32 * s + e], bb = kr[32 * (s + H2) + e];
          const float c = cr[32 * s + e], sn = sr[32 * s + e];
          kf[s][e] = static_cast<__bf16>(a * c - bb * sn);
          kf[s + H2][e] = static_cast<__bf16>(a * sn + bb * c);
        }
#pragma unroll
      for (int s = 0; s < DS; ++s) {
        unsigned w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = (unsigned)f32_to_bf16(vrow[32 * s + 2 * e]) |
                 ((unsigned)f32_to_bf16(vrow[32 * s + 2 * e + 1]) << 16);
        vr[s] = make_uint4(w[0], w[1], w[2], w[3]);
        bf16_t* wk = const_cast<bf16_t*>(pk) + 32 * s;
        bf16_t* wv = const_cast<bf16_t*>(pv) + 32 * s;
        *reinterpret_cast<bf16x8_t*>(wk) = kf[s];
        *reinterpret_cast<uint4*>(wv) = vr[s];
      }
    }
  }
  // the query as three bf16 terms (columns past G are zero)
  bf16x8_t qb[3][DS];
#pragma unroll
  for (int s = 0; s < DS; ++s)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float v = r16 < G ? qv[s][e] : 0.f;
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const __bf16 b = static_cast<__bf16>(v);
        qb[t][s][e] = b;
        v -= static_cast<float>(b);
      }
    }
  // values transposed into this wavefront's LDS tile (zero past the context:
  // a stale slot may hold anything, and 0 x NaN is NaN)
  const bool valid = jl < n;
#pragma unroll
  for (int s = 0; s < DS; ++s) {
    const unsigned w4[4] = {vr[s].x, vr[s].y, vr[s].z, vr[s].w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const unsigned w = valid ? w4[e] : 0u;
      vt[wave][32 * s + 8 * g4 + 2 * e][r16] = (bf16_t)(w & 0xffffu);
      vt[wave][32 * s + 8 * g4 + 2 * e + 1][r16] = (bf16_t)(w >> 16);
    }
  }

  // S^T: lane holds S[position 4 g4 + i][head r16]
  floatx4_t sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < DS; ++s)
#pragma unroll
    for (int t = 0; t < 3; ++t)
      sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[s], qb[t][s], sc, 0, 0, 0);
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (start + 16 * wave + 4 * g4 + i >= n) sc[i] = -INFINITY;
    m = fmaxf(m, sc[i]);
  }
  m = fmaxf(m, __shfl_xor(m, 16));
  m = fmaxf(m, __shfl_xor(m, 32));
  float p[4], l = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    p[i] = sc[i] == -INFINITY ? 0.f : __expf(sc[i] - m);
    l += p[i];
  }
  l += __shfl_xor(l, 16);
  l += __shfl_xor(l, 32);
  // P as three bf16 terms in the A-operand order (head r16, positions 4 g4 + i)
  short4_t pa[3];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float v = p[i];
#pragma unroll
    for (int t = 0; t < 3; ++t) {
      const __bf16 b = static_cast<__bf16>(v);
      pa[t][i] = __builtin_bit_cast(short, b);
      v -= static_cast<float>(b);
    }
  }
  __syncthreads();  // the value tiles are in LDS

  // O = P V: lane holds O[head 4 g4 + i][dimension 16 u + r16]
  floatx4_t o[DT];
#pragma unroll
  for (int u = 0; u < DT; ++u) {
    o[u] = floatx4_t{0.f, 0.f, 0.f, 0.f};
    const short4_t vb = *reinterpret_cast<const short4_t*>(&vt[wave][16 * u + r16][4 * g4]);
#pragma unroll
    for (int t = 0; t < 3; ++t)
      o[u] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa[t], vb, o[u], 0, 0, 0);
  }
  // combine the four wavefronts
  if (g4 == 0 && r16 < G) { wm[wave][r16] = m; wl[wave][r16] = l; }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int h = 4 * g4 + i;
    if (h < G) {
#pragma unroll
      for (int u = 0; u < DT; ++u) wo[wave][h][16 * u + r16] = o[u][i];
    }
  }
  __syncthreads();
  for (int idx = tid; idx < G * HD; idx += 256) {
    const int h = idx / HD, d = idx % HD;
    float M = wm[0][h];
#pragma unroll
    for (int w = 1; w < 4; ++w) M = fmaxf(M, wm[w][h]);
    float acc = 0.f, L = 0.f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float e = wm[w][h] == -INFINITY ? 0.f : __expf(wm[w][h] - M);
      acc += e * wo[w][h][d];
      L += e * wl[w][h];
    }
    const int hh = g * G + h;
    part_o[((size_t)hh * nsplit + split) * HD + d] = acc;
    if (d == 0) {
      part_ml[((size_t)hh * nsplit + split) * 2 + 0] = M;
      part_ml[((size_t)hh * nsplit + split) * 2 + 1] = L;
    }
  }
  return n;
}

// A split of `span` consecutive 64-position sub-chunks (long contexts, so that
// the splits of a head stay few enough for the merge in the last split block):
// positions [64 span split, 64 span (split + 1)) of KV head g, all G query
// heads, by a workgroup of TEAMS x 4 wavefronts.  Team t takes sub-chunks t,
// t + TEAMS, ..., each multiplied as in attn_split_mfma (wavefront w of the
// team: positions 16 w .. 16 w + 15 of it); a wavefront carries its (max, sum)
// and output rows across its sub-chunks (online softmax: the running values
// are rescaled by e^(m_old - m_new) when the max grows), and all 4 TEAMS
// wavefronts are combined at the end.  The teams' wavefronts hide each other's
// load and matrix-chain latencies (one team of four walking every sub-chunk
// leaves under one wavefront per SIMD on the chip: 8.2K positions 18.5 us per
// layer, two teams with two sub-chunks in flight each 14.1 us).  The query's
// bf16 terms sit in LDS (the same fragments in every wavefront) to keep the
// registers within four wavefronts per SIMD.  The split's page-table entries
// are requested with the query.  Writes and returns as attn_split_mfma.
constexpr int kMaxSpan = 8;
template <int HD, int G, int TEAMS>
__device__ __forceinline__ int attn_span_mfma(const float* __restrict__ q_in, const KvLayout& kv,
                                              const DecodeState* __restrict__ st,
                                              float* __restrict__ part_o,
                                              float* __restrict__ part_ml, int g, int split,
                                              int nsplit, int span) {
  constexpr int DS = HD / 32;  // 32-deep steps of S^T
  constexpr int DT = HD / 16;  // 16-wide output tiles of P V
  constexpr int VP = 16 + 4;   // LDS row of one dimension's 16 positions
  constexpr int NW = 4 * TEAMS;
  __shared__ bf16_t vt[NW][HD][VP];
  __shared__ float wm[NW][G], wl[NW][G];
  __shared__ float wo[NW][G][HD];

  const int Hkv = kv.n_kv;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int team = wave >> 2, wq = wave & 3;
  const int r16 = lane & 15, g4 = lane >> 4;
  const int start = split * kChunk * span;
  const int ps = __ffs(kv.page) - 1;
  const bf16_t* base = static_cast<const bf16_t*>(kv.base);
  const size_t head_stride = (size_t)kv.page * HD;

  // this lane's position in each of its team's sub-chunks and the page, the
  // query and the context length, requested together
  constexpr int MJ = (kMaxSpan + TEAMS - 1) / TEAMS;  // sub-chunks per team at most
  int phys[MJ];
#pragma unroll
  for (int j = 0; j < MJ; ++j) {
    const int c = team + TEAMS * j;
    const int jc = min(start + c * kChunk + 16 * wq + r16, kv.max_pos - 1);
    phys[j] = c < span ? kv.table[jc >> ps] : 0;
  }
  float qv[DS][8];
  {
    const float* qr = q_in + ((size_t)g * G + min(r16, G - 1)) * HD + 8 * g4;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const float4 a = *reinterpret_cast<const float4*>(qr + 32 * s);
      const float4 b = *reinterpret_cast<const float4*>(qr + 32 * s + 4);
      qv[s][0] = a.x; qv[s][1] = a.y; qv[s][2] = a.z; qv[s][3] = a.w;
      qv[s][4] = b.x; qv[s][5] = b.y; qv[s][6] = b.z; qv[s][7] = b.w;
    }
  }
  const int n = st->pos + 1;
  if (start >= n) return 0;
  const int nsub = min(span, (n - start + kChunk - 1) / kChunk);
  const int nj = nsub > team ? (nsub - team + TEAMS - 1) / TEAMS : 0;  // this team's sub-chunks

  bf16x8_t kf[1][DS];  // one sub-chunk per wavefront at a time
  uint4 vr[1][DS];
  auto load = [&](int b, int j) {
    const int c = team + TEAMS * j;
    const int jc = min(start + c * kChunk + 16 * wq + r16, kv.max_pos - 1);
    int pp = phys[0];
#pragma unroll
    for (int i = 1; i < MJ; ++i) pp = j == i ? phys[i] : pp;
    const bf16_t* pk = base + (((size_t)pp * 2 + 0) * Hkv + g) * head_stride +
                       (size_t)(jc & (kv.page - 1)) * HD + 8 * g4;
    const bf16_t* pv = pk + (size_t)Hkv * head_stride;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      kf[b][s] = *reinterpret_cast<const bf16x8_t*>(pk + 32 * s);
      vr[b][s] = *reinterpret_cast<const uint4*>(pv + 32 * s);
    }
  };
  // the query as three bf16 terms (columns past G are zero), in LDS: every
  // wavefront reads the same fragments, which would hold 48 registers
  __shared__ bf16x8_t qlds[3][DS][64];
  if (wave == 0) {
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      bf16x8_t qt[3];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float v = r16 < G ? qv[s][e] : 0.f;
#pragma unroll
        for (int t = 0; t < 3; ++t) {
          const __bf16 b = static_cast<__bf16>(v);
          qt[t][e] = b;
          v -= static_cast<float>(b);
        }
      }
#pragma unroll
      for (int t = 0; t < 3; ++t) qlds[t][s][lane] = qt[t];
    }
  }
  __syncthreads();
  if (nj > 0) load(0, 0);

  float m_run = -INFINITY, l_run = 0.f;  // of head r16 over this wavefront's positions
  floatx4_t o[DT];                       // lane: O[head 4 g4 + i][dimension 16 u + r16]
#pragma unroll
  for (int u = 0; u < DT; ++u) o[u] = floatx4_t{0.f, 0.f, 0.f, 0.f};
  auto process = [&](int b, int j) {
    const int c0 = start + (team + TEAMS * j) * kChunk + 16 * wq;  // first position
    // values transposed into this wavefront's LDS tile (zero past the context);
    // the tile is the wavefront's own, and the previous sub-chunk's reads of it
    // have returned (their matrix ops consumed them) before these stores
    const bool valid = c0 + r16 < n;
#pragma unroll
    for (int s = 0; s < DS; ++s) {
      const unsigned w4[4] = {vr[b][s].x, vr[b][s].y, vr[b][s].z, vr[b][s].w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const unsigned w = valid ? w4[e] : 0u;
        vt[wave][32 * s + 8 * g4 + 2 * e][r16] = (bf16_t)(w & 0xffffu);
        vt[wave][32 * s + 8 * g4 + 2 * e + 1][r16] = (bf16_t)(w >> 16);
      }
    }
    // the tile's stores are done before any lane reads it (lgkmcnt 0 alone)
    __builtin_amdgcn_s_waitcnt(0xC07F);
    __builtin_amdgcn_wave_barrier();
    floatx4_t sc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < DS; ++s)
#pragma unroll
      for (int t = 0; t < 3; ++t)
        sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[b][s], qlds[t][s][lane], sc, 0, 0, 0);
    float mc = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (c0 + 4 * g4 + i >= n) sc[i] = -INFINITY;
      mc = fmaxf(mc, sc[i]);
    }
    mc = fmaxf(mc, __shfl_xor(mc, 16));
    mc = fmaxf(mc, __shfl_xor(mc, 32));
    const float m_new = fmaxf(m_run, mc);
    const float corr = m_new == -INFINITY ? 1.f : __expf(m_run - m_new);
    float p[4], lc = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      p[i] = sc[i] == -INFINITY ? 0.f : __expf(sc[i] - m_new);
      lc += p[i];
    }
    lc += __shfl_xor(lc, 16);
    lc += __shfl_xor(lc, 32);
    l_run = l_run * corr + lc;
    m_run = m_new;
    short4_t pa[3];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v = p[i];
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        const __bf16 bb = static_cast<__bf16>(v);
        pa[t][i] = __builtin_bit_cast(short, bb);
        v -= static_cast<float>(bb);
      }
    }
    // rescale the output rows (heads 4 g4 + i) by their heads' factors
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float cr = __shfl(corr, 4 * g4 + i);
#pragma unroll
      for (int u = 0; u < DT; ++u) o[u][i] *= cr;
    }
#pragma unroll
    for (int u = 0; u < DT; ++u) {
      const short4_t vb = *reinterpret_cast<const short4_t*>(&vt[wave][16 * u + r16][4 * g4]);
#pragma unroll
      for (int t = 0; t < 3; ++t)
        o[u] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(pa[t], vb, o[u], 0, 0, 0);
    }
  };
  for (int j = 0; j < nj; ++j) {
    if (j > 0) load(0, j);
    process(0, j);
  }

  // combine the wavefronts (one without positions has max -inf and weight 0)
  if (g4 == 0 && r16 < G) { wm[wave][r16] = m_run; wl[wave][r16] = l_run; }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int h = 4 * g4 + i;
    if (h < G) {
#pragma unroll
      for (int u = 0; u < DT; ++u) wo[wave][h][16 * u + r16] = o[u][i];
    }
  }
  __syncthreads();
  for (int idx = tid; idx < G * HD; idx += 64 * NW) {
    const int h = idx / HD, d = idx % HD;
    float M = wm[0][h];
#pragma unroll
    for (int w = 1; w < NW; ++w) M = fmaxf(M, wm[w][h]);
    float acc = 0.f, L = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float e = wm[w][h] == -INFINITY ? 0.f : __expf(wm[w][h] - M);
      acc += e * wo[w][h][d];
      L += e * wl[w][h];
    }
    const int hh = g * G + h;
    part_o[((size_t)hh * nsplit + split) * HD + d] = acc;
    if (d == 0) {
      part_ml[((size_t)hh * nsplit + split) * 2 + 0] = M;
      part_ml[((size_t)hh * nsplit + split) * 2 + 1] = L;
    }
  }
  return n;
}

}  // namespace wici
