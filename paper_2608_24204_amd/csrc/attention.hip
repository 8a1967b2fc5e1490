// Causal grouped-query attention over the paged KV cache.
//
// Decode (one query position per head): split-K over the context.  Grid =
// (nsplit, n_kv_heads); a block loads each cached key/value of its range once and
// serves all query heads of the KV head's group with it (GQA), so every cached
// byte is read once per step.  The new position's k/v are rotated, rounded to the
// storage type, written to the cache and used straight from LDS (no block reads a
// position another block of the same launch writes).  A second tiny kernel merges
// the splits with their (max, sum) statistics.
//
// Prefill: one block per (64 queries, query head), keys streamed through LDS in
// blocks of 64 with an online softmax, fp32 throughout.
#include "common.h"
#include "kernels.h"

namespace wici {

constexpr int kMaxGroup = 8;   // query heads per KV head
constexpr int kMaxChunk = 256; // positions per decode split

__device__ __forceinline__ size_t kv_off(const KvLayout& kv, int pos, int which, int h) {
  const int phys = kv.table[pos / kv.page], slot = pos % kv.page;
  return ((((size_t)phys * 2 + which) * kv.n_kv + h) * kv.page + slot) * (size_t)kv.hd;
}

// ------------------------------------------------------------------- decode
template <int HD, typename KT>
__global__ __launch_bounds__(256) void k_attn_decode(const float* __restrict__ qkv, int Hq,
                                                     const float* __restrict__ cos_t,
                                                     const float* __restrict__ sin_t,
                                                     KvLayout kv,
                                                     const DecodeState* __restrict__ st,
                                                     int nsplit, float* __restrict__ part_o,
                                                     float* __restrict__ part_ml) {
  constexpr int LPP = HD / 8;   // lanes per position (8 elements each)
  constexpr int PPW = 64 / LPP; // positions per wave per pass
  constexpr int PPB = 4 * PPW;  // positions per block per pass
  constexpr int HALF = HD / 2;
  __shared__ float qs[kMaxGroup][HD];
  __shared__ float sc[kMaxGroup][kMaxChunk];
  __shared__ float knew[HD], vnew[HD];
  __shared__ float accs[4][kMaxGroup][HD];
  __shared__ float mls[kMaxGroup][2];

  const int split = blockIdx.x, g = blockIdx.y;
  const int Hkv = kv.n_kv, G = Hq / Hkv;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int pos = st->pos, n = pos + 1;
  const int chunk = (n + nsplit - 1) / nsplit;
  const int start = split * chunk, end = min(n, start + chunk);
  const KT* base = static_cast<const KT*>(kv.base);

  if (start >= end) {  // empty split: contributes nothing to the merge
    for (int i = tid; i < G * HD; i += 256) {
      const int h = g * G + i / HD;
      part_o[((size_t)h * nsplit + split) * HD + i % HD] = 0.f;
    }
    if (tid < G) {
      const int h = g * G + tid;
      part_ml[((size_t)h * nsplit + split) * 2 + 0] = -INFINITY;
      part_ml[((size_t)h * nsplit + split) * 2 + 1] = 0.f;
    }
    return;
  }

  // rotated, pre-scaled queries of the group
  const float scale = 1.0f / sqrtf((float)HD);
  const float* cr = cos_t + (size_t)pos * HALF;
  const float* sr = sin_t + (size_t)pos * HALF;
  for (int i = tid; i < G * HALF; i += 256) {
    const int h = i / HALF, j = i % HALF;
    const float* z = qkv + (size_t)(g * G + h) * HD;
    const float a = z[j], b = z[j + HALF], c = cr[j], s = sr[j];
    qs[h][j] = (a * c - b * s) * scale;
    qs[h][j + HALF] = (a * s + b * c) * scale;
  }
  const bool has_new = end == n;
  if (has_new) {
    const float* kz = qkv + (size_t)Hq * HD + (size_t)g * HD;
    const float* vz = kz + (size_t)Hkv * HD;
    KT* kd = const_cast<KT*>(base) + kv_off(kv, pos, 0, g);
    KT* vd = const_cast<KT*>(base) + kv_off(kv, pos, 1, g);
    for (int j = tid; j < HALF; j += 256) {
      const float a = kz[j], b = kz[j + HALF], c = cr[j], s = sr[j];
      const float ra = Elem<KT>::round(a * c - b * s), rb = Elem<KT>::round(a * s + b * c);
      knew[j] = ra;
      knew[j + HALF] = rb;
      Elem<KT>::store(kd + j, ra);
      Elem<KT>::store(kd + j + HALF, rb);
    }
    for (int e = tid; e < HD; e += 256) {
      const float v = Elem<KT>::round(vz[e]);
      vnew[e] = v;
      Elem<KT>::store(vd + e, v);
    }
  }
  __syncthreads();

  const int pg = lane / LPP, sub = lane % LPP;
  float qr[kMaxGroup][8];
#pragma unroll
  for (int h = 0; h < kMaxGroup; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) qr[h][e] = h < G ? qs[h][sub * 8 + e] : 0.f;

  // scores
  for (int j0 = start; j0 < end; j0 += PPB) {
    const int j = j0 + wave * PPW + pg;
    float kk[8];
    if (j < end) {
      if (j == pos) {
#pragma unroll
        for (int e = 0; e < 8; ++e) kk[e] = knew[sub * 8 + e];
      } else {
        load8(base + kv_off(kv, j, 0, g) + sub * 8, kk);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) kk[e] = 0.f;
    }
#pragma unroll
    for (int h = 0; h < kMaxGroup; ++h) {
      if (h < G) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) s += qr[h][e] * kk[e];
#pragma unroll
        for (int m = LPP / 2; m >= 1; m >>= 1) s += __shfl_xor(s, m);
        if (sub == 0 && j < end) sc[h][j - start] = s;
      }
    }
  }
  __syncthreads();

  // softmax statistics per head (one wave per head)
  const int len = end - start;
  for (int h = wave; h < G; h += 4) {
    float m = -INFINITY;
    for (int i = lane; i < len; i += 64) m = fmaxf(m, sc[h][i]);
    m = wave_max(m);
    float l = 0.f;
    for (int i = lane; i < len; i += 64) {
      const float p = expf(sc[h][i] - m);
      sc[h][i] = p;
      l += p;
    }
    l = wave_sum(l);
    if (lane == 0) { mls[h][0] = m; mls[h][1] = l; }
  }
  __syncthreads();

  // weighted values
  float acc[kMaxGroup][8];
#pragma unroll
  for (int h = 0; h < kMaxGroup; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.f;
  for (int j0 = start; j0 < end; j0 += PPB) {
    const int j = j0 + wave * PPW + pg;
    if (j < end) {
      float vv[8];
      if (j == pos) {
#pragma unroll
        for (int e = 0; e < 8; ++e) vv[e] = vnew[sub * 8 + e];
      } else {
        load8(base + kv_off(kv, j, 1, g) + sub * 8, vv);
      }
#pragma unroll
      for (int h = 0; h < kMaxGroup; ++h) {
        if (h < G) {
          const float p = sc[h][j - start];
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[h][e] += p * vv[e];
        }
      }
    }
  }
#pragma unroll
  for (int h = 0; h < kMaxGroup; ++h) {
    if (h < G) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float a = acc[h][e];
#pragma unroll
        for (int m = LPP; m < 64; m <<= 1) a += __shfl_xor(a, m);
        if (pg == 0) accs[wave][h][sub * 8 + e] = a;
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < G * HD; i += 256) {
    const int hl = i / HD, d = i % HD, h = g * G + hl;
    part_o[((size_t)h * nsplit + split) * HD + d] =
        accs[0][hl][d] + accs[1][hl][d] + accs[2][hl][d] + accs[3][hl][d];
  }
  if (tid < G) {
    const int h = g * G + tid;
    part_ml[((size_t)h * nsplit + split) * 2 + 0] = mls[tid][0];
    part_ml[((size_t)h * nsplit + split) * 2 + 1] = mls[tid][1];
  }
}

// out[h, d] = sum_s e^(m_s - M) o_s[d] / sum_s e^(m_s - M) l_s
template <int HD>
__global__ __launch_bounds__(HD) void k_attn_combine(const float* __restrict__ part_o,
                                                     const float* __restrict__ part_ml,
                                                     int nsplit, float* __restrict__ out) {
  const int h = blockIdx.x, d = threadIdx.x;
  const float* ml = part_ml + (size_t)h * nsplit * 2;
  float M = -INFINITY;
  for (int s = 0; s < nsplit; ++s) M = fmaxf(M, ml[2 * s]);
  float L = 0.f, o = 0.f;
  for (int s = 0; s < nsplit; ++s) {
    const float w = expf(ml[2 * s] - M);
    L += w * ml[2 * s + 1];
    o += w * part_o[((size_t)h * nsplit + s) * HD + d];
  }
  out[(size_t)h * HD + d] = o / L;
}

template <int HD, typename KT>
static hipError_t attn_decode_t(const float* qkv, int Hq, const float* cos_t, const float* sin_t,
                                KvLayout kv, const DecodeState* st, int nsplit, float* part_o,
                                float* part_ml, float* out, hipStream_t s) {
  hipLaunchKernelGGL((k_attn_decode<HD, KT>), dim3(nsplit, kv.n_kv), dim3(256), 0, s, qkv, Hq,
                     cos_t, sin_t, kv, st, nsplit, part_o, part_ml);
  hipLaunchKernelGGL((k_attn_combine<HD>), dim3(Hq), dim3(HD), 0, s, part_o, part_ml, nsplit,
                     out);
  return hipGetLastError();
}

hipError_t launch_attn_decode(bool kv_bf16, const float* qkv, int Hq, const float* cos_t,
                              const float* sin_t, KvLayout kv, const void* state, int nsplit,
                              float* part_o, float* part_ml, float* out, hipStream_t s) {
  const DecodeState* st = static_cast<const DecodeState*>(state);
  if (kv.hd == 128) {
    if (kv_bf16) return attn_decode_t<128, bf16_t>(qkv, Hq, cos_t, sin_t, kv, st, nsplit, part_o, part_ml, out, s);
    return attn_decode_t<128, float>(qkv, Hq, cos_t, sin_t, kv, st, nsplit, part_o, part_ml, out, s);
  }
  if (kv.hd == 64) {
    if (kv_bf16) return attn_decode_t<64, bf16_t>(qkv, Hq, cos_t, sin_t, kv, st, nsplit, part_o, part_ml, out, s);
    return attn_decode_t<64, float>(qkv, Hq, cos_t, sin_t, kv, st, nsplit, part_o, part_ml, out, s);
  }
  return hipErrorInvalidValue;
}

// ------------------------------------------------------------------- prefill
template <int HD, typename KT>
__global__ __launch_bounds__(256) void k_attn_prefill(const float* __restrict__ qkv, int T,
                                                      int p0, int Hq, KvLayout kv,
                                                      float* __restrict__ out) {
  constexpr int BQ = 64, BKEY = 64, DPT = HD / 4;
  __shared__ float Ks[BKEY][HD + 4];
  __shared__ float Vs[BKEY][HD + 4];
  const int qb = blockIdx.x * BQ, h = blockIdx.y;
  const int Hkv = kv.n_kv, g = h / (Hq / Hkv);
  const int tid = threadIdx.x, ql = tid >> 2, part = tid & 3;
  const int t = qb + ql;
  const bool valid = t < T;
  const int qpos = p0 + t;
  const int width = (Hq + 2 * Hkv) * HD;
  const float scale = 1.0f / sqrtf((float)HD);
  const KT* base = static_cast<const KT*>(kv.base);

  float q[DPT], acc[DPT];
  const float* qrow = qkv + (size_t)(valid ? t : 0) * width + (size_t)h * HD + part * DPT;
#pragma unroll
  for (int e = 0; e < DPT; ++e) { q[e] = qrow[e] * scale; acc[e] = 0.f; }
  float m = -INFINITY, l = 0.f;
  const int kend = p0 + min(T, qb + BQ);

  for (int kb = 0; kb < kend; kb += BKEY) {
    __syncthreads();
    for (int idx = tid; idx < BKEY * (HD / 8); idx += 256) {
      const int jj = idx / (HD / 8), c = (idx % (HD / 8)) * 8, j = kb + jj;
      float kk[8], vv[8];
      if (j < kend) {
        load8(base + kv_off(kv, j, 0, g) + c, kk);
        load8(base + kv_off(kv, j, 1, g) + c, vv);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) { kk[e] = 0.f; vv[e] = 0.f; }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) { Ks[jj][c + e] = kk[e]; Vs[jj][c + e] = vv[e]; }
    }
    __syncthreads();
    float s[BKEY];
    float bm = -INFINITY;
#pragma unroll
    for (int jj = 0; jj < BKEY; ++jj) {
      float d = 0.f;
#pragma unroll
      for (int e = 0; e < DPT; ++e) d += q[e] * Ks[jj][part * DPT + e];
      d += __shfl_xor(d, 1);
      d += __shfl_xor(d, 2);
      const int j = kb + jj;
      s[jj] = (j <= qpos && j < kend) ? d : -INFINITY;
      bm = fmaxf(bm, s[jj]);
    }
    const float mn = fmaxf(m, bm);
    if (mn == -INFINITY) continue;  // no visible key yet (cannot happen for key 0)
    const float corr = expf(m - mn);
    l *= corr;
#pragma unroll
    for (int e = 0; e < DPT; ++e) acc[e] *= corr;
#pragma unroll
    for (int jj = 0; jj < BKEY; ++jj) {
      const float p = expf(s[jj] - mn);
      l += p;
#pragma unroll
      for (int e = 0; e < DPT; ++e) acc[e] += p * Vs[jj][part * DPT + e];
    }
    m = mn;
  }
  if (valid) {
    float* o = out + (size_t)t * Hq * HD + (size_t)h * HD + part * DPT;
    const float inv = 1.0f / l;
#pragma unroll
    for (int e = 0; e < DPT; ++e) o[e] = acc[e] * inv;
  }
}

template <int HD, typename KT>
static hipError_t attn_prefill_t(const float* qkv, int T, int p0, int Hq, KvLayout kv,
                                 float* out, hipStream_t s) {
  hipLaunchKernelGGL((k_attn_prefill<HD, KT>), dim3((T + 63) / 64, Hq), dim3(256), 0, s, qkv, T,
                     p0, Hq, kv, out);
  return hipGetLastError();
}

hipError_t launch_attn_prefill(bool kv_bf16, const float* qkv, int T, int p0, int Hq,
                               KvLayout kv, float* out, hipStream_t s) {
  if (kv.hd == 128) {
    if (kv_bf16) return attn_prefill_t<128, bf16_t>(qkv, T, p0, Hq, kv, out, s);
    return attn_prefill_t<128, float>(qkv, T, p0, Hq, kv, out, s);
  }
  if (kv.hd == 64) {
    if (kv_bf16) return attn_prefill_t<64, bf16_t>(qkv, T, p0, Hq, kv, out, s);
    return attn_prefill_t<64, float>(qkv, T, p0, Hq, kv, out, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace wici
