// Kernels of the batched decode step: B sequences (clients sharing one copy of
// the weights, each with its own KV cache and position) advance one token in one
// pass over the weights.  Row b of every activation matrix is sequence b; what
// differs per sequence (position, KV pages, token history) comes from a device
// array of SeqDesc.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace wici {

// tokens[b] = sequence b's input token (its state's token)
__global__ void k_gather_tokens(const SeqDesc* __restrict__ seqs, int B,
                                int32_t* __restrict__ tokens) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b < B) tokens[b] = static_cast<const DecodeState*>(seqs[b].state)->token;
}

hipError_t launch_gather_tokens(const SeqDesc* seqs, int B, int32_t* tokens, hipStream_t st) {
  hipLaunchKernelGGL(k_gather_tokens, dim3((B + 63) / 64), dim3(64), 0, st, seqs, B, tokens);
  return hipGetLastError();
}

// Row b of qkv: rotate its query heads in place (and scale them by q_scale), rotate
// its key heads and append keys and values to sequence b's cache at its position.
template <typename KT>
__global__ __launch_bounds__(256) void k_rope_append_batch(float* __restrict__ qkv, int Hq,
                                                           const float* __restrict__ cos_t,
                                                           const float* __restrict__ sin_t,
                                                           const SeqDesc* __restrict__ seqs,
                                                           int layer, KvLayout kv, float q_scale) {
  const int b = blockIdx.x;
  const SeqDesc sd = seqs[b];
  const int pos = static_cast<const DecodeState*>(sd.state)->pos;
  const int hd = kv.hd, half = hd >> 1, Hkv = kv.n_kv;
  float* row = qkv + (size_t)b * (Hq + 2 * Hkv) * hd;
  const float* cr = cos_t + (size_t)pos * half;
  const float* sr = sin_t + (size_t)pos * half;
  KT* base = reinterpret_cast<KT*>(static_cast<char*>(sd.kv) + (size_t)layer * sd.kv_layer_stride);
  const int phys = sd.table[pos / kv.page], slot = pos % kv.page;
  for (int i = threadIdx.x; i < (Hq + Hkv) * half; i += blockDim.x) {
    const int h = i / half, j = i % half;
    float* z = row + h * hd;
    const float a = z[j], bb = z[j + half], c = cr[j], s = sr[j];
    const float ra = a * c - bb * s, rb = a * s + bb * c;
    if (h < Hq) {
      z[j] = ra * q_scale;
      z[j + half] = rb * q_scale;
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
    Elem<KT>::store(dst + e, row[(Hq + Hkv) * hd + i]);
  }
}

// The same on 4-element slices (head dimension a multiple of 8) with every load
// of a thread's slices issued before any is used (the loop form above waits out
// each iteration's loads); rotated in place, each slice read and written by one
// thread.  Same operations per element: bit-identical results.
template <typename KT, int MAXI>
__global__ __launch_bounds__(256) void k_rope_append_batch4(float* __restrict__ qkv, int Hq,
                                                            const float* __restrict__ cos_t,
                                                            const float* __restrict__ sin_t,
                                                            const SeqDesc* __restrict__ seqs,
                                                            int layer, KvLayout kv, float q_scale) {
  const int b = blockIdx.x, tid = threadIdx.x;
  const SeqDesc sd = seqs[b];
  const int hd = kv.hd, half = hd >> 1, Hkv = kv.n_kv, q4 = half >> 2;
  float* row = qkv + (size_t)b * (Hq + 2 * Hkv) * hd;
  const int nrot = (Hq + Hkv) * q4, nval = Hkv * hd / 4;  // slices
  float4 a[MAXI], bb[MAXI], v[MAXI];
#pragma unroll
  for (int k = 0; k < MAXI; ++k) {
    const int i = min(tid + 256 * k, nrot - 1), h = i / q4, j = 4 * (i % q4);
    a[k] = *reinterpret_cast<const float4*>(row + h * hd + j);
    bb[k] = *reinterpret_cast<const float4*>(row + h * hd + j + half);
    v[k] = *reinterpret_cast<const float4*>(row + (Hq + Hkv) * hd + 4 * min(tid + 256 * k, nval - 1));
  }
  const int pos = static_cast<const DecodeState*>(sd.state)->pos;
  KT* base = reinterpret_cast<KT*>(static_cast<char*>(sd.kv) + (size_t)layer * sd.kv_layer_stride);
  const int phys = sd.table[pos / kv.page], slot = pos % kv.page;
  float4 c[MAXI], sn[MAXI];
#pragma unroll
  for (int k = 0; k < MAXI; ++k) {
    const int i = min(tid + 256 * k, nrot - 1), j = 4 * (i % q4);
    c[k] = *reinterpret_cast<const float4*>(cos_t + (size_t)pos * half + j);
    sn[k] = *reinterpret_cast<const float4*>(sin_t + (size_t)pos * half + j);
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
      ra.x = a[k].x * c[k].x - bb[k].x * sn[k].x; rb.x = a[k].x * sn[k].x + bb[k].x * c[k].x;
      ra.y = a[k].y * c[k].y - bb[k].y * sn[k].y; rb.y = a[k].y * sn[k].y + bb[k].y * c[k].y;
      ra.z = a[k].z * c[k].z - bb[k].z * sn[k].z; rb.z = a[k].z * sn[k].z + bb[k].z * c[k].z;
      ra.w = a[k].w * c[k].w - bb[k].w * sn[k].w; rb.w = a[k].w * sn[k].w + bb[k].w * c[k].w;
      if (h < Hq) {
        float* z = row + h * hd;
        *reinterpret_cast<float4*>(z + j) =
            make_float4(ra.x * q_scale, ra.y * q_scale, ra.z * q_scale, ra.w * q_scale);
        *reinterpret_cast<float4*>(z + j + half) =
            make_float4(rb.x * q_scale, rb.y * q_scale, rb.z * q_scale, rb.w * q_scale);
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

hipError_t launch_rope_append_batch(bool kv_bf16, float* qkv, int B, int Hq, const float* cos_t,
                                    const float* sin_t, const SeqDesc* seqs, int layer,
                                    KvLayout kv, float q_scale, hipStream_t st) {
  constexpr int MAXI = 4;
  if (kv.hd % 8 == 0 && (Hq + kv.n_kv) * (kv.hd / 8) <= 256 * MAXI &&
      kv.n_kv * kv.hd / 4 <= 256 * MAXI) {
    if (kv_bf16)
      hipLaunchKernelGGL((k_rope_append_batch4<bf16_t, MAXI>), dim3(B), dim3(256), 0, st, qkv,
                         Hq, cos_t, sin_t, seqs, layer, kv, q_scale);
    else
      hipLaunchKernelGGL((k_rope_append_batch4<float, MAXI>), dim3(B), dim3(256), 0, st, qkv,
                         Hq, cos_t, sin_t, seqs, layer, kv, q_scale);
    return hipGetLastError();
  }
  if (kv_bf16)
    hipLaunchKernelGGL(k_rope_append_batch<bf16_t>, dim3(B), dim3(256), 0, st, qkv, Hq, cos_t,
                       sin_t, seqs, layer, kv, q_scale);
  else
    hipLaunchKernelGGL(k_rope_append_batch<float>, dim3(B), dim3(256), 0, st, qkv, Hq, cos_t,
                       sin_t, seqs, layer, kv, q_scale);
  return hipGetLastError();
}

// Greedy token of each row of logits [B, V] (lowest index among equal maxima;
// a non-finite logit marks the row failed), then sequence b's state advances:
// token, position + 1, and the token recorded in its history.
__global__ __launch_bounds__(1024) void k_argmax_rows(const float* __restrict__ logits, int V,
                                                     const SeqDesc* __restrict__ seqs) {
  __shared__ float sv[16];
  __shared__ int si[16];
  __shared__ int sbad[16];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const float* row = logits + (size_t)b * V;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  int bad = 0;
  // eight loads in flight per thread (one at a time the row's 500 KB took ~47 us
  // of load latency); the comparison picks the same element in any order
  constexpr int U = 8;
  for (int i0 = tid; i0 < V; i0 += 1024 * U) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = row[min(i0 + 1024 * u, V - 1)];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i = i0 + 1024 * u;
      if (i < V) {
        bad |= !isfinite(v[u]);
        if (am_better(v[u], i, bv, bi)) { bv = v[u]; bi = i; }
      }
    }
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
    for (int k = 1; k < 16; ++k) {
      if (am_better(sv[k], si[k], bv, bi)) { bv = sv[k]; bi = si[k]; }
      bad |= sbad[k];
    }
    DecodeState* st = static_cast<DecodeState*>(seqs[b].state);
    const int pos = st->pos + 1;
    const int tok = bad ? -1 : bi;
    st->bad = bad;
    st->token = tok;
    st->pos = pos;
    seqs[b].hist[pos - 1] = tok;
  }
}

hipError_t launch_argmax_rows(const float* logits, int B, int V, const SeqDesc* seqs,
                              hipStream_t st) {
  hipLaunchKernelGGL(k_argmax_rows, dim3(B), dim3(1024), 0, st, logits, V, seqs);
  return hipGetLastError();
}

}  // namespace wici
