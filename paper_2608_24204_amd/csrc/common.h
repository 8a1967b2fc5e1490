// Device-side helpers shared by the HIP kernels of libwici (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wici {

typedef uint16_t bf16_t;  // bf16 bit pattern in memory

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(bf16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// Nearest bf16 (ties to even; NaN stays NaN): gfx950's packed conversion
// instruction (v_cvt_pk_bf16_f32), one instruction for two values instead of the
// integer rounding sequence.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, static_cast<__bf16>(f));
}

// Storage conversions for the two supported element types.
template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ __forceinline__ static float load(const float* p) { return *p; }
  __device__ __forceinline__ static float round(float v) { return v; }
  __device__ __forceinline__ static void store(float* p, float v) { *p = v; }
};
template <> struct Elem<bf16_t> {
  __device__ __forceinline__ static float load(const bf16_t* p) { return bf16_to_f32(*p); }
  __device__ __forceinline__ static float round(float v) { return bf16_to_f32(f32_to_bf16(v)); }
  __device__ __forceinline__ static void store(bf16_t* p, float v) { *p = f32_to_bf16(v); }
};

// Load 8 consecutive elements (16-byte aligned for bf16, 32-byte for fp32) as fp32.
__device__ __forceinline__ void load8(const bf16_t* p, float* o) {
  uint4 v = *reinterpret_cast<const uint4*>(p);
  o[0] = __uint_as_float(v.x << 16); o[1] = __uint_as_float(v.x & 0xffff0000u);
  o[2] = __uint_as_float(v.y << 16); o[3] = __uint_as_float(v.y & 0xffff0000u);
  o[4] = __uint_as_float(v.z << 16); o[5] = __uint_as_float(v.z & 0xffff0000u);
  o[6] = __uint_as_float(v.w << 16); o[7] = __uint_as_float(v.w & 0xffff0000u);
}
__device__ __forceinline__ void load8(const float* p, float* o) {
  float4 a = reinterpret_cast<const float4*>(p)[0];
  float4 b = reinterpret_cast<const float4*>(p)[1];
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
  o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}

// ---- cross-lane reductions -------------------------------------------------------
// DPP row operations move data between lanes of a 16-lane row inside the VALU
// (a few cycles) instead of through the LDS crossbar (ds_bpermute, ~100 cycles).
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}
constexpr int kDppXor1 = 0xb1;         // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4e;         // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // lane i <-> 7-i within each 8 lanes
constexpr int kDppMirror = 0x140;      // lane i <-> 15-i within each 16 lanes

// Sum over aligned groups of N lanes (N = 2, 4, 8, 16, 32 or 64); every lane of a
// group receives the group's sum.
template <int N>
__device__ __forceinline__ float group_sum(float v) {
  if (N >= 2) v += dpp<kDppXor1>(v);
  if (N >= 4) v += dpp<kDppXor2>(v);
  if (N >= 8) v += dpp<kDppHalfMirror>(v);
  if (N >= 16) v += dpp<kDppMirror>(v);
  if (N >= 32) v += __shfl_xor(v, 16);
  if (N >= 64) v += __shfl_xor(v, 32);
  return v;
}
template <int N>
__device__ __forceinline__ float group_max(float v) {
  if (N >= 2) v = fmaxf(v, dpp<kDppXor1>(v));
  if (N >= 4) v = fmaxf(v, dpp<kDppXor2>(v));
  if (N >= 8) v = fmaxf(v, dpp<kDppHalfMirror>(v));
  if (N >= 16) v = fmaxf(v, dpp<kDppMirror>(v));
  if (N >= 32) v = fmaxf(v, __shfl_xor(v, 16));
  if (N >= 64) v = fmaxf(v, __shfl_xor(v, 32));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) { return group_sum<64>(v); }
__device__ __forceinline__ float wave_max(float v) { return group_max<64>(v); }

// Sum over a 256-thread block; every thread gets the result.  `red` holds >= 4 floats.
__device__ __forceinline__ float block256_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

__device__ __forceinline__ float silu(float z) { return z / (1.0f + expf(-z)); }

// Activation operands of the prefill matrix products.  With nt = 0 the values are
// stored as fp32; with nt = 1..3 each fp32 value v is stored as nt bf16 terms in
// separate planes (plane_stride elements apart): t0 = bf16(v), t1 = bf16(v - t0),
// t2 = bf16(v - t0 - t1).  Each subtraction is exact in fp32, so three terms
// carry v to about 2^-24 relative and the sum of the terms' products with exact
// bf16 weights is an fp32-accurate product.
struct ActBuf {
  float* f32;         // nt == 0
  bf16_t* planes;     // nt >= 1: [nt][rows][ld]
  size_t plane_stride;
  int nt;
};

__device__ __forceinline__ void store_act(const ActBuf& a, size_t idx, float v) {
  if (a.nt == 0) {
    a.f32[idx] = v;
    return;
  }
  float r = v;
  for (int p = 0; p < a.nt; ++p) {
    const bf16_t t = f32_to_bf16(r);
    a.planes[p * a.plane_stride + idx] = t;
    r -= bf16_to_f32(t);
  }
}

// Four consecutive values (idx a multiple of 4): the same terms as four
// store_act calls, written as one 8-byte store per plane (16 bytes for fp32).
__device__ __forceinline__ void store_act4(const ActBuf& a, size_t idx, float4 v) {
  if (a.nt == 0) {
    *reinterpret_cast<float4*>(a.f32 + idx) = v;
    return;
  }
  float r[4] = {v.x, v.y, v.z, v.w};
  for (int p = 0; p < a.nt; ++p) {
    bf16_t t[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      t[e] = f32_to_bf16(r[e]);
      r[e] -= bf16_to_f32(t[e]);
    }
    *reinterpret_cast<uint2*>(a.planes + p * a.plane_stride + idx) =
        make_uint2((uint32_t)t[0] | ((uint32_t)t[1] << 16), (uint32_t)t[2] | ((uint32_t)t[3] << 16));
  }
}

// Greedy-argmax order: larger value wins, lower index wins among equal values.
__device__ __forceinline__ bool am_better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

struct DecodeState {  // device-resident step state
  int32_t pos;        // number of cached positions
  int32_t token;      // last emitted (or host-given) token
  int32_t bad;        // nonzero: a logit was NaN/Inf in the last argmax
  int32_t fault;      // nonzero: the split blocks of an in-launch merge (a decode
                      // attention's KV head, a batched product's tile) ran on
                      // different XCDs; sticky until reset
  int32_t done;       // host mirror only: set to 1 by the final argmax kernel after
                      // the fields above (the host clears it before the step)
};

// ---- exchange between the workgroups of one XCD (in-launch merges) ----------
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

// The XCC (XCD) the wavefront runs on: hardware register XCC_ID, bits 0-3.
__device__ __forceinline__ int xcc_id() {
  return (int)(__builtin_amdgcn_s_getreg((20) | (0 << 6) | ((4 - 1) << 11)) & 0xf);
}

// 16 bytes at byte offset `off` of the buffer `r`, read past the L1 (sc0).
__device__ __forceinline__ u32x4_t load_l2(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 1);
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, size_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
}

}  // namespace wici
