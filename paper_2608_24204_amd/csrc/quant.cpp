// Block-scaled 8-bit weight quantisation on the host (at weight load).
//
// A row of a matrix [rows, cols] is cut into blocks of 32 consecutive weights;
// each block stores one half-precision scale d = fp16(max|w| / 127) and 32 codes
// q = clamp(rint(w / d), -127, 127) (q = 0 when d == 0), all decisions in float32
// with ties to even.  This reads the paper's quantised models (about 8.5 bits
// per weight, Sec. "Experiment Setup", Tab. "model_conf") as 32 bytes of codes
// plus a 2-byte scale per 32 weights.  Codes are stored offset by 128 (q + 128 in
// an unsigned byte) so the GEMV can convert them with the byte-to-float
// instructions; scales are stored as half-precision bit patterns.
#include <cmath>
#include <cstdint>
#include <cstring>
#include <thread>
#include <vector>

#include "../../include/wici.h"

namespace {

float bits_f32(uint32_t u) { float f; std::memcpy(&f, &u, 4); return f; }
uint32_t f32_bits(float f) { uint32_t u; std::memcpy(&u, &f, 4); return u; }

// float32 -> IEEE half, round to nearest, ties to even (subnormals, overflow to
// infinity; NaN stays NaN).
uint16_t f32_to_f16(float f) {
  const uint32_t x = f32_bits(f);
  const uint16_t sign = (uint16_t)((x >> 16) & 0x8000u);
  const uint32_t a = x & 0x7fffffffu;
  if (a >= 0x7f800000u) return sign | (a > 0x7f800000u ? 0x7e00u : 0x7c00u);
  if (a >= 0x477ff000u) return sign | 0x7c00u;  // >= 65520 rounds past 65504
  if (a >= 0x38800000u) {                        // normal half (>= 2^-14)
    const uint32_t e = (a >> 23) - 112u, m = a & 0x7fffffu;
    uint32_t h = (e << 10) | (m >> 13);
    const uint32_t rem = m & 0x1fffu;
    if (rem > 0x1000u || (rem == 0x1000u && (h & 1u))) ++h;  // carries into the exponent
    return sign | (uint16_t)h;
  }
  // subnormal half: multiples of 2^-24; |f| * 2^24 is exact, nearbyint is RNE
  const float scaled = bits_f32(a) * 16777216.0f;
  return sign | (uint16_t)std::nearbyint(scaled);
}

float f16_to_f32(uint16_t h) {
  const uint32_t sign = (uint32_t)(h & 0x8000u) << 16, e = (h >> 10) & 0x1fu, m = h & 0x3ffu;
  if (e == 0) return bits_f32(sign) + (sign ? -1.f : 1.f) * (float)m * (1.0f / 16777216.0f);
  if (e == 31) return bits_f32(sign | 0x7f800000u | (m << 13));
  return bits_f32(sign | ((e + 112u) << 23) | (m << 13));
}

float load_f32(const void* src, int32_t dtype, size_t i) {
  if (dtype == WICI_BF16) {
    const uint16_t b = static_cast<const uint16_t*>(src)[i];
    return bits_f32((uint32_t)b << 16);
  }
  return static_cast<const float*>(src)[i];
}

// rows [r0, r1); returns false on a non-finite weight or an overflowing scale
bool quantize_rows(const void* src, int32_t dtype, int64_t cols, int64_t r0, int64_t r1,
                   uint8_t* codes, uint16_t* scales) {
  const int64_t nb = cols / 32;
  float w[32];
  for (int64_t r = r0; r < r1; ++r)
    for (int64_t b = 0; b < nb; ++b) {
      const size_t base = (size_t)r * cols + (size_t)b * 32;
      float amax = 0.f;
      for (int i = 0; i < 32; ++i) {
        w[i] = load_f32(src, dtype, base + i);
        if (!std::isfinite(w[i])) return false;
        amax = std::fmax(amax, std::fabs(w[i]));
      }
      const uint16_t hd = f32_to_f16(amax / 127.0f);
      if ((hd & 0x7c00u) == 0x7c00u) return false;
      const float d = f16_to_f32(hd);
      scales[(size_t)r * nb + b] = hd;
      uint8_t* q = codes + base;
      for (int i = 0; i < 32; ++i) {
        float c = 0.f;
        if (d != 0.f) {
          c = std::nearbyint(w[i] / d);
          c = std::fmin(std::fmax(c, -127.f), 127.f);
        }
        q[i] = (uint8_t)((int)c + 128);
      }
    }
  return true;
}

}  // namespace

extern "C" wici_status wici_quantize_q8(const void* src, int32_t src_dtype, int64_t rows,
                                        int64_t cols, uint8_t* codes, uint16_t* scales) {
  if (!src || !codes || !scales || rows < 1 || cols < 32 || cols % 32 ||
      (src_dtype != WICI_F32 && src_dtype != WICI_BF16))
    return WICI_E_ARG;
  const int64_t work = rows * cols;
  unsigned nt = std::thread::hardware_concurrency();
  if (nt == 0) nt = 1;
  if (nt > 32) nt = 32;
  if (work < (int64_t)1 << 22) nt = 1;
  if ((int64_t)nt > rows) nt = (unsigned)rows;
  std::vector<char> ok(nt, 1);
  if (nt == 1) {
    ok[0] = quantize_rows(src, src_dtype, cols, 0, rows, codes, scales);
  } else {
    std::vector<std::thread> th;
    for (unsigned t = 0; t < nt; ++t) {
      const int64_t r0 = rows * t / nt, r1 = rows * (t + 1) / nt;
      th.emplace_back([&, t, r0, r1] {
        ok[t] = quantize_rows(src, src_dtype, cols, r0, r1, codes, scales);
      });
    }
    for (auto& x : th) x.join();
  }
  for (char c : ok)
    if (!c) return WICI_E_ARG;
  return WICI_OK;
}
