// Drives wici_quantize_q8 (host code) over small and threaded shapes, f32 and
// bf16 inputs, zeros, subnormals, a non-finite weight and an overflowing block
// scale, plus argument errors, on exactly sized buffers; built by the test suite
// under the compiler's address, undefined-behaviour and thread sanitizers.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <random>
#include <vector>
#include "../../include/wici.h"

static uint16_t to_bf16(float f) { uint32_t u; std::memcpy(&u, &f, 4); return (uint16_t)((u + 0x7fff + ((u >> 16) & 1)) >> 16); }

static int run(int64_t rows, int64_t cols, int dtype, int mode, unsigned seed) {
  std::mt19937 g(seed);
  std::normal_distribution<float> nd(0.f, 0.02f);
  std::vector<float> f((size_t)rows * cols);
  for (auto& v : f) v = nd(g);
  if (mode == 1) for (size_t i = 0; i < f.size(); i += 97) f[i] = 0.f;          // zeros
  if (mode == 2) for (size_t i = 0; i < f.size(); ++i) f[i] = 1e-40f * (i % 7);  // subnormals
  if (mode == 3) f[f.size() / 2] = NAN;                                           // non-finite
  if (mode == 4) f[0] = 1e9f;                                                     // scale overflow
  std::vector<uint16_t> b(f.size());
  for (size_t i = 0; i < f.size(); ++i) b[i] = to_bf16(f[i]);
  std::vector<uint8_t> codes(f.size());
  std::vector<uint16_t> scales(f.size() / 32);
  const void* src = dtype == WICI_F32 ? (const void*)f.data() : (const void*)b.data();
  return wici_quantize_q8(src, dtype, rows, cols, codes.data(), scales.data());
}

int main(int argc, char** argv) {
  // "threads": only the shapes large enough for the threaded path (for the
  // thread sanitizer); otherwise every shape, dtype and input kind
  const bool threads_only = argc > 1 && std::strcmp(argv[1], "threads") == 0;
  int bad = 0;
  const int64_t shapes[][2] = {{1, 32}, {3, 64}, {7, 4096}, {1024, 4096}, {2048, 2080}, {4097, 1024}};
  for (auto& s : shapes)
    for (int dt : {WICI_F32, WICI_BF16})
      for (int mode = 0; mode < 5; ++mode) {
        if (threads_only && (s[0] * s[1] < ((int64_t)1 << 22) || (mode != 0 && mode != 3))) continue;
        int r = run(s[0], s[1], dt, mode, 1234 + mode);
        int want = (mode == 3 || mode == 4) ? WICI_E_ARG : WICI_OK;
        if (r != want) { std::printf("rows %lld cols %lld dtype %d mode %d -> %d (want %d)\n", (long long)s[0], (long long)s[1], dt, mode, r, want); ++bad; }
      }
  uint8_t c[64]; uint16_t sc[2]; float x[64] = {0};
  if (wici_quantize_q8(nullptr, WICI_F32, 1, 64, c, sc) != WICI_E_ARG) ++bad;
  if (wici_quantize_q8(x, WICI_F32, 1, 48, c, sc) != WICI_E_ARG) ++bad;
  if (wici_quantize_q8(x, 7, 1, 64, c, sc) != WICI_E_ARG) ++bad;
  if (wici_quantize_q8(x, WICI_F32, 0, 64, c, sc) != WICI_E_ARG) ++bad;
  std::printf("%s (%d mismatches)\n", bad ? "FAIL" : "ok", bad);
  return bad != 0;
}
