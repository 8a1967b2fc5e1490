// Drives wici_md5 (host code) over RFC 1321 suite messages, every length up to
// 300 bytes and a few large ones, each in an exactly sized heap buffer; built by
// the test suite under the address and undefined-behaviour sanitizers.
#include <cstdint>
#include <initializer_list>
#include <cstdio>
#include <cstring>
#include <cstdlib>
#include "../../include/wici.h"
int main() {
  int bad = 0;
  struct { const char* m; const char* d; } suite[] = {
    {"", "d41d8cd98f00b204e9800998ecf8427e"}, {"abc", "900150983cd24fb0d6963f7d28e17f72"},
    {"message digest", "f96b697d7cb7938d525a2f31aaf161d0"}};
  for (auto& t : suite) {
    size_t n = std::strlen(t.m);
    uint8_t* buf = (uint8_t*)std::malloc(n ? n : 1);
    std::memcpy(buf, t.m, n);
    uint8_t out[16]; char hex[33];
    if (wici_md5(buf, n, out) != WICI_OK) ++bad;
    for (int i = 0; i < 16; ++i) std::snprintf(hex + 2 * i, 3, "%02x", out[i]);
    if (std::strcmp(hex, t.d)) { std::printf("digest mismatch for '%s'\n", t.m); ++bad; }
    std::free(buf);
  }
  // every length up to 300 bytes and a few large ones, buffers sized exactly
  for (size_t n : {0ul, 1ul, 55ul, 56ul, 63ul, 64ul, 65ul, 119ul, 120ul, 127ul, 128ul, 129ul, 300ul, 1000003ul, 8388608ul}) {
    uint8_t* buf = (uint8_t*)std::malloc(n ? n : 1);
    for (size_t i = 0; i < n; ++i) buf[i] = (uint8_t)(i * 131 + 7);
    uint8_t out[16];
    if (wici_md5(buf, n, out) != WICI_OK) ++bad;
    std::free(buf);
  }
  for (size_t n = 0; n <= 300; ++n) {
    uint8_t* buf = (uint8_t*)std::malloc(n ? n : 1);
    std::memset(buf, 0x5a, n);
    uint8_t out[16];
    if (wici_md5(buf, n, out) != WICI_OK) ++bad;
    std::free(buf);
  }
  if (wici_md5(nullptr, 4, nullptr) == WICI_OK) ++bad;
  std::printf("%s (%d problems)\n", bad ? "FAIL" : "ok", bad);
  return bad != 0;
}
