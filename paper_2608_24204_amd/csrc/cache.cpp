// Content-addressed weight loading (the paper's model caching, Sec. "Model
// Caching"): a tensor above a size threshold is named by the MD5 of its bytes;
// the library keeps a store of such tensors as files named by the hash, so a
// caller that sends only hashes has every stored tensor loaded from the store
// and uploads just the misses, which are then saved.  Tensors below the
// threshold are always sent (hashing them costs more than sending them).
//
// MD5 follows RFC 1321: 64-byte blocks, four rounds of sixteen steps with the
// per-step constants floor(2^32 |sin(i + 1)|) and rotations of the RFC,
// little-endian words, the message length in bits appended after a 1 bit.
#include <algorithm>
#include <array>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include <hip/hip_runtime.h>

#include "../../include/wici.h"

namespace {

struct Md5 {
  uint32_t h[4] = {0x67452301u, 0xefcdab89u, 0x98badcfeu, 0x10325476u};
  uint64_t len = 0;
  uint8_t buf[64];
  size_t nbuf = 0;

  static uint32_t K(int i) {  // floor(2^32 * |sin(i + 1)|), built once (thread-safe)
    static const std::array<uint32_t, 64> k = [] {
      std::array<uint32_t, 64> t{};
      for (int j = 0; j < 64; ++j)
        t[j] = (uint32_t)(std::fabs(std::sin((double)(j + 1))) * 4294967296.0);
      return t;
    }();
    return k[i];
  }
  static uint32_t rol(uint32_t x, int c) { return (x << c) | (x >> (32 - c)); }

  void block(const uint8_t* p) {
    static const int r[4][4] = {{7, 12, 17, 22}, {5, 9, 14, 20}, {4, 11, 16, 23}, {6, 10, 15, 21}};
    uint32_t w[16];
    for (int i = 0; i < 16; ++i)
      w[i] = (uint32_t)p[4 * i] | (uint32_t)p[4 * i + 1] << 8 | (uint32_t)p[4 * i + 2] << 16 |
             (uint32_t)p[4 * i + 3] << 24;
    uint32_t a = h[0], b = h[1], c = h[2], d = h[3];
    for (int i = 0; i < 64; ++i) {
      uint32_t f;
      int g;
      const int round = i / 16;
      if (round == 0) { f = (b & c) | (~b & d); g = i; }
      else if (round == 1) { f = (d & b) | (~d & c); g = (5 * i + 1) % 16; }
      else if (round == 2) { f = b ^ c ^ d; g = (3 * i + 5) % 16; }
      else { f = c ^ (b | ~d); g = (7 * i) % 16; }
      const uint32_t t = d;
      d = c;
      c = b;
      b = b + rol(a + f + K(i) + w[g], r[round][i % 4]);
      a = t;
    }
    h[0] += a; h[1] += b; h[2] += c; h[3] += d;
  }
  void update(const uint8_t* p, size_t n) {
    len += n;
    if (nbuf) {
      const size_t take = std::min(n, 64 - nbuf);
      std::memcpy(buf + nbuf, p, take);
      nbuf += take; p += take; n -= take;
      if (nbuf == 64) { block(buf); nbuf = 0; }
    }
    for (; n >= 64; p += 64, n -= 64) block(p);
    if (n) { std::memcpy(buf, p, n); nbuf = n; }
  }
  void final(uint8_t out[16]) {
    const uint64_t bits = len * 8;
    const uint8_t one = 0x80, zero = 0;
    update(&one, 1);
    while (nbuf != 56) update(&zero, 1);
    uint8_t l[8];
    for (int i = 0; i < 8; ++i) l[i] = (uint8_t)(bits >> (8 * i));
    update(l, 8);
    for (int i = 0; i < 4; ++i)
      for (int j = 0; j < 4; ++j) out[4 * i + j] = (uint8_t)(h[i] >> (8 * j));
  }
};

std::string hex(const uint8_t* md5) {
  static const char* d = "0123456789abcdef";
  std::string s(32, '0');
  for (int i = 0; i < 16; ++i) { s[2 * i] = d[md5[i] >> 4]; s[2 * i + 1] = d[md5[i] & 15]; }
  return s;
}

bool read_file(const std::string& path, size_t bytes, std::vector<char>* out) {
  FILE* f = std::fopen(path.c_str(), "rb");
  if (!f) return false;
  std::fseek(f, 0, SEEK_END);
  const long n = std::ftell(f);
  std::fseek(f, 0, SEEK_SET);
  bool ok = n >= 0 && (size_t)n == bytes;
  if (ok) {
    out->resize(bytes);
    ok = std::fread(out->data(), 1, bytes, f) == bytes;
  }
  std::fclose(f);
  return ok;
}

bool write_file(const std::string& path, const void* data, size_t bytes) {
  const std::string tmp = path + ".part";
  FILE* f = std::fopen(tmp.c_str(), "wb");
  if (!f) return false;
  const bool ok = std::fwrite(data, 1, bytes, f) == bytes;
  if (std::fclose(f) != 0 || !ok) { std::remove(tmp.c_str()); return false; }
  return std::rename(tmp.c_str(), path.c_str()) == 0;
}

size_t tensor_bytes(const wici_tensor& t) {
  const size_t n = (size_t)t.shape[0] * (t.ndim == 2 ? (size_t)t.shape[1] : 1);
  return n * (t.dtype == WICI_BF16 ? 2 : 4);
}

}  // namespace

extern "C" wici_status wici_md5(const void* data, size_t bytes, uint8_t* out16) {
  if ((!data && bytes) || !out16) return WICI_E_ARG;
  Md5 m;
  m.update(static_cast<const uint8_t*>(data), bytes);
  m.final(out16);
  return WICI_OK;
}

extern "C" wici_status wici_load_weights_cached(wici_model* m, const wici_tensor* tensors,
                                                const uint8_t* hashes, int32_t n_tensors,
                                                const char* store_dir, int64_t threshold_bytes,
                                                int32_t* outcome) {
  if (!m) return WICI_E_ARG;
  if (n_tensors < 0 || (n_tensors > 0 && (!tensors || !outcome)) || !store_dir ||
      threshold_bytes < 0)
    return WICI_E_ARG;
  // decide each tensor's source before uploading anything
  std::vector<wici_tensor> up;
  std::vector<std::vector<char>> bufs(n_tensors);
  std::vector<std::pair<std::string, int>> to_save;  // (path, index into up)
  for (int i = 0; i < n_tensors; ++i) {
    wici_tensor t = tensors[i];
    if (t.ndim < 1 || t.ndim > 2 || t.shape[0] < 0 || (t.ndim == 2 && t.shape[1] < 0))
      return WICI_E_ARG;
    const size_t bytes = tensor_bytes(t);
    if ((int64_t)bytes < threshold_bytes) {  // always sent
      if (!t.data) return WICI_E_ARG;
      outcome[i] = WICI_CACHE_SENT;
      up.push_back(t);
      continue;
    }
    uint8_t md5[16];
    if (hashes) {
      std::memcpy(md5, hashes + 16 * (size_t)i, 16);
    } else {
      if (!t.data) return WICI_E_ARG;
      std::vector<char> host;
      const void* src = t.data;
      if (t.on_device) {
        host.resize(bytes);
        if (hipMemcpy(host.data(), t.data, bytes, hipMemcpyDeviceToHost) != hipSuccess)
          return WICI_E_HIP;
        src = host.data();
      }
      wici_md5(src, bytes, md5);
    }
    const std::string path = std::string(store_dir) + "/" + hex(md5);
    if (read_file(path, bytes, &bufs[i])) {
      t.data = bufs[i].data();
      t.on_device = 0;
      outcome[i] = WICI_CACHE_HIT;
      up.push_back(t);
    } else if (t.data) {
      if (hashes) {
        // the file will be named by this hash: a given hash must be the data's
        // own, or the store would serve the wrong tensor for it from then on
        std::vector<char> host;
        const void* src = t.data;
        if (t.on_device) {
          host.resize(bytes);
          if (hipMemcpy(host.data(), t.data, bytes, hipMemcpyDeviceToHost) != hipSuccess)
            return WICI_E_HIP;
          src = host.data();
        }
        uint8_t own[16];
        wici_md5(src, bytes, own);
        if (std::memcmp(own, md5, 16) != 0) return WICI_E_ARG;
      }
      outcome[i] = WICI_CACHE_SAVED;
      to_save.emplace_back(path, (int)up.size());
      up.push_back(t);
    } else {
      outcome[i] = WICI_CACHE_NEEDED;
    }
  }
  const wici_status st = wici_load_weights(m, up.data(), (int32_t)up.size());
  if (st != WICI_OK) return st;
  for (const auto& s : to_save) {
    const wici_tensor& t = up[s.second];
    const size_t bytes = tensor_bytes(t);
    std::vector<char> host;
    const void* src = t.data;
    if (t.on_device) {
      host.resize(bytes);
      if (hipMemcpy(host.data(), t.data, bytes, hipMemcpyDeviceToHost) != hipSuccess)
        return WICI_E_HIP;
      src = host.data();
    }
    (void)write_file(s.first, src, bytes);  // a store that cannot be written only costs hits
  }
  return WICI_OK;
}
