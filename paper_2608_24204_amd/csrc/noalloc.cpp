// The streaming-read diagnostic for callers that cannot allocate device memory
// (code under HIP graph capture, serving loops that must not allocate, harnesses
// that forbid it).  wici_stream_read takes its workspace (per-thread partial
// results, then their XOR) from the caller; wici_stream_read_noalloc keeps it in
// the file-scope device array below instead, so the call allocates nothing.
//
// The array is one per GPU: each device that loads this library holds its own
// copy, at its own address, until the process ends.  Host code must never pass
// the array's name to a kernel (on the host it is only a stand-in for the
// symbol): its device address is looked up once per device, with that device
// current, on the first call there, and kept.  Every call on a GPU uses that
// GPU's copy, so calls that overlap on one GPU race; the partial results of a
// call are all written before they are read, so nothing has to start at zero.
#include <hip/hip_runtime.h>

#include <mutex>

#include "common.h"
#include "kernels.h"
#include "wici.h"

namespace {

constexpr int kMaxGrid = 4096;                         // workgroups of one read
constexpr size_t kResult = (size_t)256 * kMaxGrid;     // word holding the checksum
constexpr size_t kScratchWords = kResult + 64;         // 4 MiB + 256 bytes

static __device__ __align__(256) unsigned scratch[kScratchWords];

constexpr int kMaxDevices = 64;
std::mutex g_mutex;
unsigned* g_scratch[kMaxDevices] = {};

// Device address of `scratch` on the current device (looked up on first use).
hipError_t scratch_here(unsigned** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = static_cast<unsigned*>(p);
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

}  // namespace

extern "C" wici_status wici_stream_read_noalloc(const void* d_buf, size_t bytes, int32_t grid,
                                                void* hip_stream, uint32_t* checksum) {
  if (!d_buf || !checksum || grid < 1 || bytes < 16384 || bytes % 16384) return WICI_E_ARG;
  if (grid > kMaxGrid) return WICI_E_ARG;
  unsigned* s = nullptr;
  if (scratch_here(&s) != hipSuccess) return WICI_E_HIP;
  hipStream_t st = static_cast<hipStream_t>(hip_stream);
  hipError_t e = wici::launch_stream_read(d_buf, bytes, grid, s, st);
  if (e == hipSuccess) e = wici::launch_xor_reduce(s, 256 * grid, s + kResult, st);
  if (e == hipSuccess) e = hipMemcpyAsync(checksum, s + kResult, 4, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  return e == hipSuccess ? WICI_OK : WICI_E_HIP;
}
