// The allocation-free forward entry point: fno_spectral_conv_fwd with the
// workspace taken from a fixed device array of this library instead of the
// caller's buffer, for callers that cannot allocate device memory (code
// under HIP graph capture, serving loops, harnesses that forbid it).
//
// `scratch` is a file-scope device array of FNO_NOALLOC_SCRATCH_BYTES; every
// GPU the library runs on holds its own copy until the process ends.  Host
// code never passes the array's name to a kernel or a copy: its device
// address is looked up once per device (hipGetSymbolAddress, with that
// device current, on the entry point's first call there) and that address
// is what the forward call receives as its workspace.  Calls share the
// array: two calls that overlap on one GPU race on it.  No kernel of the
// forward path needs the workspace cleared, so nothing is zeroed.
#include <hip/hip_runtime.h>

#include <mutex>

#include "fno_host.h"

namespace {

static __device__ __align__(256) unsigned char scratch[FNO_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch`.
fno_status scratch_for_current_device(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return FNO_ERR_HIP;
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return FNO_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FNO_OK;
}

}  // namespace

extern "C" fno_status fno_spectral_conv_fwd_noalloc(const fno_conv_desc* desc, const void* x,
                                                     const fno_weights* w, void* y,
                                                     void* x_hat_out, hipStream_t stream) {
  void* ws = nullptr;
  const fno_status st = scratch_for_current_device(&ws);
  if (st != FNO_OK) return st;
  return fno::fwd_impl(desc, x, w, y, x_hat_out, ws, FNO_NOALLOC_SCRATCH_BYTES, stream, false);
}
