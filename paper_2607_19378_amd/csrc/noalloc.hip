// hyenand_fftconv_noalloc: the gated FFT convolution for callers that cannot
// allocate device memory (code under HIP graph capture, serving loops,
// harnesses that forbid hipMalloc).  It is hyenand_fftconv with the
// library's own device scratch as the workspace: one file-scope array per
// GPU, reserved when the library's code object is loaded there and kept
// until the process ends.
#include <stdio.h>

#include <mutex>

#include <hip/hip_runtime.h>

#include "../../include/hyenand.h"

namespace hyenand {
hyenand_status set_last_error(hyenand_status s, const char* msg);
}

namespace {

constexpr size_t kScratchBytes = size_t(128) << 20;

// The scratch array.  In host code its name stands for a host-side shadow,
// not a device address: only the per-device pointer that
// hipGetSymbolAddress returns is ever passed on.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
struct DeviceScratch {
  std::once_flag once;
  hipError_t err = hipSuccess;
  void* ptr = nullptr;
};
DeviceScratch g_scratch[kMaxDevices];

// This device's copy of the array, looked up once per device with that
// device current.
hipError_t scratch_on(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  DeviceScratch& d = g_scratch[dev];
  std::call_once(d.once, [&d, dev] {
    int prev = 0;
    d.err = hipGetDevice(&prev);
    if (d.err == hipSuccess && prev != dev) d.err = hipSetDevice(dev);
    if (d.err == hipSuccess) d.err = hipGetSymbolAddress(&d.ptr, HIP_SYMBOL(scratch));
    if (prev != dev) {
      const hipError_t r = hipSetDevice(prev);
      if (d.err == hipSuccess) d.err = r;
    }
    if (d.err == hipSuccess && d.ptr == nullptr) d.err = hipErrorInvalidSymbol;
  });
  *out = d.ptr;
  return d.err;
}

}  // namespace

extern "C" {

hyenand_status hyenand_fftconv_noalloc(const void* x1, const void* x2, const void* v, const void* k,
                                       const void* D, void* y, int ndim, const int64_t* dims,
                                       hyenand_pad_mode pad_mode, hyenand_dtype dtype, void* stream) {
  size_t need = 0;
  const hyenand_status st = hyenand_fftconv_workspace_min(ndim, dims, pad_mode, dtype, &need);
  if (st != HYENAND_OK) return st;
  if (need > kScratchBytes) {
    char msg[256];
    snprintf(msg, sizeof msg,
             "this shape needs %zu bytes of workspace; the no-allocation entry point's scratch holds %zu "
             "(use hyenand_fftconv with a workspace)",
             need, kScratchBytes);
    return hyenand::set_last_error(HYENAND_ERR_UNSUPPORTED, msg);
  }
  if (!x1 || !x2 || !v || !k || !D || !y)
    return hyenand::set_last_error(HYENAND_ERR_INVALID_ARGUMENT, "a tensor pointer is NULL");
  void* ws = nullptr;
  size_t ws_bytes = 0;
  if (need > 0) {  // the single-pass plans use no workspace and never touch the scratch
    int dev = 0;
    hipError_t e = stream ? hipStreamGetDevice((hipStream_t)stream, &dev) : hipGetDevice(&dev);
    if (e == hipSuccess) e = scratch_on(dev, &ws);
    if (e != hipSuccess) {
      char msg[256];
      snprintf(msg, sizeof msg, "device scratch lookup: HIP error %d: %s", (int)e, hipGetErrorString(e));
      return hyenand::set_last_error(HYENAND_ERR_HIP, msg);
    }
    ws_bytes = kScratchBytes;
  }
  return hyenand_fftconv(x1, x2, v, k, D, y, ndim, dims, pad_mode, dtype, ws, ws_bytes, stream);
}

}  // extern "C"
