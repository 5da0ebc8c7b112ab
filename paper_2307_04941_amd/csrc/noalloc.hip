// conv2d_fwd_f32_noalloc: the plain convolution for callers that cannot
// allocate device memory.  The workspace that conv2d_fwd_f32 takes from its
// stream-ordered pool (split-K partials, the NCHW filter copy) comes instead
// from one fixed array per device, placed in device memory when the code
// object is loaded, and the selector only considers plans whose workspace
// fits in it.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <string>
#include <unordered_map>

#include "mg3m.h"
#include "mg3m_internal.h"

namespace {

constexpr size_t kScratchBytes = (size_t)MG3M_NOALLOC_SCRATCH_BYTES;

// The scratch array.  In host code this name is a host-side stand-in: only
// the per-device address from hipGetSymbolAddress is ever passed to kernels.
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct ScratchAddrs {
  std::mutex mu;
  std::unordered_map<int, void*> by_device;
};
ScratchAddrs& scratch_addrs() {
  static ScratchAddrs* s = new ScratchAddrs();   // never destroyed: usable from exit-time destructors
  return *s;
}

// Device address of the scratch array on the device of `stream` (the current
// device for the default stream), looked up once per device with that device
// current, then kept.
int scratch_on(void* stream, void** addr, std::string* err) {
  int dev = 0;
  hipError_t e = stream != nullptr ? hipStreamGetDevice(static_cast<hipStream_t>(stream), &dev)
                                   : hipGetDevice(&dev);
  if (e != hipSuccess) {
    *err = std::string("device of the stream: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  ScratchAddrs& sa = scratch_addrs();
  std::lock_guard<std::mutex> lock(sa.mu);
  auto it = sa.by_device.find(dev);
  if (it != sa.by_device.end()) {
    *addr = it->second;
    return MG3M_OK;
  }
  int prev = 0;
  e = hipGetDevice(&prev);
  if (e == hipSuccess && prev != dev) e = hipSetDevice(dev);
  if (e != hipSuccess) {
    *err = std::string("select the stream's device: ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  void* p = nullptr;
  e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  const hipError_t restore = prev != dev ? hipSetDevice(prev) : hipSuccess;
  if (e != hipSuccess || p == nullptr) {
    *err = std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e);
    return MG3M_ERR_HIP;
  }
  if (restore != hipSuccess) {
    *err = std::string("restore the current device: ") + hipGetErrorString(restore);
    return MG3M_ERR_HIP;
  }
  sa.by_device.emplace(dev, p);
  *addr = p;
  return MG3M_OK;
}

}  // namespace

extern "C" int conv2d_fwd_f32_noalloc(const float* x, const float* w, float* y, int N, int C, int H,
                                      int W, int K, int R, int S, int stride, int pad, int layout,
                                      void* stream) {
  try {
    mg3m::clear_error();
    // the pointer checks of conv2d_fwd_f32, made before the scratch look-up
    if (x == nullptr || w == nullptr || y == nullptr)
      return mg3m::set_error(MG3M_ERR_NULL, "x, w and y must be non-NULL");
    if (((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(w) | reinterpret_cast<uintptr_t>(y)) & 3) != 0)
      return mg3m::set_error(MG3M_ERR_ALIGN, "x, w and y must be 4-byte aligned");
    mg3m::ConvGeom g{N, C, H, W, K, R, S, stride, stride, pad, pad, layout, false};
    g.ws_cap = kScratchBytes;
    // Shape and plan first (host only): a shape that no plan fits is rejected
    // before the scratch array is looked up.
    mg3m::ConvShape s;
    mg3m::Plan p;
    if (int rc = mg3m::conv_plan(g, nullptr, &s, &p)) return rc;
    void* ws = nullptr;
    std::string err;
    if (int rc = scratch_on(stream, &ws, &err)) return mg3m::set_error(rc, err);
    return mg3m::conv_run(x, w, y, g, ws, kScratchBytes, false, nullptr, nullptr, 0, stream);
  } catch (...) {
    return mg3m::set_error(MG3M_ERR_HIP, "unknown exception");
  }
}
