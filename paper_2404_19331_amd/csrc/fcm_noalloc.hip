// fcm_noalloc.hip -- fcm_dw_pw_noalloc: the DW->PW module for callers that cannot
// allocate device memory (code under HIP graph capture, tight serving loops, harnesses
// that forbid hipMalloc). A split plan's partial sums go to `scratch`, a fixed device
// array of FCM_NOALLOC_SCRATCH_BYTES that each GPU holds from module load until the
// process ends, instead of a caller workspace.
#include <hip/hip_runtime.h>

#include <mutex>
#include <string>
#include <vector>

#include "fcm_host.h"

namespace fcm {

// Split partial sums of fcm_dw_pw_noalloc ([split][work tile][pixel][channel] fp32 /
// int32). Every split writes all of its partial sums before the combining kernel reads
// them, so the array needs no clearing between calls. In host code this name is only a
// handle: the device address comes from hipGetSymbolAddress, per device.
static __device__ __align__(256) unsigned char scratch[FCM_NOALLOC_SCRATCH_BYTES];

// Device address of the current device's `scratch`, resolved once per device with that
// device current; NULL (and a message) if the runtime cannot resolve it.
static void* scratch_address() {
  static std::mutex mu;
  static std::vector<void*> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) {
    fail(FCM_EDEVICE, "fcm_dw_pw_noalloc: no current HIP device");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(mu);
  if ((int)cache.size() <= dev) cache.resize(dev + 1, nullptr);
  if (!cache[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      fail(FCM_EDEVICE, std::string("fcm_dw_pw_noalloc: hipGetSymbolAddress(scratch) failed: ") + hipGetErrorString(e));
      return nullptr;
    }
    cache[dev] = ptr;
  }
  return cache[dev];
}

}  // namespace fcm

using namespace fcm;

extern "C" fcm_status fcm_dw_pw_noalloc(const fcm_desc* desc, const void* x, const void* w_dw, const void* b_dw,
                                        const void* w_pw, const void* b_pw, void* y, const fcm_plan_t* plan,
                                        void* stream) {
  void* ws = scratch_address();
  if (!ws) return FCM_EDEVICE;
  const void* w[3] = {w_dw, w_pw, nullptr};
  const void* b[3] = {b_dw, b_pw, nullptr};
  // plan NULL: the best plan whose partial sums fit the array; an explicit plan that needs
  // more is refused (FCM_EINVAL) before anything is launched
  return launch_module(FCM_OP_DW_PW, desc, x, w, b, y, plan, ws, (int64_t)FCM_NOALLOC_SCRATCH_BYTES, stream);
}
