// Library-owned device scratch of the allocation-free forward entry point (tfm_layer_fwd_noalloc
// in include/tfm_layer.h).  One file-scope array; every GPU the library runs on holds its own
// copy at its own address until the process ends.  In host code the array's name is only a
// host-side stand-in: its device address is looked up once per device with hipGetSymbolAddress
// (with that device current) and host code uses that pointer alone.
#include <hip/hip_runtime.h>

#include <mutex>

#include "static_scratch.h"

namespace tfm {

namespace {

__device__ __attribute__((aligned(256))) char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];

}  // namespace

hipError_t static_scratch(hipStream_t stream, void** ptr) {
  *ptr = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (stream) {
    // the scratch of the stream's device is the one its kernels may touch: require it current
    hipDevice_t sdev = 0;
    e = hipStreamGetDevice(stream, &sdev);
    if (e != hipSuccess) return e;
    if ((int)sdev != dev) return hipErrorInvalidDevice;
  }
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_ptr[dev] = p;
  }
  *ptr = g_ptr[dev];
  return hipSuccess;
}

}  // namespace tfm
