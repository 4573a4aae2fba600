// The owner-map buffer of dv_stream_in_noalloc: a static device array, so
// that the call allocates nothing.  The loader reserves one copy per GPU
// when the library's code object is first loaded there; it is held until
// the process ends.  Host code must not pass the array's name to a kernel
// (in host code it names a host-side stand-in): each device's address is
// looked up once, with that device current, and kept.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "../../include/dv.h"

namespace {

static __device__ __align__(256) int32_t scratch[DV_NOALLOC_MAX_BLOCKS];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
int32_t* g_addr[kMaxDevices];  // device address of `scratch` per device, once looked up

}  // namespace

namespace dv {

// The current device's copy of the array: DV_OK and its address, DV_ERR_HIP
// if the runtime cannot name the device or the symbol, DV_ERR_INVALID when
// `stream` (not the null stream) belongs to another device, whose kernels
// would then reach this device's copy, DV_ERR_UNSUPPORTED for a device index
// past the table above.
int noalloc_owner_map(hipStream_t stream, int32_t** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return DV_ERR_HIP;
  if (stream) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice(stream, &sdev) != hipSuccess) return DV_ERR_HIP;
    if (sdev != dev) return DV_ERR_INVALID;
  }
  if (dev < 0 || dev >= kMaxDevices) return DV_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return DV_ERR_HIP;
    g_addr[dev] = static_cast<int32_t*>(p);
  }
  *out = g_addr[dev];
  return DV_OK;
}

}  // namespace dv
