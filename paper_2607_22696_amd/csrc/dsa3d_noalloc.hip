// dsa3d_backward_noalloc: the backward run in a fixed scratch buffer of the library, for
// callers that cannot allocate device memory.  The buffer is a file-scope device array;
// host code never passes the array's name to a kernel (on the host that name is only a
// stand-in, not a device address): the device address is looked up with
// hipGetSymbolAddress once per device, with that device current, and kept per device.
#include <hip/hip_runtime.h>

#include <mutex>

#include "backward_entry.h"
#include "dsa3d.h"
#include "dsa3d_internal.h"

namespace {

static __device__ __align__(256) unsigned char scratch[DSA3D_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_lock;
void* g_scratch[kMaxDevices];  // device address of `scratch` on each device (null: not yet)

// Address of the current device's scratch array, looked up on the first call on that device.
hipError_t scratch_on_current_device(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> hold(g_lock);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *ptr = g_scratch[dev];
  return hipSuccess;
}

}  // namespace

extern "C" dsa3d_status dsa3d_backward_noalloc(const dsa3d_desc* desc, const void* q,
                                               const void* k, const void* v,
                                               const float* offsets, const void* out,
                                               const float* lse, const void* dout, float* dq,
                                               float* dk, float* dv, float* d_offsets,
                                               hipStream_t stream) {
  const dsa3d::BackwardArgs a{q, k, v, offsets, out, lse, dout, dq, dk, dv, d_offsets};
  dsa3d::Geometry g;
  // every host check (including the size against the scratch) before the device is touched
  const dsa3d_status st =
      dsa3d::check_backward_call(desc, a, nullptr, 0, DSA3D_NOALLOC_SCRATCH_BYTES, &g);
  if (st != DSA3D_OK) return st;
  void* ws = nullptr;
  if (scratch_on_current_device(&ws) != hipSuccess) return DSA3D_ERR_DEVICE;
  const hipError_t e = dsa3d::launch_backward(g, desc->dtype == DSA3D_BF16, q, k, v, nullptr,
                                              offsets, lse, dout, dq, dk, dv, d_offsets, nullptr,
                                              ws, stream, nullptr);
  return e == hipSuccess ? DSA3D_OK : DSA3D_ERR_DEVICE;
}
