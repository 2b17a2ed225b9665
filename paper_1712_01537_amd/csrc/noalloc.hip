// oc_conv_fwd_noalloc: the convolution forward with its workspace in a
// file-scope device array instead of a caller buffer, for callers that cannot
// allocate device memory (code under graph capture, tight serving loops,
// harnesses that forbid allocation).
//
// The array lives in every device the library runs on until the process
// ends.  Host code never passes the array's name to a kernel (in host code it
// names a host-side stand-in, not device memory): its device address is
// taken once per device with hipGetSymbolAddress, with that device current,
// on the first call there, and kept.  Every call on a device shares that
// device's array and leaves the last call's contents in it; the forward
// writes every workspace entry it reads, so nothing has to start at zero.
// Calls that overlap on one device (on different streams, or from different
// threads without ordering) race on the array.
#include <mutex>

#include "common.h"

namespace {

constexpr size_t SCRATCH_BYTES = size_t(32) << 20;  // 32 MiB per device
constexpr int MAX_DEVICES = 64;

__device__ __align__(256) unsigned char scratch[SCRATCH_BYTES];

std::mutex g_mu;
void* g_ptr[MAX_DEVICES] = {};

// Device address of `scratch` on the current device (taken once per device).
oc_status scratch_ptr(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES)
    return oc::fail(OC_ERR_DEVICE, "oc_conv_fwd_noalloc: no current device");
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return oc::fail(OC_ERR_DEVICE, "oc_conv_fwd_noalloc: scratch address unavailable: %s",
                      hipGetErrorString(e));
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return OC_OK;
}

}  // namespace

extern "C" oc_status oc_conv_fwd_noalloc(const oc_octree* t, int32_t l, int32_t K,
                                         int32_t stride, oc_dtype dt, const void* x, int32_t cin,
                                         const void* w, int32_t cout, float* y, int32_t flags,
                                         hipStream_t s) {
  oc_status st = oc::conv_check(t, l, K, stride, dt, cin, cout, "oc_conv_fwd_noalloc");
  if (st != OC_OK) return st;
  if (stride != 1)  // the strided forward may call the GEMM library, which allocates
    return oc::fail(OC_ERR_UNSUPPORTED, "oc_conv_fwd_noalloc: stride %d not supported", stride);
  const size_t need = oc_conv_fwd_workspace(t, l, K, stride, dt, cin, cout);
  if (need > SCRATCH_BYTES)
    return oc::fail(OC_ERR_UNSUPPORTED,
                    "oc_conv_fwd_noalloc: this call needs %zu bytes of workspace, more than the "
                    "%zu of the static scratch; use oc_conv_fwd with a workspace",
                    need, SCRATCH_BYTES);
  void* p = nullptr;
  if (need) {
    st = scratch_ptr(&p);
    if (st != OC_OK) return st;
  }
  return oc_conv_fwd(t, l, K, stride, dt, x, cin, w, cout, y, p, need, flags, s);
}
