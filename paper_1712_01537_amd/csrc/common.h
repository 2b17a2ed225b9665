// Internal declarations shared by the HIP sources of liboc.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdint>
#include <cstdio>

#include "oc.h"

constexpr int OC_MAX_DEPTH = 8;

struct oc_octree {
  int32_t depth = 0, full_depth = 0, batch = 0;
  int64_t N[OC_MAX_DEPTH + 1] = {};
  int64_t M[OC_MAX_DEPTH + 1] = {};
  uint32_t* keys[OC_MAX_DEPTH + 1] = {};
  int32_t* labels[OC_MAX_DEPTH + 1] = {};
  int32_t* rows[OC_MAX_DEPTH + 1] = {};
  int32_t* nbr[OC_MAX_DEPTH + 1] = {};
  float* signal = nullptr;
  void* block = nullptr;
  oc_allocator alloc{};
  hipStream_t stream = nullptr;
};

namespace oc {

// Thread-local message of the last failure, returned by oc_last_error().
void set_error(const char* fmt, ...);
oc_status fail(oc_status s, const char* fmt, ...);

// Allocation through the caller's allocator, or hipMalloc when none.
void* dev_alloc(const oc_allocator& a, size_t bytes, hipStream_t s);
void dev_free(const oc_allocator& a, void* p, hipStream_t s);

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align256(size_t v) { return (v + 255) & ~size_t(255); }

// Check a level argument and return its sizes.
oc_status check_tree_level(const oc_octree* t, int32_t l, int32_t min_l);

// Argument checks of a convolution call (depth, kernel size, stride, dtype,
// channel counts), as oc_conv_fwd and oc_conv_bwd do them; `who` names the
// caller in the message.
oc_status conv_check(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                     int32_t cin, int32_t cout, const char* who);

// Compute units of the current device (cached per device).
int cu_count();

// Fill n 32-bit words of dev memory with v (a kernel, not a memset node).
void fill_u32(void* p, uint32_t v, int64_t n, hipStream_t s);

// Events set by oc_profile_next for the calling thread, returned once and
// cleared (both null when none are pending).
void take_profile_events(hipEvent_t* start, hipEvent_t* stop);

// The next pair of the event arrays armed by oc_profile_calls for the calling
// thread (both null when none is armed or the arrays are used up).
void take_call_events(hipEvent_t* start, hipEvent_t* stop);

// Launch a kernel of the library; while oc_profile_calls is armed on the
// calling thread it is bracketed by the next pair of the armed events.
template <typename F, typename... Args>
inline void launch(F kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s,
                   Args... args) {
  hipEvent_t a, b;
  take_call_events(&a, &b);
  hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, a, b, 0, args...);
}

// Launch the kernel that does a call's main arithmetic; it takes the
// pending events of oc_profile_next if any, else a pair of oc_profile_calls.
template <typename F, typename... Args>
inline void launch_main(F kernel, dim3 grid, dim3 block, hipStream_t s, Args... args) {
  hipEvent_t a, b;
  take_profile_events(&a, &b);
  if (!a) take_call_events(&a, &b);
  hipExtLaunchKernelGGL(kernel, grid, block, 0, s, a, b, 0, args...);
}

}  // namespace oc

#define OC_HIP_CHECK(call)                                                                    \
  do {                                                                                        \
    hipError_t e_ = (call);                                                                   \
    if (e_ != hipSuccess)                                                                     \
      return oc::fail(OC_ERR_DEVICE, "%s failed: %s", #call, hipGetErrorString(e_));          \
  } while (0)

// After a group of launches: report launch errors (bad configuration, or an
// earlier asynchronous fault) as OC_ERR_DEVICE.
#define OC_LAUNCH_CHECK()                                                                     \
  do {                                                                                        \
    hipError_t e_ = hipGetLastError();                                                        \
    if (e_ != hipSuccess)                                                                     \
      return oc::fail(OC_ERR_DEVICE, "kernel launch failed: %s", hipGetErrorString(e_));     \
  } while (0)
