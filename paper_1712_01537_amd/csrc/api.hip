// Error reporting, allocation and octree accessors of the C ABI.
#include <cstring>

#include <atomic>

#include "common.h"

namespace {
thread_local char g_msg[512] = "";
thread_local hipEvent_t g_prof_start = nullptr, g_prof_stop = nullptr;
// oc_profile_calls: armed event arrays, their capacity and the count used
thread_local hipEvent_t* g_call_start = nullptr;
thread_local hipEvent_t* g_call_stop = nullptr;
thread_local int32_t g_call_cap = 0;
thread_local int32_t* g_call_used = nullptr;
}

namespace oc {

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
}

oc_status fail(oc_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_msg, sizeof(g_msg), fmt, ap);
  va_end(ap);
  return s;
}

void* dev_alloc(const oc_allocator& a, size_t bytes, hipStream_t s) {
  if (bytes == 0) bytes = 256;
  if (a.alloc) return a.alloc(a.ctx, bytes, s);
  void* p = nullptr;
  if (hipMalloc(&p, bytes) != hipSuccess) return nullptr;
  return p;
}

void dev_free(const oc_allocator& a, void* p, hipStream_t s) {
  if (!p) return;
  if (a.free) {
    a.free(a.ctx, p, s);
    return;
  }
  // hipFree waits for the device, so pending work on the buffer completes.
  (void)hipFree(p);
}

int cu_count() {
  static std::atomic<int> cached[64];
  int d = 0;
  if (hipGetDevice(&d) != hipSuccess || d < 0) d = 0;
  std::atomic<int>* slot = d < 64 ? &cached[d] : nullptr;
  int n = slot ? slot->load(std::memory_order_relaxed) : 0;
  if (n > 0) return n;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, d) != hipSuccess || n < 1)
    n = 1;
  if (slot) slot->store(n, std::memory_order_relaxed);
  return n;
}

void take_profile_events(hipEvent_t* start, hipEvent_t* stop) {
  *start = g_prof_start;
  *stop = g_prof_stop;
  g_prof_start = g_prof_stop = nullptr;
}

void take_call_events(hipEvent_t* start, hipEvent_t* stop) {
  *start = *stop = nullptr;
  if (!g_call_used || *g_call_used >= g_call_cap) return;
  const int32_t i = (*g_call_used)++;
  *start = g_call_start[i];
  *stop = g_call_stop[i];
}

oc_status check_tree_level(const oc_octree* t, int32_t l, int32_t min_l) {
  if (!t) return fail(OC_ERR_ARG, "octree is NULL");
  if (l < min_l || l > t->depth)
    return fail(OC_ERR_ARG, "depth %d not in %d..%d", l, min_l, t->depth);
  return OC_OK;
}

}  // namespace oc

extern "C" {

oc_status oc_octree_level(const oc_octree* t, int32_t l, oc_level* out) {
  oc_status st = oc::check_tree_level(t, l, 0);
  if (st != OC_OK) return st;
  if (!out) return oc::fail(OC_ERR_ARG, "oc_octree_level: out is NULL");
  out->depth = l;
  out->num_octants = t->N[l];
  out->num_nonempty = t->M[l];
  out->keys = t->keys[l];
  out->labels = t->labels[l];
  out->rows_of_label = t->rows[l];
  out->nbr = t->nbr[l];
  return OC_OK;
}

oc_status oc_octree_info(const oc_octree* t, int32_t* depth, int32_t* full_depth, int32_t* batch) {
  if (!t) return oc::fail(OC_ERR_ARG, "octree is NULL");
  if (depth) *depth = t->depth;
  if (full_depth) *full_depth = t->full_depth;
  if (batch) *batch = t->batch;
  return OC_OK;
}

const float* oc_octree_signal(const oc_octree* t) { return t ? t->signal : nullptr; }

void oc_octree_free(oc_octree* t) {
  if (!t) return;
  oc::dev_free(t->alloc, t->block, t->stream);
  delete t;
}

oc_status oc_profile_calls(hipEvent_t* starts, hipEvent_t* stops, int32_t cap, int32_t* used) {
  if (!starts && !stops && !used) {
    g_call_start = g_call_stop = nullptr;
    g_call_used = nullptr;
    g_call_cap = 0;
    return OC_OK;
  }
  if (!starts || !stops || !used || cap < 0)
    return oc::fail(OC_ERR_ARG, "oc_profile_calls: give both arrays and the count, or none");
  g_call_start = starts;
  g_call_stop = stops;
  g_call_cap = cap;
  g_call_used = used;
  *used = 0;
  return OC_OK;
}

const char* oc_status_str(oc_status s) {
  switch (s) {
    case OC_OK: return "ok";
    case OC_ERR_ARG: return "invalid argument";
    case OC_ERR_RANGE: return "point outside the unit cube";
    case OC_ERR_NOMEM: return "out of device memory";
    case OC_ERR_DEVICE: return "device error";
    case OC_ERR_UNSUPPORTED: return "unsupported";
  }
  return "unknown status";
}

const char* oc_last_error(void) { return g_msg; }

oc_status oc_profile_next(hipEvent_t start, hipEvent_t stop) {
  if ((start == nullptr) != (stop == nullptr))
    return oc::fail(OC_ERR_ARG, "oc_profile_next: give both events or neither");
  g_prof_start = start;
  g_prof_stop = stop;
  return OC_OK;
}

}  // extern "C"
