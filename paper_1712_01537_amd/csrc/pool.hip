// 2x2x2 max-pooling and max-unpooling across depths through the label
// buffer (Sec. 3.2 "Pooling" and "Unpooling", Fig. 5 of O-CNN).
//
// The eight children of the non-empty octant with label p occupy rows
// 8(p-1)..8(p-1)+7 of the finer depth, so pooling is a max over 8 contiguous
// rows; the paper's temporary packed array is fused away: the kernel writes
// the row of the parent directly (found through the label of that row), and
// empty parents get zeros.  One thread handles VEC consecutive channels of one
// row; a wavefront therefore streams whole rows (coalesced), and the eight
// child rows it reads are one contiguous 8*C*4-byte span.
#include "common.h"

namespace {

constexpr int TB = 256;

template <int VEC>
struct Vec;
template <>
struct Vec<1> {
  using f = float;
  using u8 = uint8_t;
};
template <>
struct Vec<4> {
  using f = float4;
  using u8 = uchar4;
};

__device__ __forceinline__ float comp(const float& v, int) { return v; }
__device__ __forceinline__ float comp(const float4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}
__device__ __forceinline__ void set(float& v, int, float a) { v = a; }
__device__ __forceinline__ void set(float4& v, int i, float a) {
  if (i == 0) v.x = a;
  else if (i == 1) v.y = a;
  else if (i == 2) v.z = a;
  else v.w = a;
}
__device__ __forceinline__ uint8_t comp(const uint8_t& v, int) { return v; }
__device__ __forceinline__ uint8_t comp(const uchar4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}
__device__ __forceinline__ void set(uint8_t& v, int, uint8_t a) { v = a; }
__device__ __forceinline__ void set(uchar4& v, int i, uint8_t a) {
  if (i == 0) v.x = a;
  else if (i == 1) v.y = a;
  else if (i == 2) v.z = a;
  else v.w = a;
}

// y[i] (depth l-1) = max over the children of row i, sw = first argmax.
template <int VEC>
__global__ __launch_bounds__(TB) void k_pool_fwd(const float* __restrict__ x,
                                                 const int32_t* __restrict__ labels, int64_t n_out,
                                                 int cv, float* __restrict__ y,
                                                 uint8_t* __restrict__ sw) {
  using F = typename Vec<VEC>::f;
  using U = typename Vec<VEC>::u8;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_out * cv) return;
  const int64_t i = t / cv;
  const int cc = (int)(t - i * cv);
  const int32_t L = labels[i];
  F out;
  if (L == 0) {
    for (int e = 0; e < VEC; ++e) set(out, e, 0.0f);
    reinterpret_cast<F*>(y)[t] = out;
    return;
  }
  const int64_t g = L - 1;
  const F* src = reinterpret_cast<const F*>(x) + (8 * g) * cv + cc;
  F best = src[0];
  U arg;
  for (int e = 0; e < VEC; ++e) set(arg, e, (uint8_t)0);
#pragma unroll
  for (int k = 1; k < 8; ++k) {
    const F v = src[(int64_t)k * cv];
#pragma unroll
    for (int e = 0; e < VEC; ++e)
      if (comp(v, e) > comp(best, e)) {  // strict: the first maximum wins ties
        set(best, e, comp(v, e));
        set(arg, e, (uint8_t)k);
      }
  }
  reinterpret_cast<F*>(y)[t] = best;
  reinterpret_cast<U*>(sw)[g * cv + cc] = arg;
}

// Routing through the switches (pool backward == unpool forward):
// out[8g + k][c] = (sw[g][c] == k) ? in[rows[g]][c] : 0 for every child row.
// With ymask, the routed value is also zeroed where ymask[rows[g]][c] <= 0.
template <int VEC>
__global__ __launch_bounds__(TB) void k_route_down(const float* __restrict__ in,
                                                   const float* __restrict__ ymask,
                                                   const uint8_t* __restrict__ sw,
                                                   const int32_t* __restrict__ rows, int64_t n_l,
                                                   int cv, float* __restrict__ out) {
  using F = typename Vec<VEC>::f;
  using U = typename Vec<VEC>::u8;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_l * cv) return;
  const int64_t row = t / cv;
  const int cc = (int)(t - row * cv);
  const int64_t g = row >> 3;
  const uint8_t k = (uint8_t)(row & 7);
  const U s = reinterpret_cast<const U*>(sw)[g * cv + cc];
  const int64_t src = (int64_t)rows[g] * cv + cc;
  const F v = reinterpret_cast<const F*>(in)[src];
  F m;
  if (ymask) m = reinterpret_cast<const F*>(ymask)[src];
  F o;
#pragma unroll
  for (int e = 0; e < VEC; ++e)
    set(o, e, comp(s, e) == k && (!ymask || comp(m, e) > 0.0f) ? comp(v, e) : 0.0f);
  reinterpret_cast<F*>(out)[t] = o;
}

// Unpool backward: dx[i][c] = dy[8g + sw[g][c]][c] for label L = g+1 > 0.
template <int VEC>
__global__ __launch_bounds__(TB) void k_route_up(const float* __restrict__ dy,
                                                 const uint8_t* __restrict__ sw,
                                                 const int32_t* __restrict__ labels,
                                                 int64_t n_out, int cv, float* __restrict__ dx) {
  using F = typename Vec<VEC>::f;
  using U = typename Vec<VEC>::u8;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_out * cv) return;
  const int64_t i = t / cv;
  const int cc = (int)(t - i * cv);
  const int32_t L = labels[i];
  F o;
  if (L == 0) {
    for (int e = 0; e < VEC; ++e) set(o, e, 0.0f);
  } else {
    const int64_t g = L - 1;
    const U s = reinterpret_cast<const U*>(sw)[g * cv + cc];
    const float* base = dy + (8 * g) * (int64_t)(cv * VEC) + (int64_t)cc * VEC;
#pragma unroll
    for (int e = 0; e < VEC; ++e) set(o, e, base[(int64_t)comp(s, e) * cv * VEC + e]);
  }
  reinterpret_cast<F*>(dx)[t] = o;
}

inline unsigned grid_for(int64_t n) { return (unsigned)oc::cdiv(n, TB); }

oc_status check_common(const oc_octree* t, int32_t l, int32_t c, const void* a, const void* b,
                       const void* s, const char* who) {
  oc_status st = oc::check_tree_level(t, l, 1);
  if (st != OC_OK) return st;
  if (c < 1 || c > 65536) return oc::fail(OC_ERR_ARG, "%s: channels %d out of range", who, c);
  if (!a || !b || !s) return oc::fail(OC_ERR_ARG, "%s: NULL buffer", who);
  return OC_OK;
}

bool vec4_ok(int c, const void* a, const void* b, const void* s) {
  return c % 4 == 0 && ((uintptr_t)a % 16 == 0) && ((uintptr_t)b % 16 == 0) &&
         ((uintptr_t)s % 4 == 0);
}

}  // namespace

extern "C" {

oc_status oc_pool_fwd(const oc_octree* t, int32_t l, const float* x, int32_t c, float* y,
                      uint8_t* sw, hipStream_t s) {
  oc_status st = check_common(t, l, c, x, y, sw, "oc_pool_fwd");
  if (st != OC_OK) return st;
  const int64_t n = t->N[l - 1];
  if (n == 0) return OC_OK;
  if (vec4_ok(c, x, y, sw)) {
    const int cv = c / 4;
    oc::launch_main(k_pool_fwd<4>, dim3(grid_for(n * cv)), dim3(TB), s, x,
                       (const int32_t*)t->labels[l - 1], n, cv, y, sw);
  } else {
    oc::launch_main(k_pool_fwd<1>, dim3(grid_for(n * c)), dim3(TB), s, x,
                       (const int32_t*)t->labels[l - 1], n, c, y, sw);
  }
  OC_LAUNCH_CHECK();
  return OC_OK;
}

static oc_status route_down(const oc_octree* t, int32_t l, const float* in, const float* ymask,
                            const uint8_t* sw, int32_t c, float* out, hipStream_t s,
                            const char* who) {
  oc_status st = check_common(t, l, c, in, out, sw, who);
  if (st != OC_OK) return st;
  const int64_t n = t->N[l];
  if (n == 0) return OC_OK;
  if (vec4_ok(c, in, out, sw) && (uintptr_t)ymask % 16 == 0) {
    const int cv = c / 4;
    oc::launch_main(k_route_down<4>, dim3(grid_for(n * cv)), dim3(TB), s, in, ymask, sw,
                       (const int32_t*)t->rows[l - 1], n, cv, out);
  } else {
    oc::launch_main(k_route_down<1>, dim3(grid_for(n * c)), dim3(TB), s, in, ymask, sw,
                       (const int32_t*)t->rows[l - 1], n, c, out);
  }
  OC_LAUNCH_CHECK();
  return OC_OK;
}

oc_status oc_pool_bwd(const oc_octree* t, int32_t l, const float* dy, const uint8_t* sw, int32_t c,
                      const float* y, float* dx, hipStream_t s) {
  return route_down(t, l, dy, y, sw, c, dx, s, "oc_pool_bwd");
}

oc_status oc_unpool_fwd(const oc_octree* t, int32_t l, const float* x, const uint8_t* sw,
                        int32_t c, float* y, hipStream_t s) {
  return route_down(t, l, x, nullptr, sw, c, y, s, "oc_unpool_fwd");
}

oc_status oc_unpool_bwd(const oc_octree* t, int32_t l, const float* dy, const uint8_t* sw,
                        int32_t c, float* dx, hipStream_t s) {
  oc_status st = check_common(t, l, c, dy, dx, sw, "oc_unpool_bwd");
  if (st != OC_OK) return st;
  const int64_t n = t->N[l - 1];
  if (n == 0) return OC_OK;
  if (vec4_ok(c, dy, dx, sw)) {
    const int cv = c / 4;
    oc::launch_main(k_route_up<4>, dim3(grid_for(n * cv)), dim3(TB), s, dy, sw,
                       (const int32_t*)t->labels[l - 1], n, cv, dx);
  } else {
    oc::launch_main(k_route_up<1>, dim3(grid_for(n * c)), dim3(TB), s, dy, sw,
                       (const int32_t*)t->labels[l - 1], n, c, dx);
  }
  OC_LAUNCH_CHECK();
  return OC_OK;
}

}  // extern "C"
