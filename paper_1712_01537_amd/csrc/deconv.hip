// Octree deconvolution (Sec. 3.2 "Deconvolution"): the transposed
// convolution.  The paper obtains it by swapping the convolution's forward
// and backward passes, and so does this file: with w the weight
// [K^3][cout][cin] of the convolution cout -> cin that the deconvolution
// transposes,
//   forward       y  = input gradient of that convolution for upstream x,
//   input grad    dx = that convolution's forward applied to dy,
//   weight grad   dw = that convolution's weight gradient with dy as its
//                      input and x as its upstream gradient.
// Every pass therefore runs on the convolution kernels (matrix cores; stride
// 1 group tiles, stride 2^r gathered-row GEMMs), with their fixed-order
// reductions: results are reproducible bit for bit.  Stride 2^r maps depth
// l-r to depth l, the transpose of the stride-2^r convolution at depth l.
//
// bf16 (x and w bf16): the convolution's upstream gradient is an fp32
// argument that its bf16 backward rounds to bf16, so the forward widens x to
// fp32 first (exact; the rounding then changes nothing); the backward rounds
// dy to bf16, the operand precision of the bf16 passes, as the convolution's
// backward does with its upstream gradient.
#include <algorithm>

#include "common.h"

namespace {

constexpr int TB = 256;

__global__ __launch_bounds__(TB) void k_dc_widen(const uint16_t* __restrict__ in, int64_t n,
                                                 float* __restrict__ out) {
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e < n) out[e] = __uint_as_float((uint32_t)in[e] << 16);
}

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__global__ __launch_bounds__(TB) void k_dc_round(const float* __restrict__ in, int64_t n,
                                                 uint16_t* __restrict__ out) {
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e >= n) return;
  const uint32_t u = __float_as_uint(in[e]);
  out[e] = (u & 0x7f800000u) == 0x7f800000u
               ? (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u))
               : (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

inline unsigned grid_for(int64_t n) { return (unsigned)oc::cdiv(n, TB); }

oc_status check_deconv(const oc_octree* t, int32_t l, int32_t stride, oc_dtype dt, int32_t flags,
                       const char* who) {
  oc_status st = oc::check_tree_level(t, l, 1);
  if (st != OC_OK) return st;
  if (stride < 1 || (stride & (stride - 1)) != 0 || stride > (1 << l))
    return oc::fail(OC_ERR_ARG, "%s: stride %d not a power of two up to 2^depth", who, stride);
  if (dt != OC_F32 && dt != OC_BF16) return oc::fail(OC_ERR_ARG, "%s: bad dtype %d", who, (int)dt);
  if (flags != 0) return oc::fail(OC_ERR_ARG, "%s: flags must be 0", who);
  return OC_OK;
}

// Rows of the deconvolution's input (depth l - r) and output (depth l).
void rows_of(const oc_octree* t, int32_t l, int32_t stride, int64_t* n_in, int64_t* n_out) {
  *n_out = t->N[l];
  *n_in = t->N[l - __builtin_ctz((unsigned)stride)];
}

}  // namespace

extern "C" {

size_t oc_deconv_fwd_workspace(const oc_octree* t, int32_t l, int32_t K, int32_t stride,
                               oc_dtype dt, int32_t cin, int32_t cout) {
  if (check_deconv(t, l, stride, dt, 0, "oc_deconv_fwd_workspace") != OC_OK) return 0;
  int64_t n_in, n_out;
  rows_of(t, l, stride, &n_in, &n_out);
  const size_t wide = dt == OC_BF16 ? oc::align256((size_t)n_in * cin * 4) : 0;
  return wide + oc_conv_bwd_workspace(t, l, K, stride, dt, cout, cin);
}

oc_status oc_deconv_fwd(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                        const void* x, int32_t cin, const void* w, int32_t cout, float* y,
                        void* ws, size_t ws_bytes, int32_t flags, hipStream_t s) {
  oc_status st = check_deconv(t, l, stride, dt, flags, "oc_deconv_fwd");
  if (st != OC_OK) return st;
  if (!x || !w || !y) return oc::fail(OC_ERR_ARG, "oc_deconv_fwd: NULL buffer");
  st = oc::conv_check(t, l, K, stride, dt, cout, cin, "oc_deconv_fwd");
  if (st != OC_OK) return st;
  const size_t need = oc_deconv_fwd_workspace(t, l, K, stride, dt, cin, cout);
  if (need && (!ws || ws_bytes < need))
    return oc::fail(OC_ERR_ARG, "oc_deconv_fwd: workspace %zu bytes < %zu", ws ? ws_bytes : 0,
                    need);
  const float* xf = static_cast<const float*>(x);
  char* rest = (char*)ws;
  size_t rest_bytes = ws_bytes;
  if (dt == OC_BF16) {
    int64_t n_in, n_out;
    rows_of(t, l, stride, &n_in, &n_out);
    const int64_t n = n_in * cin;
    float* xw = (float*)rest;
    if (n > 0) oc::launch(k_dc_widen, dim3(grid_for(n)), dim3(TB), 0, s, (const uint16_t*)x, n, xw);
    xf = xw;
    const size_t used = oc::align256((size_t)n * 4);
    rest += used;
    rest_bytes -= used;
  }
  return oc_conv_bwd(t, l, K, stride, dt, nullptr, cout, w, cin, nullptr, xf, y, nullptr, rest,
                     rest_bytes, 0, s);
}

size_t oc_deconv_bwd_workspace(const oc_octree* t, int32_t l, int32_t K, int32_t stride,
                               oc_dtype dt, int32_t cin, int32_t cout) {
  if (check_deconv(t, l, stride, dt, 0, "oc_deconv_bwd_workspace") != OC_OK) return 0;
  int64_t n_in, n_out;
  rows_of(t, l, stride, &n_in, &n_out);
  const size_t wide = dt == OC_BF16 ? oc::align256((size_t)n_out * cout * 2) +
                                          oc::align256((size_t)n_in * cin * 4)
                                    : 0;
  return wide + std::max(oc_conv_fwd_workspace(t, l, K, stride, dt, cout, cin),
                         oc_conv_bwd_workspace(t, l, K, stride, dt, cout, cin));
}

oc_status oc_deconv_bwd(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                        const void* x, int32_t cin, const void* w, int32_t cout, const float* dy,
                        float* dx, float* dw, void* ws, size_t ws_bytes, int32_t flags,
                        hipStream_t s) {
  oc_status st = check_deconv(t, l, stride, dt, flags, "oc_deconv_bwd");
  if (st != OC_OK) return st;
  if (!w || !dy) return oc::fail(OC_ERR_ARG, "oc_deconv_bwd: NULL w or dy");
  if (dw && !x) return oc::fail(OC_ERR_ARG, "oc_deconv_bwd: dw needs x");
  if (!dx && !dw) return OC_OK;
  // every argument check of both passes before anything is enqueued
  st = oc::conv_check(t, l, K, stride, dt, cout, cin, "oc_deconv_bwd");
  if (st != OC_OK) return st;
  const size_t need = oc_deconv_bwd_workspace(t, l, K, stride, dt, cin, cout);
  if (need && (!ws || ws_bytes < need))
    return oc::fail(OC_ERR_ARG, "oc_deconv_bwd: workspace %zu bytes < %zu", ws ? ws_bytes : 0,
                    need);
  const void* dyc = dy;  // the convolution's input: dy (bf16: rounded)
  const float* xf = static_cast<const float*>(x);  // its upstream gradient: x (bf16: widened)
  char* rest = (char*)ws;
  size_t rest_bytes = ws_bytes;
  if (dt == OC_BF16) {
    int64_t n_in, n_out;
    rows_of(t, l, stride, &n_in, &n_out);
    uint16_t* d16 = (uint16_t*)rest;
    const int64_t nd = n_out * cout, nx = n_in * cin;
    if (nd > 0) oc::launch(k_dc_round, dim3(grid_for(nd)), dim3(TB), 0, s, dy, nd, d16);
    dyc = d16;
    size_t used = oc::align256((size_t)nd * 2);
    float* xw = (float*)(rest + used);
    if (dw && nx > 0)
      oc::launch(k_dc_widen, dim3(grid_for(nx)), dim3(TB), 0, s, (const uint16_t*)x, nx, xw);
    xf = xw;
    used += oc::align256((size_t)nx * 4);
    rest += used;
    rest_bytes -= used;
  }
  if (dx) {
    st = oc_conv_fwd(t, l, K, stride, dt, dyc, cout, w, cin, dx, rest, rest_bytes, 0, s);
    if (st != OC_OK) return st;
  }
  if (dw)
    st = oc_conv_bwd(t, l, K, stride, dt, dyc, cout, w, cin, nullptr, xf, nullptr, dw, rest,
                     rest_bytes, 0, s);
  return st;
}

}  // extern "C"
