// Octree deconvolution (Sec. 3.2 "Deconvolution"): the transposed
// convolution.  The paper obtains it by swapping the convolution's forward
// and backward passes, and so does this file: with w the weight
// [K^3][cout][cin] of the convolution cout -> cin that the deconvolution
// transposes,
//   forward       y  = input gradient of that convolution for upstream x,
//   input grad    dx = that convolution's forward applied to dy,
//   weight grad   dw = that convolution's weight gradient with dy as its
//                      input and x as its upstream gradient.
// Every pass therefore runs on the convolution kernels (matrix cores for
// stride 1, column buffers and GEMMs for stride 2), with their fixed-order
// reductions: results are reproducible bit for bit.  Stride 2 maps depth l-1
// to depth l, the transpose of the stride-2 convolution at depth l.
#include <algorithm>

#include "common.h"

namespace {

oc_status check_deconv(const oc_octree* t, int32_t l, int32_t stride, oc_dtype dt, int32_t flags,
                       const char* who) {
  oc_status st = oc::check_tree_level(t, l, 1);
  if (st != OC_OK) return st;
  if (stride != 1 && stride != 2)
    return oc::fail(OC_ERR_UNSUPPORTED, "%s: stride %d not 1 or 2", who, stride);
  if (dt != OC_F32) return oc::fail(OC_ERR_UNSUPPORTED, "%s: only OC_F32 is supported", who);
  if (flags != 0) return oc::fail(OC_ERR_ARG, "%s: flags must be 0", who);
  return OC_OK;
}

}  // namespace

extern "C" {

size_t oc_deconv_fwd_workspace(const oc_octree* t, int32_t l, int32_t K, int32_t stride,
                               oc_dtype dt, int32_t cin, int32_t cout) {
  if (check_deconv(t, l, stride, dt, 0, "oc_deconv_fwd_workspace") != OC_OK) return 0;
  return oc_conv_bwd_workspace(t, l, K, stride, dt, cout, cin);
}

oc_status oc_deconv_fwd(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                        const void* x, int32_t cin, const void* w, int32_t cout, float* y,
                        void* ws, size_t ws_bytes, int32_t flags, hipStream_t s) {
  oc_status st = check_deconv(t, l, stride, dt, flags, "oc_deconv_fwd");
  if (st != OC_OK) return st;
  if (!x || !w || !y) return oc::fail(OC_ERR_ARG, "oc_deconv_fwd: NULL buffer");
  return oc_conv_bwd(t, l, K, stride, dt, nullptr, cout, w, cin, nullptr,
                     static_cast<const float*>(x), y, nullptr, ws, ws_bytes, 0, s);
}

size_t oc_deconv_bwd_workspace(const oc_octree* t, int32_t l, int32_t K, int32_t stride,
                               oc_dtype dt, int32_t cin, int32_t cout) {
  if (check_deconv(t, l, stride, dt, 0, "oc_deconv_bwd_workspace") != OC_OK) return 0;
  return std::max(oc_conv_fwd_workspace(t, l, K, stride, dt, cout, cin),
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
    return oc::fail(OC_ERR_ARG, "oc_deconv_bwd: workspace %zu bytes < %zu", ws ? ws_bytes : 0, need);
  if (dx) {
    st = oc_conv_fwd(t, l, K, stride, dt, dy, cout, w, cin, dx, ws, ws_bytes, 0, s);
    if (st != OC_OK) return st;
  }
  if (dw)
    st = oc_conv_bwd(t, l, K, stride, dt, dy, cout, w, cin, nullptr, static_cast<const float*>(x),
                     nullptr, dw, ws, ws_bytes, 0, s);
  return st;
}

}  // extern "C"
