// Launchers of the first-layer convolution kernels (conv_cin.hip): K = 3 with
// 3 or 4 input channels (the input signal), fp32.
#pragma once

#include "common.h"

namespace oc {

// True when conv_cin_fwd / conv_cin_dw take this shape (K = 3, cin 3 or 4,
// cout a positive multiple of 16).
bool conv_cin_supported(int K, int cin, int cout);

// y [N_l][cout] = conv(x [N_l][cin], w [27][cin][cout]), stride 1; relu != 0
// applies max(0, .).
void conv_cin_fwd(const oc_octree* t, int l, const float* x, int cin, const float* w, int cout,
                  float* y, int relu, hipStream_t s);

// The same with ReLU (relu != 0) and the 2x2x2 max-pool in the epilogue:
// yp [N_{l-1}][cout] (rows of empty octants zero), sw [M_{l-1}][cout] as
// the pooling's switches; yp 16-byte and sw 4-byte aligned.
void conv_cin_pool_fwd(const oc_octree* t, int l, const float* x, int cin, const float* w,
                       int cout, float* yp, uint8_t* sw, int relu, hipStream_t s);

// Number of [27][cin][cout] fp32 partial sums conv_cin_dw needs.
size_t conv_cin_dw_parts(const oc_octree* t, int l, int cin, int cout);

// dw [27][cin][cout] = weight gradient for upstream gradient dy [N_l][cout];
// part holds conv_cin_dw_parts() partial sums.  defer: leave the partial
// sums in part (dw not written).
void conv_cin_dw(const oc_octree* t, int l, const float* x, int cin, const float* dy, int cout,
                 float* dw, float* part, hipStream_t s, bool defer = false);

// Name of the kernel of pass 0 (forward), 2 (weight gradient) or 3 (the
// pooled forward).
void conv_cin_kernel_name(int cin, int pass, char* buf, size_t n);

// Fixed-order sum of np partials of n fp32 entries (conv_mfma.hip).
void sum_partials(const float* part, int np, int64_t n, float* out, hipStream_t s);

}  // namespace oc
