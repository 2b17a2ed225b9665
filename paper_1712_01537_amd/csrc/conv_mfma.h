// Launchers of the fp32 matrix-core convolution kernels (conv_mfma.hip).
#pragma once

#include "common.h"

namespace oc {

// Name (with template arguments) of the main kernel of pass 0 (forward),
// 1 (input gradient), 2 (weight gradient) or 3 (conv + pool forward) of a
// stride-1 convolution.
void conv_s1_kernel_name(const oc_octree* t, int l, int K, int cin, int cout, int pass, char* buf,
                         size_t n);

// Bytes of split-reduction workspace the stride-1 group-tile kernel needs for
// kk reduction channels and nn output channels at depth l (0: none).
size_t conv_s1_tile_ws(const oc_octree* t, int l, int K, int kk, int nn);

// y [N_l][cout] = conv(x [N_l][cin], w [K^3][cin][cout]), stride 1; relu != 0
// applies max(0, .) to the output.  ws: conv_s1_tile_ws(t, l, K, cin, cout)
// bytes.
void conv_s1_fwd_f32(const oc_octree* t, int l, int K, const float* x, int cin, const float* w,
                     int cout, float* y, int relu, float* ws, hipStream_t s);

// True when the forward kernel of this stride-1 fp32 shape pools in its
// epilogue (or through its split sum): conv_s1_pool_fwd_f32 then needs
// conv_s1_tile_ws(t, l, K, cin, cout) bytes of workspace and writes no
// depth-l output.
bool conv_s1_pool_fused(const oc_octree* t, int l, int K, int cin, int cout);

// yp [N_{l-1}][cout], sw [M_{l-1}][cout] = 2x2x2 max-pool (first maximum
// over children 0..7) of the stride-1 convolution of x, ReLU'd when relu;
// rows of empty octants zero.  Only for shapes conv_s1_pool_fused takes; yp
// 16-byte and sw 4-byte aligned.
void conv_s1_pool_fwd_f32(const oc_octree* t, int l, int K, const float* x, int cin,
                          const float* w, int cout, float* yp, uint8_t* sw, int relu, float* ws,
                          hipStream_t s);

// dx [N_l][cin] = input gradient of a stride-1 convolution for upstream
// gradient dy [N_l][cout].  ws: conv_s1_tile_ws(t, l, K, cout, cin) bytes.
void conv_s1_bwd_data_f32(const oc_octree* t, int l, int K, const float* dy, int cout,
                          const float* w, int cin, float* dx, float* ws, hipStream_t s);

// The same input gradient routed through the 2x2x2 max-pool from depth l+1
// that produced x: dxf [N_{l+1}][cin] = the pool backward of it (switches sw
// [M_l][cin], the gradient kept where the pooled value mask [N_l][cin] is
// > 0; mask NULL: everywhere).  cin % 4 == 0, dxf 16-byte and sw 4-byte
// aligned.  dx [N_l][cin] is scratch (written only when the reduction is not
// split), ws as conv_s1_bwd_data_f32.  Equal, bit for bit, to
// conv_s1_bwd_data_f32 followed by the pool backward.
void conv_s1_bwd_data_pool_f32(const oc_octree* t, int l, int K, const float* dy, int cout,
                               const float* w, int cin, float* dx, const float* mask,
                               const uint8_t* sw, float* dxf, float* ws, hipStream_t s);

// Number of [K^3][cin][cout] fp32 partial sums conv_s1_bwd_weight_f32 needs.
size_t conv_s1_dw_parts(const oc_octree* t, int l, int K, int cin, int cout);

// dw [K^3][cin][cout] = weight gradient of a stride-1 convolution; part holds
// conv_s1_dw_parts() partial sums.  defer: leave the partial sums in part
// (dw not written), for a later sum_partials_multi.
void conv_s1_bwd_weight_f32(const oc_octree* t, int l, int K, const float* x, int cin,
                            const float* dy, int cout, float* dw, float* part, hipStream_t s,
                            bool defer = false);

// outs[i] = fixed-order sum of nparts[i] partials of counts[i] fp32 entries at
// parts[i], for i < n, in as few launches as possible (one per eight sets
// with 16-byte aligned buffers and counts a multiple of 4; other sets alone);
// the same bits as sum_partials of each set.
void sum_partials_multi(int n, const float* const* parts, const int* nparts,
                        const int64_t* counts, float* const* outs, hipStream_t s);

}  // namespace oc
