// Launchers of the bf16 matrix-core convolution kernels (conv_bf16.hip).
#pragma once

#include "common.h"

namespace oc {

// True when the bf16 kernels take a stride-1 convolution with these channel
// counts (both multiples of 16); other shapes run the fp32 kernels on widened
// operands.
bool conv_bf16_supported(int K, int cin, int cout);

// Name of the main kernel of pass 0 (forward), 1 (input gradient) or 2
// (weight gradient); for more than 64 reduction channels the first of the
// launches, one per 64 channels.  rows: the octants of the layer's depth
// (the 16-group forward tiles need its input to span less than 2 GiB).
void conv_bf16_kernel_name(int K, int cin, int cout, int pass, int64_t rows, char* buf,
                           size_t n);

// Workspace bytes of a forward call: the weights in MFMA order.
size_t conv_bf16_fwd_ws(int K, int cin, int cout);

// Workspace bytes of a backward call (input gradient and/or weight gradient):
// dy rounded to bf16, the flipped weights, the weight gradient's partial sums.
size_t conv_bf16_bwd_ws(const oc_octree* t, int l, int K, int cin, int cout);

// y [N_l][cout] fp32 = conv(x [N_l][cin] bf16, w [K^3][cin][cout] bf16),
// stride 1; relu != 0 applies max(0, .).  ws: conv_bf16_fwd_ws bytes.
void conv_bf16_fwd(const oc_octree* t, int l, int K, const uint16_t* x, int cin,
                   const uint16_t* w, int cout, float* y, int relu, void* ws, hipStream_t s);

// Backward of conv_bf16_fwd for the upstream gradient dy [N_l][cout] fp32,
// masked with [y > 0] when ym is not NULL, then rounded to bf16 (the MFMA
// operand).  dx [N_l][cin] and/or dw [K^3][cin][cout] (fp32, NULL to skip).
// ws: conv_bf16_bwd_ws bytes.
void conv_bf16_bwd(const oc_octree* t, int l, int K, const uint16_t* x, int cin,
                   const uint16_t* w, int cout, const float* ym, const float* dy, float* dx,
                   float* dw, void* ws, hipStream_t s);

// y[e] = bf16(x[e]) for e < n, round to nearest even (NaN stays NaN).
void round_bf16(const float* x, int64_t n, uint16_t* y, hipStream_t s);

}  // namespace oc
