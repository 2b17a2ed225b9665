// Strided octree convolution (stride 2^r, r >= 1, K = 3) on the matrix cores
// (conv_sr.hip): implicit GEMMs over gathered rows, no column buffer.
#pragma once

#include "common.h"

namespace oc {

// Workspace bytes of the forward, and of the backward for the requested
// gradients, at input depth l and stride 2^r (0 when nothing is needed).
size_t conv_s2_fwd_ws(const oc_octree* t, int l, int r, int cin, int cout, bool bf16);
size_t conv_s2_bwd_ws(const oc_octree* t, int l, int r, int cin, int cout, bool bf16, bool dx,
                      bool dw);

// y [N_{l-r}][cout] from x [N_l][cin] and w [27][cin][cout] (bf16: x and w
// bf16); relu applies max(0, .).
oc_status conv_s2_fwd(const oc_octree* t, int l, int r, const void* x, int cin, const void* w,
                      int cout, bool bf16, float* y, int relu, void* ws, hipStream_t s);

// dx [N_l][cin] and/or dw [27][cin][cout] (either may be null) for upstream
// gradient dy [N_{l-r}][cout]; ym: the forward output when the forward fused
// a ReLU (dy is masked by [ym > 0]), else null.
oc_status conv_s2_bwd(const oc_octree* t, int l, int r, const void* x, int cin, const void* w,
                      int cout, bool bf16, const float* ym, const float* dy, float* dx, float* dw,
                      void* ws, hipStream_t s);

// Name (template arguments included) of the kernel doing pass 0 (forward),
// 1 (input gradient) or 2 (weight gradient); thread-local storage.
const char* conv_sr_kernel_name(int pass, int r, bool bf16, int cin, int cout);

}  // namespace oc
