// Strided octree convolution (stride 2^r, r >= 1, K = 3) on the matrix cores
// (conv_sr.hip): implicit GEMMs over gathered rows, no column buffer.
#pragma once

#include "common.h"

namespace oc {

// Labels of the depths l-r+1 .. l-1 (lab[j] = depth l-r+1+j), the depths a
// stride-2^r neighbourhood descends through.
struct SrLabels {
  const int32_t* lab[OC_MAX_DEPTH];
};

// First-child row (depth l) of the depth-(l-1) octant Q_o = 2^(r-1) P + a
// (P: the coordinates of output p, a non-empty depth-(l-r) octant; a in
// {-1, 0}^3, o = 4 [ax = 0] + 2 [ay = 0] + [az = 0]), or -1 when Q_o is not
// in the octree or empty.  nbr: the group table of depth l-r+1 (the group of
// p's children).  The 27 taps of the stride-2^r neighbourhood read children
// of these eight octants (tap k: o = sr_tap_o(k), child sr_tap_c(k)).
__device__ __forceinline__ int32_t sr_first_child(const int32_t* __restrict__ nbr,
                                                  const SrLabels& L, int64_t p, int o, int r) {
  const int ax = (o >> 2) & 1, ay = (o >> 1) & 1, az = o & 1;  // 1: offset 0, 0: offset -1
  int32_t f = nbr[27 * p + ax * 9 + ay * 3 + az];  // first child (depth l-r+1) of p's neighbour
  const int32_t cb = 4 * (1 - ax) + 2 * (1 - ay) + (1 - az);  // child 1 where a = -1
  for (int j = 0; j < r - 1 && f >= 0; ++j) {
    const int32_t lb = L.lab[j][f + cb];
    f = lb > 0 ? 8 * (lb - 1) : -1;
  }
  return f;
}
__host__ __device__ constexpr int sr_tap_o(int k) {
  return 4 * (k / 9 >= 1) + 2 * ((k / 3) % 3 >= 1) + (k % 3 >= 1);
}
__host__ __device__ constexpr int sr_tap_c(int k) {
  return 4 * (k / 9 != 1) + 2 * ((k / 3) % 3 != 1) + (k % 3 != 1);
}
inline SrLabels sr_labels(const oc_octree* t, int l, int r) {
  SrLabels L{};
  for (int j = 0; j < r - 1; ++j) L.lab[j] = t->labels[l - r + 1 + j];
  return L;
}

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
