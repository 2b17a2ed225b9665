// 2x2x2 max-pooling in the epilogue of the stride-1 convolution kernels
// (conv + ReLU + pooling in one pass: the depth-l output is never written).
// Their 16x16 MFMA accumulators hold, in lane l, four output channels
// 4(l/16) .. 4(l/16)+3 of octant row l%16 of a 16-row block; a block is two
// sibling groups (rows 0-7 and 8-15) and 16 output channels, so it pools to
// 2 x 16 outputs.  The block goes through a small LDS area of the wave (one
// 16-byte write per lane); then lane o (o = lane % 32) scans the eight
// children of group o/16 in channel o%16, in child order with a strict '>'
// (the first maximum wins, Sec. 3.2 "Pooling").  A scan costs 8 LDS reads
// and three VALU operations per child, far fewer than exchanging the eight
// children's values and indices between lanes.
#pragma once

#include "common.h"

namespace oc {

typedef float pf_v4f __attribute__((ext_vector_type(4)));

// Floats of the LDS area; row r, channel c sits at r * 16 + c, rows 8-15
// shifted by 16 floats so that the two groups' reads fall on distinct banks.
constexpr int kPoolLdsFloats = 16 * 16 + 16;

__device__ __forceinline__ int pool_lds_index(int r, int c) { return r * 16 + c + ((r >> 3) << 4); }

// Lane (i, q) = (lane % 16, lane / 16) stores its accumulator values (row i,
// channels 4q .. 4q+3).  lds: 16-byte aligned, kPoolLdsFloats floats.
__device__ __forceinline__ void pool_put(float* lds, const pf_v4f& v, int lane) {
  *reinterpret_cast<pf_v4f*>(lds + pool_lds_index(lane & 15, 4 * (lane >> 4))) = v;
}

// Lane o = lane % 32: maximum over the children of group o/16 in channel
// o%16 and the first child holding it (after pool_put by the whole wave).
__device__ __forceinline__ float pool_scan(const float* lds, int lane, uint32_t& child) {
  const int g = (lane >> 4) & 1, c = lane & 15;
  const float* p = lds + pool_lds_index(8 * g, c);
  float v[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) v[k] = p[16 * k];
  float m = v[0];
  uint32_t a = 0;
#pragma unroll
  for (int k = 1; k < 8; ++k) {
    const bool gt = v[k] > m;
    m = gt ? v[k] : m;
    a = gt ? (uint32_t)k : a;
  }
  child = a;
  return m;
}

}  // namespace oc
