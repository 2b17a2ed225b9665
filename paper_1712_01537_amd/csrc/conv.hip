// Octree convolution forward and backward (Sec. 3.2 of O-CNN).
//
// Neighbour addressing.  The children of sibling group g are rows 8g..8g+7
// of depth l; child c has in-group coordinates (c>>2, (c>>1)&1, c&1).  For a
// tap offset (dx,dy,dz) in [-r,r]^3 the neighbour's coordinate relative to
// the group's first child is u = child + d in [-r, 1+r] per axis, its parent
// lies at parent offset floor(u/2) in {-1,0,1} (r <= 2) and it is child
// (u & 1) of that parent.  nbr[g][parent offset] holds the parent's
// first-child row (or -1), so every tap is one table read plus an add: the
// (K+1)^3 union neighbourhood of the eight siblings (Sec. 3.2, Fig. 4).
//
// Stride 1 runs on the matrix-core kernels of conv_mfma.hip (fp32) and
// conv_bf16.hip (bf16 with both channel counts multiples of 16; other bf16
// shapes widen their operands to fp32, which is exact, and run the fp32
// kernels); strides 2^r on the gathered-row GEMMs of conv_sr.hip.  This file
// checks arguments, sizes the workspaces and applies the ReLU backward ahead of
// the stride-1 gradients.
#include <algorithm>

#include "common.h"
#include "conv_bf16.h"
#include "conv_mfma.h"
#include "conv_sr.h"

namespace {

constexpr int TB = 256;

// bf16 -> fp32 (exact), eight elements per thread when the buffers allow.
__global__ __launch_bounds__(TB) void k_bf16_to_f32(const uint16_t* __restrict__ in, int64_t n,
                                                    int vec, float* __restrict__ out) {
  const int64_t e = 8 * ((int64_t)blockIdx.x * TB + threadIdx.x);
  if (e >= n) return;
  if (vec && e + 8 <= n) {  // vec: in 16-byte and out 32-byte aligned
    const uint4 u = *reinterpret_cast<const uint4*>(in + e);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
    float4 a, b;
    a.x = __uint_as_float(w[0] << 16), a.y = __uint_as_float(w[0] & 0xFFFF0000u);
    a.z = __uint_as_float(w[1] << 16), a.w = __uint_as_float(w[1] & 0xFFFF0000u);
    b.x = __uint_as_float(w[2] << 16), b.y = __uint_as_float(w[2] & 0xFFFF0000u);
    b.z = __uint_as_float(w[3] << 16), b.w = __uint_as_float(w[3] & 0xFFFF0000u);
    *reinterpret_cast<float4*>(out + e) = a;
    *reinterpret_cast<float4*>(out + e + 4) = b;
  } else {
    for (int64_t i = e; i < n && i < e + 8; ++i) out[i] = __uint_as_float((uint32_t)in[i] << 16);
  }
}

void bf16_to_f32(const void* in, int64_t n, float* out, hipStream_t s) {
  if (n <= 0) return;
  const int vec = (uintptr_t)in % 16 == 0 && (uintptr_t)out % 32 == 0;
  oc::launch(k_bf16_to_f32, dim3((unsigned)oc::cdiv(n, 8 * TB)), dim3(TB), 0, s,
                     (const uint16_t*)in, n, vec, out);
}

// fp32 value rounded to the nearest bf16 (ties to even), kept as fp32.
__device__ __forceinline__ float round_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u) return f;  // inf, NaN
  return __uint_as_float((u + 0x7fffu + ((u >> 16) & 1u)) & 0xffff0000u);
}

// ReLU backward: dym[e] = y[e] > 0 ? dy[e] : 0 (y NULL: no mask), rounded to
// bf16 when rnd != 0, four entries per thread.
__global__ __launch_bounds__(TB) void k_relu_mask(const float* __restrict__ y,
                                                  const float* __restrict__ dy, int64_t n,
                                                  int vec, int rnd, float* __restrict__ dym) {
  const int64_t e = 4 * ((int64_t)blockIdx.x * TB + threadIdx.x);
  if (e >= n) return;
  if (vec && e + 4 <= n) {  // vec: y, dy (and dym) are 16-byte aligned
    float4 g = *reinterpret_cast<const float4*>(dy + e);
    if (y) {
      const float4 a = *reinterpret_cast<const float4*>(y + e);
      g = float4{a.x > 0.f ? g.x : 0.f, a.y > 0.f ? g.y : 0.f, a.z > 0.f ? g.z : 0.f,
                 a.w > 0.f ? g.w : 0.f};
    }
    if (rnd) g = float4{round_bf16(g.x), round_bf16(g.y), round_bf16(g.z), round_bf16(g.w)};
    *reinterpret_cast<float4*>(dym + e) = g;
  } else {
    for (int64_t i = e; i < n && i < e + 4; ++i) {
      const float g = y && !(y[i] > 0.f) ? 0.f : dy[i];
      dym[i] = rnd ? round_bf16(g) : g;
    }
  }
}

inline unsigned grid_for(int64_t n) { return (unsigned)oc::cdiv(n, TB); }

struct ConvShape {
  int K, K3, stride, r;  // stride 2^r
  int64_t n_in, n_out, units;  // units: output positions (rows, or groups for stride 2)
};

oc_status check_conv(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                     int32_t cin, int32_t cout, ConvShape* sh, const char* who) {
  oc_status st = oc::check_tree_level(t, l, 1);
  if (st != OC_OK) return st;
  if (dt != OC_F32 && dt != OC_BF16) return oc::fail(OC_ERR_ARG, "%s: bad dtype %d", who, (int)dt);
  if (stride < 1 || stride > (1 << OC_MAX_DEPTH) || (stride & (stride - 1)) != 0)
    return oc::fail(OC_ERR_ARG, "%s: stride %d not a power of two in 1..%d", who, stride,
                    1 << OC_MAX_DEPTH);
  if (K != 3 && K != 5) return oc::fail(OC_ERR_UNSUPPORTED, "%s: kernel size %d not 3 or 5", who, K);
  if (stride > 1 && K != 3)
    return oc::fail(OC_ERR_UNSUPPORTED, "%s: stride %d supports kernel size 3 only", who, stride);
  const int r = __builtin_ctz((unsigned)stride);
  if (l < r) return oc::fail(OC_ERR_ARG, "%s: stride %d needs depth >= %d", who, stride, r);
  if (cin < 1 || cin > 1024 || cout < 1 || cout > 1024)
    return oc::fail(OC_ERR_ARG, "%s: channels %d -> %d out of range", who, cin, cout);
  sh->K = K;
  sh->K3 = K * K * K;
  sh->stride = stride;
  sh->n_in = t->N[l];
  sh->r = r;
  sh->n_out = t->N[l - r];
  sh->units = stride == 1 ? t->N[l] : t->M[l - r];
  return OC_OK;
}

// Workspace bytes of each part of a convolution call.  A bf16 stride-1 call
// first widens its bf16 operands to fp32 in the workspace (exact) and runs
// the fp32 matrix-core kernels on them: x32 [n_in][cin], w32 [K^3][cin][cout]
// at the front of the workspace.
size_t x32_bytes(const ConvShape& sh, int cin) {
  return oc::align256((size_t)sh.n_in * cin * sizeof(float));
}
size_t w32_bytes(const ConvShape& sh, int cin, int cout) {
  return oc::align256((size_t)sh.K3 * cin * cout * sizeof(float));
}

// bf16 stride-1 calls whose channel counts the bf16 matrix-core kernels take
// The bf16 kernels address x and dy through 32-bit byte offsets: layers whose
// rows span 2 GiB or more run the fp32 kernels on widened operands instead.
bool bf16_native(const ConvShape& sh, oc_dtype dt, int cin, int cout) {
  return dt == OC_BF16 && sh.stride == 1 && oc::conv_bf16_supported(sh.K, cin, cout) &&
         sh.n_in * std::max(cin, cout) * 2 < ((int64_t)1 << 31);
}

size_t fwd_ws_bytes(const oc_octree* t, int32_t l, const ConvShape& sh, oc_dtype dt, int cin,
                    int cout) {
  if (sh.stride > 1) return oc::conv_s2_fwd_ws(t, l, sh.r, cin, cout, dt == OC_BF16);
  if (sh.n_in == 0) return 0;
  if (bf16_native(sh, dt, cin, cout)) return oc::conv_bf16_fwd_ws(sh.K, cin, cout);
  const size_t tile = oc::conv_s1_tile_ws(t, l, sh.K, cin, cout);
  return dt == OC_F32 ? tile : x32_bytes(sh, cin) + w32_bytes(sh, cin, cout) + tile;
}

// Workspace of the conv + pool forward: the fused kernels' split partials,
// or the depth-l output followed by the plain forward's workspace.
size_t yl_bytes(const ConvShape& sh, int cout) {
  return oc::align256((size_t)sh.n_in * cout * sizeof(float));
}
bool pool_fused(const oc_octree* t, int32_t l, const ConvShape& sh, oc_dtype dt, int cin,
                int cout) {
  return dt == OC_F32 && sh.n_in > 0 && oc::conv_s1_pool_fused(t, l, sh.K, cin, cout);
}
size_t pool_fwd_ws_bytes(const oc_octree* t, int32_t l, const ConvShape& sh, oc_dtype dt, int cin,
                         int cout) {
  if (sh.n_in == 0) return 0;
  if (pool_fused(t, l, sh, dt, cin, cout)) return oc::conv_s1_tile_ws(t, l, sh.K, cin, cout);
  return yl_bytes(sh, cout) + fwd_ws_bytes(t, l, sh, dt, cin, cout);
}

// The matrix-core path applies the ReLU backward once, into the workspace,
// ahead of both gradients.
size_t mask_ws_bytes(const ConvShape& sh, int cout) {
  return oc::align256((size_t)sh.n_out * cout * sizeof(float));
}

// oc_conv_bwd_pool: the depth-l input gradient (stored only when the
// reduction is not split, or for the unfused shapes), the ReLU-masked
// upstream gradient, the input gradient's partial sums.
size_t bwd_pool_ws_bytes(const oc_octree* t, int32_t l, const ConvShape& sh, int cin, int cout) {
  if (sh.n_in == 0) return 0;
  return x32_bytes(sh, cin) + mask_ws_bytes(sh, cout) + oc::conv_s1_tile_ws(t, l, sh.K, cout, cin);
}

size_t bwd_ws_bytes(const oc_octree* t, int32_t l, const ConvShape& sh, oc_dtype dt, int cin,
                    int cout) {
  if (sh.units == 0) return 0;
  const size_t entries = (size_t)sh.K3 * cin * cout;
  if (bf16_native(sh, dt, cin, cout)) return oc::conv_bf16_bwd_ws(t, l, sh.K, cin, cout);
  if (sh.stride == 1) {
    // (bf16: the widened w and x,) the ReLU-masked upstream gradient, then
    // the input gradient's and the weight gradient's partial sums: the same
    // bytes serve both in stream order
    const size_t a = oc::conv_s1_tile_ws(t, l, sh.K, cout, cin);
    const size_t b = oc::conv_s1_dw_parts(t, l, sh.K, cin, cout) * entries * sizeof(float);
    const size_t wide = dt == OC_F32 ? 0 : w32_bytes(sh, cin, cout) + x32_bytes(sh, cin);
    return wide + mask_ws_bytes(sh, cout) + std::max(a, b);
  }
  return oc::conv_s2_bwd_ws(t, l, sh.r, cin, cout, dt == OC_BF16, true, true);
}

}  // namespace

oc_status oc::conv_check(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                         int32_t cin, int32_t cout, const char* who) {
  ConvShape sh;
  return check_conv(t, l, K, stride, dt, cin, cout, &sh, who);
}

extern "C" {

const char* oc_conv_kernel(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                           int32_t cin, int32_t cout, int32_t pass) {
  static thread_local char name[128];
  name[0] = 0;
  ConvShape sh;
  if (pass < 0 || pass > 3 || (pass == 3 && stride != 1)) {
    oc::fail(OC_ERR_ARG, "oc_conv_kernel: pass %d not 0, 1, 2 or (stride 1) 3", pass);
    return name;
  }
  if (check_conv(t, l, K, stride, dt, cin, cout, &sh, "oc_conv_kernel") != OC_OK) return name;
  if (pass == 3 && !pool_fused(t, l, sh, dt, cin, cout)) pass = 0;  // conv, then the pooling
  if (bf16_native(sh, dt, cin, cout)) {
    oc::conv_bf16_kernel_name(K, cin, cout, pass, t->N[l], name, sizeof(name));
  } else if (stride == 1) {  // other bf16 shapes run the fp32 kernels on widened operands
    oc::conv_s1_kernel_name(t, l, K, cin, cout, pass, name, sizeof(name));
  } else {
    snprintf(name, sizeof(name), "%s", oc::conv_sr_kernel_name(pass, sh.r, dt == OC_BF16, cin, cout));
  }
  return name;
}

size_t oc_conv_fwd_workspace(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                             int32_t cin, int32_t cout) {
  ConvShape sh;
  if (check_conv(t, l, K, stride, dt, cin, cout, &sh, "oc_conv_fwd_workspace") != OC_OK) return 0;
  return fwd_ws_bytes(t, l, sh, dt, cin, cout);
}

oc_status oc_conv_fwd(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                      const void* x, int32_t cin, const void* w, int32_t cout, float* y,
                      void* ws, size_t ws_bytes, int32_t flags, hipStream_t s) {
  ConvShape sh;
  oc_status st = check_conv(t, l, K, stride, dt, cin, cout, &sh, "oc_conv_fwd");
  if (st != OC_OK) return st;
  if (!x || !w || !y) return oc::fail(OC_ERR_ARG, "oc_conv_fwd: NULL buffer");
  if (sh.n_out == 0) return OC_OK;
  const size_t need = fwd_ws_bytes(t, l, sh, dt, cin, cout);
  if (need && (!ws || ws_bytes < need))
    return oc::fail(OC_ERR_ARG, "oc_conv_fwd: workspace %zu bytes < %zu", ws ? ws_bytes : 0, need);
  const int relu = (flags & OC_FUSE_RELU) ? 1 : 0;
  if (bf16_native(sh, dt, cin, cout)) {
    oc::conv_bf16_fwd(t, l, K, (const uint16_t*)x, cin, (const uint16_t*)w, cout, y, relu, ws, s);
    OC_LAUNCH_CHECK();
    return OC_OK;
  }
  if (stride == 1) {
    const float *x32 = (const float*)x, *w32 = (const float*)w;
    char* rest = (char*)ws;
    if (dt == OC_BF16) {
      float* xw = (float*)rest;
      float* ww = (float*)(rest + x32_bytes(sh, cin));
      bf16_to_f32(x, sh.n_in * (int64_t)cin, xw, s);
      bf16_to_f32(w, (int64_t)sh.K3 * cin * cout, ww, s);
      x32 = xw, w32 = ww;
      rest += x32_bytes(sh, cin) + w32_bytes(sh, cin, cout);
    }
    oc::conv_s1_fwd_f32(t, l, K, x32, cin, w32, cout, y, relu, (float*)rest, s);
    OC_LAUNCH_CHECK();
    return OC_OK;
  }
  st = oc::conv_s2_fwd(t, l, sh.r, x, cin, w, cout, dt == OC_BF16, y, relu, ws, s);
  if (st != OC_OK) return st;
  OC_LAUNCH_CHECK();
  return OC_OK;
}

size_t oc_conv_pool_fwd_workspace(const oc_octree* t, int32_t l, int32_t K, oc_dtype dt,
                                  int32_t cin, int32_t cout) {
  ConvShape sh;
  if (check_conv(t, l, K, 1, dt, cin, cout, &sh, "oc_conv_pool_fwd_workspace") != OC_OK) return 0;
  return pool_fwd_ws_bytes(t, l, sh, dt, cin, cout);
}

oc_status oc_conv_pool_fwd(const oc_octree* t, int32_t l, int32_t K, oc_dtype dt, const void* x,
                           int32_t cin, const void* w, int32_t cout, float* y, uint8_t* sw,
                           void* ws, size_t ws_bytes, int32_t flags, hipStream_t s) {
  ConvShape sh;
  oc_status st = check_conv(t, l, K, 1, dt, cin, cout, &sh, "oc_conv_pool_fwd");
  if (st != OC_OK) return st;
  if (t->N[l - 1] == 0) return OC_OK;
  // (x and sw are empty, and may be NULL, when depth l has no octant)
  if ((sh.n_in > 0 && (!x || !sw)) || !w || !y)
    return oc::fail(OC_ERR_ARG, "oc_conv_pool_fwd: NULL buffer");
  if ((uintptr_t)y % 16 != 0 || (uintptr_t)sw % 4 != 0)
    return oc::fail(OC_ERR_ARG, "oc_conv_pool_fwd: y not 16-byte or sw not 4-byte aligned");
  const size_t need = pool_fwd_ws_bytes(t, l, sh, dt, cin, cout);
  if (need && (!ws || ws_bytes < need))
    return oc::fail(OC_ERR_ARG, "oc_conv_pool_fwd: workspace %zu bytes < %zu", ws ? ws_bytes : 0,
                    need);
  const int relu = (flags & OC_FUSE_RELU) ? 1 : 0;
  if (sh.n_in == 0) {  // no depth-l octant: every pooled row is zero
    oc::fill_u32(y, 0u, t->N[l - 1] * (int64_t)cout, s);
    OC_LAUNCH_CHECK();
    return OC_OK;
  }
  if (pool_fused(t, l, sh, dt, cin, cout)) {
    oc::conv_s1_pool_fwd_f32(t, l, K, (const float*)x, cin, (const float*)w, cout, y, sw, relu,
                             (float*)ws, s);
    OC_LAUNCH_CHECK();
    return OC_OK;
  }
  // other shapes: the depth-l output into the workspace, then the pooling
  float* yl = (float*)ws;
  const size_t head = yl_bytes(sh, cout);
  st = oc_conv_fwd(t, l, K, 1, dt, x, cin, w, cout, yl, (char*)ws + head, ws_bytes - head, flags,
                   s);
  if (st != OC_OK) return st;
  return oc_pool_fwd(t, l, yl, cout, y, sw, s);
}

size_t oc_conv_bwd_workspace(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                             int32_t cin, int32_t cout) {
  ConvShape sh;
  if (check_conv(t, l, K, stride, dt, cin, cout, &sh, "oc_conv_bwd_workspace") != OC_OK) return 0;
  return bwd_ws_bytes(t, l, sh, dt, cin, cout);
}

size_t oc_conv_bwd_pool_workspace(const oc_octree* t, int32_t l, int32_t K, int32_t cin,
                                  int32_t cout) {
  ConvShape sh;
  if (check_conv(t, l, K, 1, OC_F32, cin, cout, &sh, "oc_conv_bwd_pool_workspace") != OC_OK) return 0;
  return bwd_pool_ws_bytes(t, l, sh, cin, cout);
}

oc_status oc_conv_bwd_pool(const oc_octree* t, int32_t l, int32_t K, const float* w, int32_t cin,
                           int32_t cout, const float* y, const float* dy, const float* xp,
                           const uint8_t* sw, float* dxf, float* dym, void* ws, size_t ws_bytes,
                           int32_t flags, hipStream_t s) {
  ConvShape sh;
  oc_status st = check_conv(t, l, K, 1, OC_F32, cin, cout, &sh, "oc_conv_bwd_pool");
  if (st != OC_OK) return st;
  st = oc::check_tree_level(t, l + 1, 1);
  if (st != OC_OK) return st;
  if (sh.n_in == 0) return OC_OK;  // no depth-l octant: no depth-(l+1) octant either
  if (!w || !dy || !sw || !dxf) return oc::fail(OC_ERR_ARG, "oc_conv_bwd_pool: NULL buffer");
  if ((flags & OC_FUSE_RELU) && !y)
    return oc::fail(OC_ERR_ARG, "oc_conv_bwd_pool: OC_FUSE_RELU needs y");
  const size_t need = bwd_pool_ws_bytes(t, l, sh, cin, cout);
  if (!ws || ws_bytes < need)
    return oc::fail(OC_ERR_ARG, "oc_conv_bwd_pool: workspace %zu bytes < %zu", ws ? ws_bytes : 0,
                    need);
  float* dxl = (float*)ws;
  float* wsf = (float*)((char*)ws + x32_bytes(sh, cin));
  if (flags & OC_FUSE_RELU) {  // dy masked with [y > 0] (into dym when given)
    float* m = dym ? dym : wsf;
    const int64_t n = sh.n_out * (int64_t)cout;
    const int vec = (uintptr_t)y % 16 == 0 && (uintptr_t)dy % 16 == 0 && (uintptr_t)m % 16 == 0;
    oc::launch(k_relu_mask, dim3((unsigned)oc::cdiv(n, 4 * TB)), dim3(TB), 0, s, y, dy, n, vec, 0,
               m);
    dy = m;
  }
  wsf = (float*)((char*)wsf + mask_ws_bytes(sh, cout));
  if (cin % 4 == 0 && (uintptr_t)dxf % 16 == 0 && (uintptr_t)sw % 4 == 0 &&
      (!xp || (uintptr_t)xp % 16 == 0)) {
    oc::conv_s1_bwd_data_pool_f32(t, l, K, dy, cout, w, cin, dxl, xp, sw, dxf, wsf, s);
    OC_LAUNCH_CHECK();
    return OC_OK;
  }
  // other shapes: the depth-l input gradient, then the pool backward
  oc::conv_s1_bwd_data_f32(t, l, K, dy, cout, w, cin, dxl, wsf, s);
  OC_LAUNCH_CHECK();
  return oc_pool_bwd(t, l + 1, dxl, sw, cin, xp, dxf, s);
}

oc_status oc_conv_bwd(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                      const void* x, int32_t cin, const void* w, int32_t cout, const float* y,
                      const float* dy, float* dx, float* dw, void* ws, size_t ws_bytes,
                      int32_t flags, hipStream_t s) {
  ConvShape sh;
  oc_status st = check_conv(t, l, K, stride, dt, cin, cout, &sh, "oc_conv_bwd");
  if (st != OC_OK) return st;
  if (!w || !dy) return oc::fail(OC_ERR_ARG, "oc_conv_bwd: NULL w or dy");
  if ((flags & OC_FUSE_RELU) && !y) return oc::fail(OC_ERR_ARG, "oc_conv_bwd: OC_FUSE_RELU needs y");
  if (dw && !x) return oc::fail(OC_ERR_ARG, "oc_conv_bwd: dw needs x");
  const size_t need = (dx || dw) ? bwd_ws_bytes(t, l, sh, dt, cin, cout) : 0;
  if (need && (!ws || ws_bytes < need))
    return oc::fail(OC_ERR_ARG, "oc_conv_bwd: workspace %zu bytes < %zu", ws ? ws_bytes : 0, need);
  const float* ym = (flags & OC_FUSE_RELU) ? y : nullptr;
  if (stride > 1) {
    st = oc::conv_s2_bwd(t, l, sh.r, x, cin, w, cout, dt == OC_BF16, ym, dy, dx, dw, ws, s);
    if (st != OC_OK) return st;
    OC_LAUNCH_CHECK();
    return OC_OK;
  }
  if (bf16_native(sh, dt, cin, cout)) {
    if (sh.units == 0) {
      if (dw) oc::fill_u32(dw, 0u, (int64_t)sh.K3 * cin * cout, s);
    } else if (dx || dw) {
      oc::conv_bf16_bwd(t, l, K, (const uint16_t*)x, cin, (const uint16_t*)w, cout, ym, dy, dx, dw,
                        ws, s);
    }
    OC_LAUNCH_CHECK();
    return OC_OK;
  }
  // stride 1: matrix-core kernels
  float* wsf = (float*)ws;
  if (dt == OC_BF16 && (dx || dw)) {  // the bf16 operands widened to fp32 (exact)
    float* ww = wsf;
    float* xw = (float*)((char*)ws + w32_bytes(sh, cin, cout));
    if (dx) bf16_to_f32(w, (int64_t)sh.K3 * cin * cout, ww, s);
    if (dw) bf16_to_f32(x, sh.n_in * (int64_t)cin, xw, s);
    w = ww;
    x = xw;
    wsf = (float*)((char*)ws + w32_bytes(sh, cin, cout) + x32_bytes(sh, cin));
  }
  if (dx || dw) {
    // dy masked once (and for bf16 rounded to bf16, the operand precision of
    // the bf16 backward), read by both gradients
    const int rnd = dt == OC_BF16;
    if ((ym || rnd) && sh.n_out > 0) {
      const int64_t n = sh.n_out * (int64_t)cout;
      const int vec = ((!ym || (uintptr_t)ym % 16 == 0) && (uintptr_t)dy % 16 == 0 &&
                       (uintptr_t)wsf % 16 == 0);
      oc::launch(k_relu_mask, dim3((unsigned)oc::cdiv(n, 4 * TB)), dim3(TB), 0, s, ym, dy,
                         n, vec, rnd, wsf);
      dy = wsf;
    }
    wsf = (float*)((char*)wsf + mask_ws_bytes(sh, cout));
  }
  if (dx && sh.n_in > 0) oc::conv_s1_bwd_data_f32(t, l, K, dy, cout, (const float*)w, cin, dx, wsf, s);
  if (dw) {
    if (sh.units == 0)
      oc::fill_u32(dw, 0u, (int64_t)sh.K3 * cin * cout, s);
    else
      oc::conv_s1_bwd_weight_f32(t, l, K, (const float*)x, cin, dy, cout, dw, wsf, s,
                                 (flags & OC_DEFER_DW) != 0);
  }
  OC_LAUNCH_CHECK();
  return OC_OK;
}

oc_status oc_conv_dw_partials(const oc_octree* t, int32_t l, int32_t K, int32_t stride,
                              oc_dtype dt, int32_t cin, int32_t cout, size_t* offset,
                              int32_t* nparts, int64_t* count) {
  ConvShape sh;
  oc_status st = check_conv(t, l, K, stride, dt, cin, cout, &sh, "oc_conv_dw_partials");
  if (st != OC_OK) return st;
  if (!offset || !nparts || !count)
    return oc::fail(OC_ERR_ARG, "oc_conv_dw_partials: NULL output pointer");
  *count = (int64_t)sh.K3 * cin * cout;
  *offset = 0;
  *nparts = 0;
  // strided and native-bf16 layers, and layers without groups, write dw directly
  if (stride > 1 || bf16_native(sh, dt, cin, cout) || sh.units == 0) return OC_OK;
  // oc_conv_bwd's stride-1 workspace: (bf16: widened w and x,) the masked dy,
  // then the weight gradient's partial sums
  size_t off = mask_ws_bytes(sh, cout);
  if (dt == OC_BF16) off += w32_bytes(sh, cin, cout) + x32_bytes(sh, cin);
  *offset = off;
  *nparts = (int32_t)oc::conv_s1_dw_parts(t, l, K, cin, cout);
  return OC_OK;
}

oc_status oc_sum_partials(int32_t n, const float* const* parts, const int32_t* nparts,
                          const int64_t* counts, float* const* outs, hipStream_t s) {
  if (n < 0) return oc::fail(OC_ERR_ARG, "oc_sum_partials: n = %d < 0", (int)n);
  if (n == 0) return OC_OK;
  if (!parts || !nparts || !counts || !outs)
    return oc::fail(OC_ERR_ARG, "oc_sum_partials: NULL array");
  for (int i = 0; i < n; ++i) {
    if (nparts[i] < 1 || counts[i] < 0 || (counts[i] > 0 && (!parts[i] || !outs[i])))
      return oc::fail(OC_ERR_ARG, "oc_sum_partials: set %d: %d partials of %lld entries", i,
                      (int)nparts[i], (long long)counts[i]);
  }
  oc::sum_partials_multi(n, parts, (const int*)nparts, counts, outs, s);
  OC_LAUNCH_CHECK();
  return OC_OK;
}

oc_status oc_round_bf16(int64_t n, const float* x, uint16_t* y, hipStream_t s) {
  if (n < 0) return oc::fail(OC_ERR_ARG, "oc_round_bf16: n = %lld < 0", (long long)n);
  if (n == 0) return OC_OK;
  if (!x || !y) return oc::fail(OC_ERR_ARG, "oc_round_bf16: NULL buffer");
  oc::round_bf16(x, n, y, s);
  OC_LAUNCH_CHECK();
  return OC_OK;
}

}  // extern "C"
