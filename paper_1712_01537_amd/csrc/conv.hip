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
// Backward w.r.t. the input.  For stride 1, j is the neighbour of i at
// offset d iff i is the neighbour of j at offset -d, and every octant of
// depth l is both an input and an output row; hence dX = conv(dY, W') with
// W'[k] = W[K^3-1-k]^T, evaluated by the forward gather.  For stride 2 each
// input octant receives from at most 2^(number of odd child bits) outputs,
// reached through the same table.
// Backward w.r.t. the weights: dW[k] = sum_i X[n(i,k)]^T dY[i], split over
// row chunks into partial sums that a second kernel adds in a fixed order
// (no floating-point atomics, so results are reproducible bit for bit).
#include <algorithm>

#include "common.h"
#include "conv_mfma.h"

namespace {

constexpr int TB = 256;

__device__ __forceinline__ float ld(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float ld(const uint16_t* p, int64_t i) {
  return __uint_as_float((uint32_t)p[i] << 16);
}

// Source row of tap (dx,dy,dz) of child c in group g, or -1.
__device__ __forceinline__ int32_t tap_row(const int32_t* nb, int c, int dx, int dy, int dz) {
  const int ux = (c >> 2) + dx, uy = ((c >> 1) & 1) + dy, uz = (c & 1) + dz;
  const int32_t base = nb[((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1)];
  return base < 0 ? -1 : base + 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1);
}

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
  hipLaunchKernelGGL(k_bf16_to_f32, dim3((unsigned)oc::cdiv(n, 8 * TB)), dim3(TB), 0, s,
                     (const uint16_t*)in, n, vec, out);
}

// ReLU backward: dym[e] = y[e] > 0 ? dy[e] : 0, four entries per thread.
__global__ __launch_bounds__(TB) void k_relu_mask(const float* __restrict__ y,
                                                  const float* __restrict__ dy, int64_t n,
                                                  int vec, float* __restrict__ dym) {
  const int64_t e = 4 * ((int64_t)blockIdx.x * TB + threadIdx.x);
  if (e >= n) return;
  if (vec && e + 4 <= n) {  // vec: y, dy (and dym) are 16-byte aligned
    const float4 a = *reinterpret_cast<const float4*>(y + e);
    const float4 g = *reinterpret_cast<const float4*>(dy + e);
    *reinterpret_cast<float4*>(dym + e) = float4{a.x > 0.f ? g.x : 0.f, a.y > 0.f ? g.y : 0.f,
                                                 a.z > 0.f ? g.z : 0.f, a.w > 0.f ? g.w : 0.f};
  } else {
    for (int64_t i = e; i < n; ++i) dym[i] = y[i] > 0.f ? dy[i] : 0.f;
  }
}

// Forward.  stride 1: output row i = group i>>3, child i&7.  stride 2:
// output row i of depth l-1 with label L > 0 evaluates child 0 of group L-1.
template <typename T>
__global__ __launch_bounds__(TB) void k_conv_fwd_simple(const int32_t* __restrict__ nbr,
                                                        const int32_t* __restrict__ labels_out,
                                                        int64_t n_out, int stride, int K,
                                                        const T* __restrict__ x, int cin,
                                                        const T* __restrict__ w, int cout,
                                                        float* __restrict__ y, int relu) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_out * cout) return;
  const int64_t i = t / cout;
  const int co = (int)(t - i * cout);
  int64_t g;
  int c;
  if (stride == 1) {
    g = i >> 3;
    c = (int)(i & 7);
  } else {
    const int32_t L = labels_out[i];
    if (L == 0) {
      y[t] = 0.0f;
      return;
    }
    g = L - 1;
    c = 0;
  }
  const int r = (K - 1) / 2;
  const int32_t* nb = nbr + 27 * g;
  float acc = 0.0f;
  int k = 0;
  for (int dx = -r; dx <= r; ++dx)
    for (int dy = -r; dy <= r; ++dy)
      for (int dz = -r; dz <= r; ++dz, ++k) {
        const int32_t src = tap_row(nb, c, dx, dy, dz);
        if (src < 0) continue;
        for (int ci = 0; ci < cin; ++ci)
          acc = fmaf(ld(x, (int64_t)src * cin + ci), ld(w, ((int64_t)k * cin + ci) * cout + co), acc);
      }
  y[t] = relu ? fmaxf(acc, 0.0f) : acc;
}

// Upstream gradient with the fused-ReLU mask applied.
__device__ __forceinline__ float dy_eff(const float* dy, const float* y, int64_t idx) {
  const float g = dy[idx];
  return y ? (y[idx] > 0.0f ? g : 0.0f) : g;
}

// Backward data, stride 1: dX[j][ci] = sum_k sum_co dY[n(j,k)][co] W[K^3-1-k][ci][co].
template <typename T>
__global__ __launch_bounds__(TB) void k_conv_bwd_data_s1_simple(
    const int32_t* __restrict__ nbr, int64_t n, int K, const float* __restrict__ dy,
    const float* __restrict__ y, int cout, const T* __restrict__ w, int cin,
    float* __restrict__ dx) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n * cin) return;
  const int64_t j = t / cin;
  const int ci = (int)(t - j * cin);
  const int r = (K - 1) / 2, K3 = K * K * K;
  const int32_t* nb = nbr + 27 * (j >> 3);
  const int c = (int)(j & 7);
  float acc = 0.0f;
  int k = 0;
  for (int ddx = -r; ddx <= r; ++ddx)
    for (int ddy = -r; ddy <= r; ++ddy)
      for (int ddz = -r; ddz <= r; ++ddz, ++k) {
        const int32_t src = tap_row(nb, c, ddx, ddy, ddz);
        if (src < 0) continue;
        const int kf = K3 - 1 - k;
        for (int co = 0; co < cout; ++co)
          acc = fmaf(dy_eff(dy, y, (int64_t)src * cout + co), ld(w, ((int64_t)kf * cin + ci) * cout + co), acc);
      }
  dx[t] = acc;
}

// Backward data, stride 2 (K = 3): input row j = 8g' + c' receives from the
// outputs whose first child sees it: parent offset p_a in {0} if c'_a = 0,
// {0, 1} if c'_a = 1, with tap d_a = c'_a - 2 p_a.
template <typename T>
__global__ __launch_bounds__(TB) void k_conv_bwd_data_s2_simple(
    const int32_t* __restrict__ nbr, const int32_t* __restrict__ rows_out, int64_t n,
    const float* __restrict__ dy, const float* __restrict__ y, int cout, const T* __restrict__ w,
    int cin, float* __restrict__ dx) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n * cin) return;
  const int64_t j = t / cin;
  const int ci = (int)(t - j * cin);
  const int32_t* nb = nbr + 27 * (j >> 3);
  const int c = (int)(j & 7);
  const int cx = c >> 2, cy = (c >> 1) & 1, cz = c & 1;
  float acc = 0.0f;
  for (int px = 0; px <= cx; ++px)
    for (int py = 0; py <= cy; ++py)
      for (int pz = 0; pz <= cz; ++pz) {
        const int32_t f = nb[(px + 1) * 9 + (py + 1) * 3 + (pz + 1)];
        if (f < 0) continue;
        const int64_t orow = rows_out[f >> 3];
        const int k = ((cx - 2 * px + 1) * 3 + (cy - 2 * py + 1)) * 3 + (cz - 2 * pz + 1);
        for (int co = 0; co < cout; ++co)
          acc = fmaf(dy_eff(dy, y, orow * cout + co), ld(w, ((int64_t)k * cin + ci) * cout + co), acc);
      }
  dx[t] = acc;
}

// Backward weights, partial sums over chunk q of the output rows.
// stride 1: rows i in [q*chunk, ...), child i&7 of group i>>3, upstream row i.
// stride 2: groups g in the chunk, child 0, upstream row rows_out[g].
template <typename T>
__global__ __launch_bounds__(TB) void k_conv_dw_partial_simple(
    const int32_t* __restrict__ nbr, const int32_t* __restrict__ rows_out, int64_t n_units,
    int stride, int K, const T* __restrict__ x, int cin, const float* __restrict__ dy,
    const float* __restrict__ y, int cout, int64_t chunk, float* __restrict__ part) {
  const int64_t entries = (int64_t)K * K * K * cin * cout;
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e >= entries) return;
  const int q = blockIdx.y;
  const int k = (int)(e / ((int64_t)cin * cout));
  const int ci = (int)((e / cout) % cin);
  const int co = (int)(e % cout);
  const int r = (K - 1) / 2;
  const int dxo = k / (K * K) - r, dyo = (k / K) % K - r, dzo = k % K - r;
  const int64_t u0 = (int64_t)q * chunk, u1 = min(n_units, u0 + chunk);
  float acc = 0.0f;
  for (int64_t u = u0; u < u1; ++u) {
    int64_t g, orow;
    int c;
    if (stride == 1) {
      g = u >> 3;
      c = (int)(u & 7);
      orow = u;
    } else {
      g = u;
      c = 0;
      orow = rows_out[u];
    }
    const int32_t src = tap_row(nbr + 27 * g, c, dxo, dyo, dzo);
    if (src < 0) continue;
    acc = fmaf(ld(x, (int64_t)src * cin + ci), dy_eff(dy, y, orow * cout + co), acc);
  }
  part[(int64_t)q * entries + e] = acc;
}

__global__ __launch_bounds__(TB) void k_reduce_parts(const float* __restrict__ part, int nparts,
                                                     int64_t entries, float* __restrict__ out) {
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e >= entries) return;
  float s = 0.0f;
  for (int q = 0; q < nparts; ++q) s += part[(int64_t)q * entries + e];
  out[e] = s;
}

inline unsigned grid_for(int64_t n) { return (unsigned)oc::cdiv(n, TB); }

struct ConvShape {
  int K, K3, stride;
  int64_t n_in, n_out, units;  // units: output positions (rows, or groups for stride 2)
};

oc_status check_conv(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                     int32_t cin, int32_t cout, ConvShape* sh, const char* who) {
  oc_status st = oc::check_tree_level(t, l, 1);
  if (st != OC_OK) return st;
  if (dt != OC_F32 && dt != OC_BF16) return oc::fail(OC_ERR_ARG, "%s: bad dtype %d", who, (int)dt);
  if (stride != 1 && stride != 2) return oc::fail(OC_ERR_ARG, "%s: stride %d not 1 or 2", who, stride);
  if (K != 3 && K != 5) return oc::fail(OC_ERR_UNSUPPORTED, "%s: kernel size %d not 3 or 5", who, K);
  if (stride == 2 && K != 3)
    return oc::fail(OC_ERR_UNSUPPORTED, "%s: stride 2 supports kernel size 3 only", who);
  if (cin < 1 || cin > 1024 || cout < 1 || cout > 1024)
    return oc::fail(OC_ERR_ARG, "%s: channels %d -> %d out of range", who, cin, cout);
  sh->K = K;
  sh->K3 = K * K * K;
  sh->stride = stride;
  sh->n_in = t->N[l];
  sh->n_out = stride == 1 ? t->N[l] : t->N[l - 1];
  sh->units = stride == 1 ? t->N[l] : t->M[l - 1];
  return OC_OK;
}

int64_t dw_chunk(const ConvShape& sh, int cin, int cout, int* nparts) {
  const int64_t entries = (int64_t)sh.K3 * cin * cout;
  const int64_t max_parts = std::max<int64_t>(1, (int64_t(64) << 20) / entries);
  int64_t parts = std::min<int64_t>(max_parts, std::max<int64_t>(1, oc::cdiv(sh.units, 2048)));
  int64_t chunk = std::max<int64_t>(1, oc::cdiv(sh.units, parts));
  *nparts = (int)std::max<int64_t>(1, oc::cdiv(sh.units, chunk));
  return chunk;
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

size_t fwd_ws_bytes(const oc_octree* t, int32_t l, const ConvShape& sh, oc_dtype dt, int cin,
                    int cout) {
  if (sh.stride != 1 || sh.n_in == 0) return 0;
  const size_t tile = oc::conv_s1_tile_ws(t, l, sh.K, cin, cout);
  return dt == OC_F32 ? tile : x32_bytes(sh, cin) + w32_bytes(sh, cin, cout) + tile;
}

// The matrix-core path applies the ReLU backward once, into the workspace,
// ahead of both gradients.
size_t mask_ws_bytes(const ConvShape& sh, int cout) {
  return oc::align256((size_t)sh.n_out * cout * sizeof(float));
}

size_t bwd_ws_bytes(const oc_octree* t, int32_t l, const ConvShape& sh, oc_dtype dt, int cin,
                    int cout) {
  if (sh.units == 0) return 0;
  const size_t entries = (size_t)sh.K3 * cin * cout;
  if (sh.stride == 1) {
    // (bf16: the widened w and x,) the ReLU-masked upstream gradient, then
    // the input gradient's and the weight gradient's partial sums: the same
    // bytes serve both in stream order
    const size_t a = oc::conv_s1_tile_ws(t, l, sh.K, cout, cin);
    const size_t b = oc::conv_s1_dw_parts(t, l, sh.K, cin, cout) * entries * sizeof(float);
    const size_t wide = dt == OC_F32 ? 0 : w32_bytes(sh, cin, cout) + x32_bytes(sh, cin);
    return wide + mask_ws_bytes(sh, cout) + std::max(a, b);
  }
  int nparts;
  dw_chunk(sh, cin, cout, &nparts);
  return (size_t)nparts * entries * sizeof(float);
}

}  // namespace

extern "C" {

const char* oc_conv_kernel(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                           int32_t cin, int32_t cout, int32_t pass) {
  static thread_local char name[128];
  name[0] = 0;
  ConvShape sh;
  if (pass < 0 || pass > 2) {
    oc::fail(OC_ERR_ARG, "oc_conv_kernel: pass %d not 0, 1 or 2", pass);
    return name;
  }
  if (check_conv(t, l, K, stride, dt, cin, cout, &sh, "oc_conv_kernel") != OC_OK) return name;
  if (stride == 1) {  // bf16 runs the fp32 kernels on widened operands
    oc::conv_s1_kernel_name(t, l, K, cin, cout, pass, name, sizeof(name));
  } else {
    const char* ty = dt == OC_F32 ? "float" : "unsigned short";
    const char* k = pass == 0   ? "k_conv_fwd_simple"
                    : pass == 2 ? "k_conv_dw_partial_simple"
                    : stride == 1 ? "k_conv_bwd_data_s1_simple"
                                  : "k_conv_bwd_data_s2_simple";
    snprintf(name, sizeof(name), "%s<%s>", k, ty);
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
  const unsigned grid = grid_for(sh.n_out * cout);
  if (dt == OC_F32)
    oc::launch_main(k_conv_fwd_simple<float>, dim3(grid), dim3(TB), s,
                       (const int32_t*)t->nbr[l], (const int32_t*)t->labels[l - 1], sh.n_out, stride,
                       K, (const float*)x, cin, (const float*)w, cout, y, relu);
  else
    oc::launch_main(k_conv_fwd_simple<uint16_t>, dim3(grid), dim3(TB), s,
                       (const int32_t*)t->nbr[l], (const int32_t*)t->labels[l - 1], sh.n_out, stride,
                       K, (const uint16_t*)x, cin, (const uint16_t*)w, cout, y, relu);
  OC_LAUNCH_CHECK();
  return OC_OK;
}

size_t oc_conv_bwd_workspace(const oc_octree* t, int32_t l, int32_t K, int32_t stride, oc_dtype dt,
                             int32_t cin, int32_t cout) {
  ConvShape sh;
  if (check_conv(t, l, K, stride, dt, cin, cout, &sh, "oc_conv_bwd_workspace") != OC_OK) return 0;
  return bwd_ws_bytes(t, l, sh, dt, cin, cout);
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
  int nparts = 0;
  const int64_t chunk = dw_chunk(sh, cin, cout, &nparts);
  const bool mfma = stride == 1;
  float* wsf = (float*)ws;
  if (mfma && dt == OC_BF16 && (dx || dw)) {  // the bf16 operands widened to fp32 (exact)
    float* ww = wsf;
    float* xw = (float*)((char*)ws + w32_bytes(sh, cin, cout));
    if (dx) bf16_to_f32(w, (int64_t)sh.K3 * cin * cout, ww, s);
    if (dw) bf16_to_f32(x, sh.n_in * (int64_t)cin, xw, s);
    w = ww;
    x = xw;
    wsf = (float*)((char*)ws + w32_bytes(sh, cin, cout) + x32_bytes(sh, cin));
  }
  if (mfma && (dx || dw)) {
    if (ym && sh.n_out > 0) {  // dy masked once, read by both gradients
      const int64_t n = sh.n_out * (int64_t)cout;
      const int vec = ((uintptr_t)y % 16 == 0 && (uintptr_t)dy % 16 == 0 && (uintptr_t)wsf % 16 == 0);
      hipLaunchKernelGGL(k_relu_mask, dim3((unsigned)oc::cdiv(n, 4 * TB)), dim3(TB), 0, s, y, dy,
                         n, vec, wsf);
      dy = wsf;
    }
    wsf = (float*)((char*)wsf + mask_ws_bytes(sh, cout));
  }
  const int64_t entries = (int64_t)sh.K3 * cin * cout;
  const int32_t* nbr = t->nbr[l];
  const int32_t* rows_out = t->rows[l - 1];
  if (dx && sh.n_in > 0 && mfma) {
    oc::conv_s1_bwd_data_f32(t, l, K, dy, cout, (const float*)w, cin, dx, wsf, s);
  } else if (dx && sh.n_in > 0) {
    const unsigned grid = grid_for(sh.n_in * cin);
    if (stride == 1) {
      if (dt == OC_F32)
        oc::launch_main(k_conv_bwd_data_s1_simple<float>, dim3(grid), dim3(TB), s, nbr,
                           sh.n_in, K, dy, ym, cout, (const float*)w, cin, dx);
      else
        oc::launch_main(k_conv_bwd_data_s1_simple<uint16_t>, dim3(grid), dim3(TB), s, nbr,
                           sh.n_in, K, dy, ym, cout, (const uint16_t*)w, cin, dx);
    } else {
      if (dt == OC_F32)
        oc::launch_main(k_conv_bwd_data_s2_simple<float>, dim3(grid), dim3(TB), s, nbr,
                           rows_out, sh.n_in, dy, ym, cout, (const float*)w, cin, dx);
      else
        oc::launch_main(k_conv_bwd_data_s2_simple<uint16_t>, dim3(grid), dim3(TB), s, nbr,
                           rows_out, sh.n_in, dy, ym, cout, (const uint16_t*)w, cin, dx);
    }
  }
  if (dw) {
    if (sh.units == 0) {
      oc::fill_u32(dw, 0u, entries, s);
    } else if (mfma) {
      oc::conv_s1_bwd_weight_f32(t, l, K, (const float*)x, cin, dy, cout, dw, wsf, s);
    } else {
      float* part = (float*)ws;
      dim3 grid(grid_for(entries), nparts);
      if (dt == OC_F32)
        oc::launch_main(k_conv_dw_partial_simple<float>, grid, dim3(TB), s, nbr, rows_out,
                           sh.units, stride, K, (const float*)x, cin, dy, ym, cout, chunk, part);
      else
        oc::launch_main(k_conv_dw_partial_simple<uint16_t>, grid, dim3(TB), s, nbr, rows_out,
                           sh.units, stride, K, (const uint16_t*)x, cin, dy, ym, cout, chunk, part);
      hipLaunchKernelGGL(k_reduce_parts, dim3(grid_for(entries)), dim3(TB), 0, s,
                         (const float*)part, nparts, entries, dw);
    }
  }
  OC_LAUNCH_CHECK();
  return OC_OK;
}

}  // extern "C"
