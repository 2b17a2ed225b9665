// Stride-2 octree convolution, K = 3 (Sec. 3.2 of O-CNN, Fig. 2): the output
// of sibling group g is the convolution evaluated at its first child (child
// 0), written to the row of g's parent at depth l-1 (rows of empty parents
// are 0).  The paper evaluates it as im2col + GEMM, and so does this file:
// a gather kernel builds the column buffer Col[g][k][c] = x[n(8g, k)][c]
// (0 for an absent neighbour; only parent offsets {-1,0}^3 are reached from
// child 0), a library GEMM multiplies it by W viewed as [27 Cin][Cout], and
// a second kernel moves each group's row to its parent's row.
//   input gradient: dCol = dY_g W^T (GEMM), then dX[j] = sum of the dCol
//     entries whose tap reads j (gather form of col2im, no atomics);
//   weight gradient: dW = Col^T dY_g (GEMM over the groups, in chunks added
//     in a fixed order through the GEMM's beta).
// dY_g[g] = dY[row of g's parent], masked by [y > 0] when the forward applied
// a ReLU.  bf16: the forward multiplies bf16 Col and W with fp32
// accumulation (exact products); the backward widens to fp32 (the upstream
// gradient is fp32).  GEMM atomics are disabled, so results are bit-for-bit
// reproducible.
#include <mutex>

#include <rocblas/rocblas.h>

#include "common.h"
#include "conv_s2.h"

namespace {

constexpr int TB = 256;
constexpr size_t COL_CAP = size_t(256) << 20;  // bytes of one column-buffer chunk

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(uint16_t v) { return __uint_as_float((uint32_t)v << 16); }

// Column buffer of groups g0 .. g0+ng-1: col[g-g0][k][c], four channels per
// thread; TI -> TO is a copy or an exact bf16 -> fp32 widening.
template <typename TI, typename TO>
__global__ __launch_bounds__(TB) void k_s2_col(const int32_t* __restrict__ nbr, int64_t g0,
                                               int64_t ng, const TI* __restrict__ x, int cin,
                                               TO* __restrict__ col) {
  const int c4n = (cin + 3) / 4;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ng * 27 * c4n) return;
  const int c4 = (int)(t % c4n);
  const int k = (int)((t / c4n) % 27);
  const int64_t gi = t / ((int64_t)27 * c4n);
  const int dx = k / 9 - 1, dy = (k / 3) % 3 - 1, dz = k % 3 - 1;  // child 0 + d
  const int32_t base = nbr[27 * (g0 + gi) + ((dx >> 1) + 1) * 9 + ((dy >> 1) + 1) * 3 + ((dz >> 1) + 1)];
  const int32_t src = base < 0 ? -1 : base + 4 * (dx & 1) + 2 * (dy & 1) + (dz & 1);
  TO* o = col + (gi * 27 + k) * cin + 4 * c4;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (4 * c4 + j >= cin) break;
    if constexpr (sizeof(TI) == sizeof(TO)) {
      o[j] = src < 0 ? TO(0) : x[(int64_t)src * cin + 4 * c4 + j];
    } else {
      o[j] = src < 0 ? 0.f : to_f(x[(int64_t)src * cin + 4 * c4 + j]);
    }
  }
}

// y[i] (depth l-1) = label L > 0 ? yg[L-1] : 0, ReLU applied if relu.
__global__ __launch_bounds__(TB) void k_s2_rows_out(const int32_t* __restrict__ labels,
                                                    int64_t n_out, const float* __restrict__ yg,
                                                    int cout, int relu, float* __restrict__ y) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_out * cout) return;
  const int64_t i = t / cout;
  const int c = (int)(t - i * cout);
  const int32_t L = labels[i];
  float v = L > 0 ? yg[(int64_t)(L - 1) * cout + c] : 0.f;
  y[t] = relu ? fmaxf(v, 0.f) : v;
}

// dyg[g] = dy[rows[g]], zero where ym[rows[g]] <= 0 (ym: the forward output
// through a fused ReLU, or null).
__global__ __launch_bounds__(TB) void k_s2_dy_rows(const int32_t* __restrict__ rows, int64_t ng,
                                                   const float* __restrict__ dy,
                                                   const float* __restrict__ ym, int cout,
                                                   float* __restrict__ dyg) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ng * cout) return;
  const int64_t g = t / cout;
  const int c = (int)(t - g * cout);
  const int64_t src = (int64_t)rows[g] * cout + c;
  const float v = dy[src];
  dyg[t] = (ym && !(ym[src] > 0.f)) ? 0.f : v;
}

// dx[j][c] for input row j = 8h + c' (child c' of group h): the outputs whose
// first child sees j sit at parent offsets p with p_a in {0} when c'_a = 0 and
// {0, 1} when c'_a = 1 (from h's parent), reading j through tap d = c' - 2p.
__global__ __launch_bounds__(TB) void k_s2_col2im(const int32_t* __restrict__ nbr, int64_t n_in,
                                                  const float* __restrict__ dcol, int cin,
                                                  float* __restrict__ dx) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_in * cin) return;
  const int64_t j = t / cin;
  const int ci = (int)(t - j * cin);
  const int32_t* nb = nbr + 27 * (j >> 3);
  const int c = (int)(j & 7);
  const int cx = c >> 2, cy = (c >> 1) & 1, cz = c & 1;
  float acc = 0.f;
  for (int px = 0; px <= cx; ++px)
    for (int py = 0; py <= cy; ++py)
      for (int pz = 0; pz <= cz; ++pz) {
        const int32_t f = nb[(px + 1) * 9 + (py + 1) * 3 + (pz + 1)];
        if (f < 0) continue;
        const int k = ((cx - 2 * px + 1) * 3 + (cy - 2 * py + 1)) * 3 + (cz - 2 * pz + 1);
        acc += dcol[((int64_t)(f >> 3) * 27 + k) * cin + ci];
      }
  dx[t] = acc;
}

__global__ __launch_bounds__(TB) void k_s2_widen(const uint16_t* __restrict__ in, int64_t n,
                                                 float* __restrict__ out) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t < n) out[t] = __uint_as_float((uint32_t)in[t] << 16);
}

inline unsigned grid_for(int64_t n) { return (unsigned)oc::cdiv(n, TB); }

// The profiling events pending for the calling thread (oc_profile_next)
// bracket the whole pass: its kernels and GEMMs.
struct PassEvents {
  hipEvent_t a = nullptr, b = nullptr;
  hipStream_t s;
  explicit PassEvents(hipStream_t st) : s(st) {
    oc::take_profile_events(&a, &b);
    if (a) (void)hipEventRecord(a, s);
  }
  ~PassEvents() {
    if (b) (void)hipEventRecord(b, s);
  }
};

// One GEMM library handle per device, its stream set under a lock at each call.
std::mutex g_blas_mu;
rocblas_handle g_blas[64] = {};

oc_status blas_for(hipStream_t s, rocblas_handle* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64)
    return oc::fail(OC_ERR_DEVICE, "stride-2 convolution: no current device");
  if (!g_blas[dev]) {
    rocblas_handle h = nullptr;
    if (rocblas_create_handle(&h) != rocblas_status_success)
      return oc::fail(OC_ERR_DEVICE, "stride-2 convolution: GEMM library handle unavailable");
    rocblas_set_atomics_mode(h, rocblas_atomics_not_allowed);
    g_blas[dev] = h;
  }
  if (rocblas_set_stream(g_blas[dev], s) != rocblas_status_success)
    return oc::fail(OC_ERR_DEVICE, "stride-2 convolution: GEMM stream not set");
  *out = g_blas[dev];
  return OC_OK;
}

// Column-major GEMM D = op(A) op(B) (+ beta D), fp32 accumulation.
oc_status gemm(hipStream_t s, bool ta, bool tb, int64_t m, int64_t n, int64_t k, const void* A,
               rocblas_datatype at, int64_t lda, const void* B, rocblas_datatype bt, int64_t ldb,
               float beta, float* D, int64_t ldd) {
  if (m == 0 || n == 0) return OC_OK;
  if (m > INT32_MAX || n > INT32_MAX || k > INT32_MAX || lda > INT32_MAX || ldb > INT32_MAX)
    return oc::fail(OC_ERR_UNSUPPORTED, "stride-2 convolution: GEMM size beyond 32 bits");
  std::lock_guard<std::mutex> lk(g_blas_mu);
  rocblas_handle h;
  oc_status st = blas_for(s, &h);
  if (st != OC_OK) return st;
  const float alpha = 1.f;
  const rocblas_status r = rocblas_gemm_ex(
      h, ta ? rocblas_operation_transpose : rocblas_operation_none,
      tb ? rocblas_operation_transpose : rocblas_operation_none, (rocblas_int)m, (rocblas_int)n,
      (rocblas_int)k, &alpha, A, at, (rocblas_int)lda, B, bt, (rocblas_int)ldb, &beta, D,
      rocblas_datatype_f32_r, (rocblas_int)ldd, D, rocblas_datatype_f32_r, (rocblas_int)ldd,
      rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
  if (r != rocblas_status_success)
    return oc::fail(OC_ERR_DEVICE, "stride-2 convolution: GEMM failed (%d)", (int)r);
  return OC_OK;
}

struct S2Shape {
  int64_t G, n_in, n_out;
  int64_t kc;  // 27 cin
  int64_t gc;  // groups per column-buffer chunk
};

S2Shape s2_shape(const oc_octree* t, int l, int cin, size_t elsize) {
  S2Shape h;
  h.G = t->M[l - 1];
  h.n_in = t->N[l];
  h.n_out = t->N[l - 1];
  h.kc = 27 * (int64_t)cin;
  h.gc = std::max<int64_t>(1, std::min<int64_t>(h.G, (int64_t)(COL_CAP / (h.kc * elsize))));
  return h;
}

}  // namespace

namespace oc {

size_t conv_s2_fwd_ws(const oc_octree* t, int l, int cin, int cout, bool bf16) {
  const S2Shape h = s2_shape(t, l, cin, bf16 ? 2 : 4);
  if (h.G == 0) return 0;
  return align256((size_t)h.gc * h.kc * (bf16 ? 2 : 4)) + align256((size_t)h.G * cout * 4);
}

size_t conv_s2_bwd_ws(const oc_octree* t, int l, int cin, int cout, bool bf16, bool dx, bool dw) {
  const S2Shape h = s2_shape(t, l, cin, 4);
  if (h.G == 0 || (!dx && !dw)) return 0;
  size_t b = align256((size_t)h.G * cout * 4);                        // dY_g
  if (bf16) b += align256((size_t)h.kc * cout * 4);                   // widened W
  const size_t a = dx ? align256((size_t)h.G * h.kc * 4) : 0;         // dCol
  const size_t c = dw ? align256((size_t)h.gc * h.kc * 4) : 0;        // Col chunk
  return b + std::max(a, c);
}

oc_status conv_s2_fwd(const oc_octree* t, int l, const void* x, int cin, const void* w, int cout,
                      bool bf16, float* y, int relu, void* ws, hipStream_t s) {
  PassEvents ev(s);
  const S2Shape h = s2_shape(t, l, cin, bf16 ? 2 : 4);
  const int32_t* nbr = t->nbr[l];
  char* p = (char*)ws;
  void* col = p;
  float* yg = (float*)(p + (h.G ? align256((size_t)h.gc * h.kc * (bf16 ? 2 : 4)) : 0));
  const rocblas_datatype dt = bf16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
  for (int64_t g0 = 0; g0 < h.G; g0 += h.gc) {
    const int64_t ng = std::min<int64_t>(h.gc, h.G - g0);
    const int64_t nt = ng * 27 * ((cin + 3) / 4);
    if (bf16)
      hipLaunchKernelGGL((k_s2_col<uint16_t, uint16_t>), dim3(grid_for(nt)), dim3(TB), 0, s, nbr,
                         g0, ng, (const uint16_t*)x, cin, (uint16_t*)col);
    else
      hipLaunchKernelGGL((k_s2_col<float, float>), dim3(grid_for(nt)), dim3(TB), 0, s, nbr, g0, ng,
                         (const float*)x, cin, (float*)col);
    // yg^T [cout][ng] = W^T-view [cout][27 cin] x Col^T-view [27 cin][ng] (column-major)
    oc_status st = gemm(s, false, false, cout, ng, h.kc, w, dt, cout, col, dt, h.kc, 0.f,
                        yg + g0 * cout, cout);
    if (st != OC_OK) return st;
  }
  hipLaunchKernelGGL(k_s2_rows_out, dim3(grid_for(h.n_out * cout)), dim3(TB), 0, s,
                     (const int32_t*)t->labels[l - 1], h.n_out, (const float*)yg, cout, relu, y);
  return OC_OK;
}

oc_status conv_s2_bwd(const oc_octree* t, int l, const void* x, int cin, const void* w, int cout,
                      bool bf16, const float* ym, const float* dy, float* dx, float* dw, void* ws,
                      hipStream_t s) {
  PassEvents ev(s);
  const S2Shape h = s2_shape(t, l, cin, 4);
  const int64_t entries = h.kc * cout;
  if (h.G == 0) {
    if (dx && h.n_in > 0) fill_u32(dx, 0u, h.n_in * cin, s);
    if (dw) fill_u32(dw, 0u, entries, s);
    return OC_OK;
  }
  const int32_t* nbr = t->nbr[l];
  char* p = (char*)ws;
  float* dyg = (float*)p;
  p += align256((size_t)h.G * cout * 4);
  const float* w32 = (const float*)w;
  if (bf16) {
    if (dx) {
      hipLaunchKernelGGL(k_s2_widen, dim3(grid_for(entries)), dim3(TB), 0, s, (const uint16_t*)w,
                         entries, (float*)p);
      w32 = (const float*)p;
    }
    p += align256((size_t)h.kc * cout * 4);
  }
  float* buf = (float*)p;
  hipLaunchKernelGGL(k_s2_dy_rows, dim3(grid_for(h.G * cout)), dim3(TB), 0, s,
                     (const int32_t*)t->rows[l - 1], h.G, dy, ym, cout, dyg);
  if (dx) {
    // dCol^T [27 cin][G] = W-view^T ... : column-major (27 cin x cout) op(A) = A^T of the
    // [cout][27 cin] view of W, times dyg^T-view [cout][G]
    oc_status st = gemm(s, true, false, h.kc, h.G, cout, w32, rocblas_datatype_f32_r, cout, dyg,
                        rocblas_datatype_f32_r, cout, 0.f, buf, h.kc);
    if (st != OC_OK) return st;
    hipLaunchKernelGGL(k_s2_col2im, dim3(grid_for(h.n_in * cin)), dim3(TB), 0, s, nbr, h.n_in,
                       (const float*)buf, cin, dx);
  }
  if (dw) {
    for (int64_t g0 = 0; g0 < h.G; g0 += h.gc) {
      const int64_t ng = std::min<int64_t>(h.gc, h.G - g0);
      const int64_t nt = ng * 27 * ((cin + 3) / 4);
      if (bf16)
        hipLaunchKernelGGL((k_s2_col<uint16_t, float>), dim3(grid_for(nt)), dim3(TB), 0, s, nbr, g0,
                           ng, (const uint16_t*)x, cin, buf);
      else
        hipLaunchKernelGGL((k_s2_col<float, float>), dim3(grid_for(nt)), dim3(TB), 0, s, nbr, g0,
                           ng, (const float*)x, cin, buf);
      // dW^T [cout][27 cin] (+)= dyg^T-view [cout][ng] x Col-view^T [ng][27 cin]
      oc_status st = gemm(s, false, true, cout, h.kc, ng, dyg + g0 * cout, rocblas_datatype_f32_r,
                          cout, buf, rocblas_datatype_f32_r, h.kc, g0 == 0 ? 0.f : 1.f, dw, cout);
      if (st != OC_OK) return st;
    }
  }
  return OC_OK;
}

}  // namespace oc
