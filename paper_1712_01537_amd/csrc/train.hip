// The rest of the O-CNN(d) training iteration around the octree operations
// (Sec. 4 "Network structure", Sec. 5 "Training details"): batch
// normalisation over the octant rows of a depth, the classification head
// (dropout, fully connected layers, softmax cross-entropy) and the SGD update
// with momentum and weight decay.
//
// Batch normalisation in training mode (the method the paper cites, Ioffe
// and Szegedy 2015): per channel, the mean and biased variance over all n
// rows of the feature map.  The statistics are reductions over up to millions
// of rows, done in double precision and in a fixed order: each block sums a
// contiguous range of rows per channel (threads over channels and rows, four
// rows in flight per thread, then the row lanes in order through LDS) into a
// partial, and one block per channel adds the partials (strided over its
// threads, then a fixed tree through LDS).  The block count gives each
// thread about 16 rows, so neither pass waits on a long chain of loads.  The
// variance is a second pass over (x - mean)^2, as the definition states (no
// sum-of-squares cancellation).  Results are reproducible bit for bit.
//
// The head works on a batch of B shapes (B x 1024 x 128 multiply-adds for the
// first FC layer at depth 6): a few microseconds of plain FMA kernels, bound
// by launch latency rather than by arithmetic.
#include <algorithm>

#include "common.h"

namespace {

constexpr int TB = 256;
constexpr int BN_MAX_BLOCKS = 1024;

inline unsigned grid_for(int64_t n) { return (unsigned)oc::cdiv(n, TB); }

// Partial blocks of a reduction over n rows of c channels: about 16 rows per
// thread.
int bn_blocks(int64_t n, int c) {
  return (int)std::max<int64_t>(1, std::min<int64_t>(BN_MAX_BLOCKS, oc::cdiv(n * c, TB * 16)));
}

// Thread layout of the reductions: channel ch = tid % cc of a group of cc
// channels (cc = min(c, 256)), row lane tid / cc of rl = 256 / cc lanes; the
// channel groups are taken in turn.
//
// mode 0: part[b][ch] = sum x over the block's rows
// mode 1: part[b][ch] = sum (x - mean)^2
// mode 2: part[b][2 ch] = sum dy, part[b][2 ch + 1] = sum dy (x - mean) invstd
__global__ __launch_bounds__(TB) void k_bn_partial(const float* __restrict__ x,
                                                   const float* __restrict__ dy, int64_t n, int c,
                                                   int mode, const float* __restrict__ mean,
                                                   const float* __restrict__ invstd,
                                                   double* __restrict__ part) {
  __shared__ double red[2][TB];
  const int tid = threadIdx.x;
  const int nb = gridDim.x, b = blockIdx.x;
  const int64_t r0 = n * b / nb, r1 = n * (b + 1) / nb;
  const int cc = c < TB ? c : TB, rl = TB / cc;
  const int lane_c = tid % cc, lane_r = tid / cc;
  const int outs = mode == 2 ? 2 : 1;
  for (int c0 = 0; c0 < c; c0 += cc) {
    const int ch = c0 + lane_c;
    double s0 = 0.0, s1 = 0.0;
    if (lane_r < rl && ch < c) {
      const double m = mode == 0 ? 0.0 : (double)mean[ch];
      const double is = mode == 2 ? (double)invstd[ch] : 0.0;
#pragma unroll 4
      for (int64_t r = r0 + lane_r; r < r1; r += rl) {
        const double v = (double)x[r * c + ch];
        if (mode == 0) {
          s0 += v;
        } else if (mode == 1) {
          s0 += (v - m) * (v - m);
        } else {
          const double g = (double)dy[r * c + ch];
          s0 += g;
          s1 += g * (v - m) * is;
        }
      }
    }
    red[0][tid] = s0;
    red[1][tid] = s1;
    __syncthreads();
    // lanes of one channel: tid = lane_c + cc * lane_r; add lane_r in order
    if (lane_r == 0 && ch < c) {
      double a0 = 0.0, a1 = 0.0;
      for (int j = 0; j < rl; ++j) {
        a0 += red[0][lane_c + cc * j];
        a1 += red[1][lane_c + cc * j];
      }
      part[((int64_t)b * c + ch) * outs] = a0;
      if (outs == 2) part[((int64_t)b * c + ch) * outs + 1] = a1;
    }
    __syncthreads();
  }
}

// Per channel (one block each), the nb partials: thread t adds partials
// t, t + TB, ... in order, then a fixed tree through LDS.
// mode 0: mean = sum / n.  mode 1: invstd = 1 / sqrt(sum / n + eps).
// mode 2: dbeta = sum dy, dgamma = sum dy x_hat.
__global__ __launch_bounds__(TB) void k_bn_final(const double* __restrict__ part, int nb, int c,
                                                 int64_t n, int mode, float eps,
                                                 float* __restrict__ out0,
                                                 float* __restrict__ out1) {
  __shared__ double red[2][TB];
  const int ch = blockIdx.x, tid = threadIdx.x;
  const int outs = mode == 2 ? 2 : 1;
  double a0 = 0.0, a1 = 0.0;
  for (int b = tid; b < nb; b += TB) {
    a0 += part[((int64_t)b * c + ch) * outs];
    if (outs == 2) a1 += part[((int64_t)b * c + ch) * outs + 1];
  }
  red[0][tid] = a0;
  red[1][tid] = a1;
  __syncthreads();
  for (int h = TB / 2; h > 0; h >>= 1) {
    if (tid < h) {
      red[0][tid] += red[0][tid + h];
      red[1][tid] += red[1][tid + h];
    }
    __syncthreads();
  }
  if (tid != 0) return;
  a0 = red[0][0];
  a1 = red[1][0];
  if (mode == 0) {
    out0[ch] = (float)(a0 / (double)n);
  } else if (mode == 1) {
    out0[ch] = (float)(1.0 / sqrt(a0 / (double)n + (double)eps));
  } else {
    out0[ch] = (float)a0;  // dbeta
    out1[ch] = (float)a1;  // dgamma
  }
}

// y = (x - mean) invstd gamma + beta, ReLU applied when relu.
__global__ __launch_bounds__(TB) void k_bn_apply(const float* __restrict__ x, int64_t n, int c,
                                                 const float* __restrict__ mean,
                                                 const float* __restrict__ invstd,
                                                 const float* __restrict__ gamma,
                                                 const float* __restrict__ beta, int relu,
                                                 float* __restrict__ y) {
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e >= n * c) return;
  const int ch = n * c <= 0xffffffffll ? (int)((uint32_t)e % (uint32_t)c) : (int)(e % c);
  float v = (x[e] - mean[ch]) * invstd[ch] * gamma[ch] + beta[ch];
  y[e] = relu ? fmaxf(v, 0.f) : v;
}

// dx = gamma invstd (dy - dbeta / n - x_hat dgamma / n).
__global__ __launch_bounds__(TB) void k_bn_bwd_apply(const float* __restrict__ x,
                                                     const float* __restrict__ dy, int64_t n,
                                                     int c, const float* __restrict__ mean,
                                                     const float* __restrict__ invstd,
                                                     const float* __restrict__ gamma,
                                                     const float* __restrict__ dgamma,
                                                     const float* __restrict__ dbeta,
                                                     float* __restrict__ dx) {
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e >= n * c) return;
  const int ch = n * c <= 0xffffffffll ? (int)((uint32_t)e % (uint32_t)c) : (int)(e % c);
  const float inv_n = 1.f / (float)n;
  const float xh = (x[e] - mean[ch]) * invstd[ch];
  dx[e] = gamma[ch] * invstd[ch] * (dy[e] - dbeta[ch] * inv_n - xh * dgamma[ch] * inv_n);
}

// y[b][o] = sum_i x[b][i] w[i][o] + bias[o].  Block (b, 16 columns): 16
// lanes over i per column, their partial sums added in lane order.
__global__ __launch_bounds__(TB) void k_fc_fwd(const float* __restrict__ x,
                                               const float* __restrict__ w,
                                               const float* __restrict__ bias, int B, int cin,
                                               int cout, float* __restrict__ y) {
  __shared__ float red[16][17];
  const int b = blockIdx.x, oc = threadIdx.x & 15, lane = threadIdx.x >> 4;
  const int o = blockIdx.y * 16 + oc;
  float a = 0.f;
  if (o < cout)
    for (int i = lane; i < cin; i += 16)
      a = fmaf(x[(int64_t)b * cin + i], w[(int64_t)i * cout + o], a);
  red[lane][oc] = a;
  __syncthreads();
  if (lane == 0 && o < cout) {
    float t = 0.f;
    for (int j = 0; j < 16; ++j) t += red[j][oc];
    y[(int64_t)b * cout + o] = t + (bias ? bias[o] : 0.f);
  }
}

// dx[b][i] = sum_o dy[b][o] w[i][o]
__global__ __launch_bounds__(TB) void k_fc_dx(const float* __restrict__ dy,
                                              const float* __restrict__ w, int B, int cin,
                                              int cout, float* __restrict__ dx) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= (int64_t)B * cin) return;
  const int b = (int)(t / cin), i = (int)(t % cin);
  float a = 0.f;
  for (int o = 0; o < cout; ++o) a = fmaf(dy[(int64_t)b * cout + o], w[(int64_t)i * cout + o], a);
  dx[t] = a;
}

// dw[i][o] = sum_b x[b][i] dy[b][o] (i < cin); db[o] = sum_b dy[b][o] (row i = cin)
__global__ __launch_bounds__(TB) void k_fc_dw(const float* __restrict__ x,
                                              const float* __restrict__ dy, int B, int cin,
                                              int cout, float* __restrict__ dw,
                                              float* __restrict__ db) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= (int64_t)(cin + 1) * cout) return;
  const int i = (int)(t / cout), o = (int)(t % cout);
  float a = 0.f;
  if (i < cin) {
    for (int b = 0; b < B; ++b) a = fmaf(x[(int64_t)b * cin + i], dy[(int64_t)b * cout + o], a);
    dw[t] = a;
  } else if (db) {
    for (int b = 0; b < B; ++b) a += dy[(int64_t)b * cout + o];
    db[o] = a;
  }
}

__global__ __launch_bounds__(TB) void k_dropout(const float* __restrict__ x,
                                                const uint8_t* __restrict__ keep, int64_t n,
                                                float scale, float* __restrict__ y) {
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e < n) y[e] = keep[e] ? x[e] * scale : 0.f;
}

// One wave per row b: lanes over the classes; the row's max, then the sum of
// exp(z - max) (double, combined across lanes by a fixed butterfly), the
// gradient row and the row's loss term.  A second kernel adds the B terms in
// row order.
__global__ __launch_bounds__(64) void k_softmax_rows(const float* __restrict__ z,
                                                     const int32_t* __restrict__ labels, int B,
                                                     int nc, float* __restrict__ dz,
                                                     float* __restrict__ rowloss) {
  const int b = blockIdx.x, t = threadIdx.x;
  const float* zr = z + (int64_t)b * nc;
  float m = -INFINITY;
  for (int j = t; j < nc; j += 64) m = fmaxf(m, zr[j]);
  for (int k = 32; k > 0; k >>= 1) m = fmaxf(m, __shfl_xor(m, k));
  double s = 0.0;
  for (int j = t; j < nc; j += 64) s += exp((double)(zr[j] - m));
  for (int k = 32; k > 0; k >>= 1) s += __shfl_xor(s, k);
  const int lab = labels[b];
  for (int j = t; j < nc; j += 64) {
    const double p = exp((double)(zr[j] - m)) / s;
    dz[(int64_t)b * nc + j] = (float)((p - (j == lab ? 1.0 : 0.0)) / (double)B);
  }
  if (t == 0) rowloss[b] = (float)(log(s) - (double)(zr[lab] - m));
}

__global__ void k_softmax_loss(const float* __restrict__ rowloss, int B, float* __restrict__ loss) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  double a = 0.0;
  for (int b = 0; b < B; ++b) a += (double)rowloss[b];
  *loss = (float)(a / (double)B);
}

__global__ __launch_bounds__(TB) void k_sgd(float* __restrict__ w, const float* __restrict__ g,
                                            float* __restrict__ v, int64_t n, float lr, float mu,
                                            float decay) {
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e >= n) return;
  const float vn = mu * v[e] + lr * (g[e] + decay * w[e]);
  v[e] = vn;
  w[e] -= vn;
}

}  // namespace

extern "C" {

size_t oc_bn_workspace(int64_t n, int32_t c) {
  if (n < 1 || c < 1) return 0;
  return oc::align256((size_t)bn_blocks(n, c) * c * 2 * sizeof(double));
}

oc_status oc_bn_fwd(int64_t n, int32_t c, const float* x, const float* gamma, const float* beta,
                    float eps, int32_t flags, float* y, float* mean, float* invstd, void* ws,
                    size_t ws_bytes, hipStream_t s) {
  if (n < 1 || c < 1 || c > 65536) return oc::fail(OC_ERR_ARG, "oc_bn_fwd: %lld rows x %d channels", (long long)n, c);
  if (!x || !gamma || !beta || !y || !mean || !invstd)
    return oc::fail(OC_ERR_ARG, "oc_bn_fwd: NULL buffer");
  if (!(eps > 0.f)) return oc::fail(OC_ERR_ARG, "oc_bn_fwd: eps must be positive");
  if (!ws || ws_bytes < oc_bn_workspace(n, c))
    return oc::fail(OC_ERR_ARG, "oc_bn_fwd: workspace %zu bytes < %zu", ws ? ws_bytes : 0,
                    oc_bn_workspace(n, c));
  const int nb = bn_blocks(n, c);
  double* part = (double*)ws;
  const unsigned gc = (unsigned)c;
  oc::launch(k_bn_partial, dim3(nb), dim3(TB), 0, s, x, (const float*)nullptr, n, (int)c, 0,
             (const float*)nullptr, (const float*)nullptr, part);
  oc::launch(k_bn_final, dim3(gc), dim3(TB), 0, s, (const double*)part, nb, (int)c, n, 0, eps,
             mean, (float*)nullptr);
  oc::launch(k_bn_partial, dim3(nb), dim3(TB), 0, s, x, (const float*)nullptr, n, (int)c, 1,
             (const float*)mean, (const float*)nullptr, part);
  oc::launch(k_bn_final, dim3(gc), dim3(TB), 0, s, (const double*)part, nb, (int)c, n, 1, eps,
             invstd, (float*)nullptr);
  oc::launch_main(k_bn_apply, dim3(grid_for(n * c)), dim3(TB), s, x, n, (int)c,
                  (const float*)mean, (const float*)invstd, gamma, beta,
                  (flags & OC_FUSE_RELU) ? 1 : 0, y);
  OC_LAUNCH_CHECK();
  return OC_OK;
}

oc_status oc_bn_bwd(int64_t n, int32_t c, const float* x, const float* dy, const float* gamma,
                    const float* mean, const float* invstd, float* dx, float* dgamma,
                    float* dbeta, void* ws, size_t ws_bytes, hipStream_t s) {
  if (n < 1 || c < 1 || c > 65536) return oc::fail(OC_ERR_ARG, "oc_bn_bwd: %lld rows x %d channels", (long long)n, c);
  if (!x || !dy || !gamma || !mean || !invstd || !dx || !dgamma || !dbeta)
    return oc::fail(OC_ERR_ARG, "oc_bn_bwd: NULL buffer");
  if (!ws || ws_bytes < oc_bn_workspace(n, c))
    return oc::fail(OC_ERR_ARG, "oc_bn_bwd: workspace %zu bytes < %zu", ws ? ws_bytes : 0,
                    oc_bn_workspace(n, c));
  const int nb = bn_blocks(n, c);
  double* part = (double*)ws;
  oc::launch(k_bn_partial, dim3(nb), dim3(TB), 0, s, x, dy, n, (int)c, 2, mean, invstd, part);
  oc::launch(k_bn_final, dim3((unsigned)c), dim3(TB), 0, s, (const double*)part, nb,
             (int)c, n, 2, 0.f, dbeta, dgamma);
  oc::launch_main(k_bn_bwd_apply, dim3(grid_for(n * c)), dim3(TB), s, x, dy, n, (int)c, mean,
                  invstd, gamma, (const float*)dgamma, (const float*)dbeta, dx);
  OC_LAUNCH_CHECK();
  return OC_OK;
}

oc_status oc_fc_fwd(int32_t B, int32_t cin, int32_t cout, const float* x, const float* w,
                    const float* bias, float* y, hipStream_t s) {
  if (B < 1 || cin < 1 || cout < 1) return oc::fail(OC_ERR_ARG, "oc_fc_fwd: bad sizes");
  if (!x || !w || !y) return oc::fail(OC_ERR_ARG, "oc_fc_fwd: NULL buffer");
  oc::launch_main(k_fc_fwd, dim3((unsigned)B, (unsigned)oc::cdiv(cout, 16)), dim3(TB), s, x, w,
                  bias, (int)B, (int)cin, (int)cout, y);
  OC_LAUNCH_CHECK();
  return OC_OK;
}

oc_status oc_fc_bwd(int32_t B, int32_t cin, int32_t cout, const float* x, const float* w,
                    const float* dy, float* dx, float* dw, float* dbias, hipStream_t s) {
  if (B < 1 || cin < 1 || cout < 1) return oc::fail(OC_ERR_ARG, "oc_fc_bwd: bad sizes");
  if (!dy || (dx && !w) || (dw && !x)) return oc::fail(OC_ERR_ARG, "oc_fc_bwd: NULL buffer");
  if (dx)
    oc::launch(k_fc_dx, dim3(grid_for((int64_t)B * cin)), dim3(TB), 0, s, dy, w, (int)B, (int)cin,
               (int)cout, dx);
  if (dw || dbias) {
    if (!dw) return oc::fail(OC_ERR_ARG, "oc_fc_bwd: dbias needs dw");
    oc::launch(k_fc_dw, dim3(grid_for((int64_t)(cin + 1) * cout)), dim3(TB), 0, s, x, dy, (int)B,
               (int)cin, (int)cout, dw, dbias);
  }
  OC_LAUNCH_CHECK();
  return OC_OK;
}

oc_status oc_dropout(int64_t n, const float* x, const uint8_t* keep, float p, float* y,
                     hipStream_t s) {
  if (n < 0 || !(p >= 0.f && p < 1.f)) return oc::fail(OC_ERR_ARG, "oc_dropout: bad size or ratio");
  if (n == 0) return OC_OK;
  if (!x || !keep || !y) return oc::fail(OC_ERR_ARG, "oc_dropout: NULL buffer");
  oc::launch(k_dropout, dim3(grid_for(n)), dim3(TB), 0, s, x, keep, n, 1.f / (1.f - p), y);
  OC_LAUNCH_CHECK();
  return OC_OK;
}

size_t oc_softmax_ce_workspace(int32_t B) { return B < 1 ? 0 : oc::align256((size_t)B * 4); }

oc_status oc_softmax_ce(int32_t B, int32_t nc, const float* z, const int32_t* labels, float* loss,
                        float* dz, void* ws, size_t ws_bytes, hipStream_t s) {
  if (B < 1 || nc < 1) return oc::fail(OC_ERR_ARG, "oc_softmax_ce: bad sizes");
  if (!z || !labels || !loss || !dz) return oc::fail(OC_ERR_ARG, "oc_softmax_ce: NULL buffer");
  if (!ws || ws_bytes < oc_softmax_ce_workspace(B))
    return oc::fail(OC_ERR_ARG, "oc_softmax_ce: workspace too small");
  oc::launch_main(k_softmax_rows, dim3((unsigned)B), dim3(64), s, z, labels, (int)B, (int)nc, dz,
                  (float*)ws);
  oc::launch(k_softmax_loss, dim3(1), dim3(64), 0, s, (const float*)ws, (int)B, loss);
  OC_LAUNCH_CHECK();
  return OC_OK;
}

oc_status oc_sgd(int64_t n, float* w, const float* g, float* v, float lr, float momentum,
                 float decay, hipStream_t s) {
  if (n < 0) return oc::fail(OC_ERR_ARG, "oc_sgd: bad size");
  if (n == 0) return OC_OK;
  if (!w || !g || !v) return oc::fail(OC_ERR_ARG, "oc_sgd: NULL buffer");
  oc::launch(k_sgd, dim3(grid_for(n)), dim3(TB), 0, s, w, g, v, n, lr, momentum, decay);
  OC_LAUNCH_CHECK();
  return OC_OK;
}

}  // extern "C"
