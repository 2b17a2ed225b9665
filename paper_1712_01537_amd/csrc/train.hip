// The rest of the O-CNN(d) training iteration around the octree operations
// (Sec. 4 "Network structure", Sec. 5 "Training details"): batch
// normalisation over the octant rows of a depth, the classification head
// (dropout, fully connected layers, softmax cross-entropy) and the SGD update
// with momentum and weight decay.
//
// Batch normalisation in training mode (the method the paper cites, Ioffe
// and Szegedy 2015): per channel, the mean and biased variance over all n
// rows of the feature map.  The statistics are reductions over up to millions
// of rows, done in double precision and in a fixed order: each block reduces
// a contiguous range of rows per channel (threads over channels and rows,
// four rows in flight per thread, then the row lanes in order through LDS)
// into a partial, and one block per channel combines the partials (strided
// over its threads, then a fixed tree through LDS).  The block count gives
// each thread about 16 rows, so no pass waits on a long chain of loads.  The
// forward takes the mean and the variance in one pass: count, mean and sum
// of squared deviations per partial (Welford's update), combined pairwise
// (Chan et al.), so the variance never subtracts two large sums.  The
// backward's two sums (dy and dy x_hat) are plain sums.  Results are
// reproducible bit for bit.
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
// Backward sums: part[b][2 ch] = sum dy, part[b][2 ch + 1] = sum dy (x - mean)
// invstd over the block's rows.
__global__ __launch_bounds__(TB) void k_bn_partial(const float* __restrict__ x,
                                                   const float* __restrict__ dy, int64_t n, int c,
                                                   const float* __restrict__ mean,
                                                   const float* __restrict__ invstd,
                                                   double* __restrict__ part) {
  __shared__ double red[2][TB];
  const int tid = threadIdx.x;
  const int nb = gridDim.x, b = blockIdx.x;
  const int64_t r0 = n * b / nb, r1 = n * (b + 1) / nb;
  const int cc = c < TB ? c : TB, rl = TB / cc;
  const int lane_c = tid % cc, lane_r = tid / cc;
  for (int c0 = 0; c0 < c; c0 += cc) {
    const int ch = c0 + lane_c;
    double s0 = 0.0, s1 = 0.0;
    if (lane_r < rl && ch < c) {
      const double m = (double)mean[ch], is = (double)invstd[ch];
#pragma unroll 4
      for (int64_t r = r0 + lane_r; r < r1; r += rl) {
        const double v = (double)x[r * c + ch];
        const double g = (double)dy[r * c + ch];
        s0 += g;
        s1 += g * (v - m) * is;
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
      part[((int64_t)b * c + ch) * 2] = a0;
      part[((int64_t)b * c + ch) * 2 + 1] = a1;
    }
    __syncthreads();
  }
}

// Forward statistics in one pass: per (block, channel) the count, mean and
// sum of squared deviations of the block's rows (Welford's update per thread,
// then the row lanes merged in order with Chan et al.'s pairwise formula),
// part[b][ch] = {n, mean, M2}.  The final kernel merges the blocks the same
// way (a fixed order), so the variance never subtracts two large sums.
struct Moments {
  double n, mean, m2;
};
__device__ __forceinline__ Moments merge(const Moments& a, const Moments& b) {
  const double n = a.n + b.n;
  if (n == 0.0) return a;
  const double d = b.mean - a.mean, f = b.n / n;
  return Moments{n, a.mean + d * f, a.m2 + b.m2 + d * d * a.n * f};
}

__global__ __launch_bounds__(TB) void k_bn_stats(const float* __restrict__ x, int64_t n, int c,
                                                 double* __restrict__ part) {
  __shared__ double red[3][TB];
  const int tid = threadIdx.x;
  const int nb = gridDim.x, b = blockIdx.x;
  const int64_t r0 = n * b / nb, r1 = n * (b + 1) / nb;
  const int cc = c < TB ? c : TB, rl = TB / cc;
  const int lane_c = tid % cc, lane_r = tid / cc;
  for (int c0 = 0; c0 < c; c0 += cc) {
    const int ch = c0 + lane_c;
    Moments m{0.0, 0.0, 0.0};
    if (lane_r < rl && ch < c) {
#pragma unroll 4
      for (int64_t r = r0 + lane_r; r < r1; r += rl) {
        const double v = (double)x[r * c + ch];
        m.n += 1.0;
        const double d = v - m.mean;
        m.mean += d / m.n;
        m.m2 += d * (v - m.mean);
      }
    }
    red[0][tid] = m.n;
    red[1][tid] = m.mean;
    red[2][tid] = m.m2;
    __syncthreads();
    if (lane_r == 0 && ch < c) {
      Moments a{0.0, 0.0, 0.0};
      for (int j = 0; j < rl; ++j) {
        const int k = lane_c + cc * j;
        a = merge(a, Moments{red[0][k], red[1][k], red[2][k]});
      }
      double* o = part + ((int64_t)b * c + ch) * 3;
      o[0] = a.n;
      o[1] = a.mean;
      o[2] = a.m2;
    }
    __syncthreads();
  }
}

// Per channel (one block each): mean and invstd = 1 / sqrt(M2 / n + eps)
// from the nb partials of k_bn_stats (thread t merges partials t, t + TB,
// ... in order, then a fixed tree through LDS).
__global__ __launch_bounds__(TB) void k_bn_stats_final(const double* __restrict__ part, int nb,
                                                       int c, float eps, float* __restrict__ mean,
                                                       float* __restrict__ invstd) {
  __shared__ double red[3][TB];
  const int ch = blockIdx.x, tid = threadIdx.x;
  Moments a{0.0, 0.0, 0.0};
  for (int b = tid; b < nb; b += TB) {
    const double* p = part + ((int64_t)b * c + ch) * 3;
    a = merge(a, Moments{p[0], p[1], p[2]});
  }
  red[0][tid] = a.n;
  red[1][tid] = a.mean;
  red[2][tid] = a.m2;
  __syncthreads();
  for (int h = TB / 2; h > 0; h >>= 1) {
    if (tid < h) {
      const Moments m = merge(Moments{red[0][tid], red[1][tid], red[2][tid]},
                              Moments{red[0][tid + h], red[1][tid + h], red[2][tid + h]});
      red[0][tid] = m.n;
      red[1][tid] = m.mean;
      red[2][tid] = m.m2;
    }
    __syncthreads();
  }
  if (tid != 0) return;
  mean[ch] = (float)red[1][0];
  invstd[ch] = (float)(1.0 / sqrt(red[2][0] / red[0][0] + (double)eps));
}

// Per channel (one block each), the nb backward partials: thread t adds
// partials t, t + TB, ... in order, then a fixed tree through LDS; dbeta =
// sum dy, dgamma = sum dy x_hat.
__global__ __launch_bounds__(TB) void k_bn_final(const double* __restrict__ part, int nb, int c,
                                                 float* __restrict__ dbeta,
                                                 float* __restrict__ dgamma) {
  __shared__ double red[2][TB];
  const int ch = blockIdx.x, tid = threadIdx.x;
  double a0 = 0.0, a1 = 0.0;
  for (int b = tid; b < nb; b += TB) {
    a0 += part[((int64_t)b * c + ch) * 2];
    a1 += part[((int64_t)b * c + ch) * 2 + 1];
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
  dbeta[ch] = (float)red[0][0];
  dgamma[ch] = (float)red[1][0];
}

// The normalised value of x in channel ch (ReLU'd when relu): one
// definition for the plain and the pooled forward.
__device__ __forceinline__ float bn_value(float x, int ch, const float* __restrict__ mean,
                                          const float* __restrict__ invstd,
                                          const float* __restrict__ gamma,
                                          const float* __restrict__ beta, int relu) {
  const float v = (x - mean[ch]) * invstd[ch] * gamma[ch] + beta[ch];
  return relu ? fmaxf(v, 0.f) : v;
}

// Normalisation (and ReLU) with the 2x2x2 max-pool: one thread per
// (depth-(l-1) row i, channel); the children of label L = g + 1 are rows
// 8g .. 8g + 7 of x, the first maximum in child order wins (strict '>'),
// empty parents get 0 and no switch.  The normalised depth-l values are not
// stored.
__global__ __launch_bounds__(TB) void k_bn_pool(const float* __restrict__ x,
                                                const int32_t* __restrict__ labels, int64_t npar,
                                                int c, const float* __restrict__ mean,
                                                const float* __restrict__ invstd,
                                                const float* __restrict__ gamma,
                                                const float* __restrict__ beta, int relu,
                                                float* __restrict__ y, uint8_t* __restrict__ sw) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= npar * c) return;
  const int64_t i = t / c;
  const int ch = (int)(t - i * c);
  const int32_t L = labels[i];
  if (L == 0) {
    y[t] = 0.f;
    return;
  }
  const int64_t g = L - 1;
  const float* src = x + 8 * g * c + ch;
  float best = bn_value(src[0], ch, mean, invstd, gamma, beta, relu);
  uint8_t arg = 0;
#pragma unroll
  for (int k = 1; k < 8; ++k) {
    const float v = bn_value(src[(int64_t)k * c], ch, mean, invstd, gamma, beta, relu);
    if (v > best) {
      best = v;
      arg = (uint8_t)k;
    }
  }
  y[t] = best;
  sw[g * c + ch] = arg;
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
  y[e] = bn_value(x[e], ch, mean, invstd, gamma, beta, relu);
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

// Mean and invstd of x [n][c] (two launches).
void bn_stats(int64_t n, int c, const float* x, float eps, float* mean, float* invstd,
              double* part, hipStream_t s) {
  const int nb = bn_blocks(n, c);
  oc::launch(k_bn_stats, dim3(nb), dim3(TB), 0, s, x, n, c, part);
  oc::launch(k_bn_stats_final, dim3((unsigned)c), dim3(TB), 0, s, (const double*)part, nb, c, eps,
             mean, invstd);
}

}  // namespace

extern "C" {

size_t oc_bn_workspace(int64_t n, int32_t c) {
  if (n < 1 || c < 1) return 0;
  return oc::align256((size_t)bn_blocks(n, c) * c * 3 * sizeof(double));
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
  bn_stats(n, c, x, eps, mean, invstd, (double*)ws, s);
  oc::launch_main(k_bn_apply, dim3(grid_for(n * c)), dim3(TB), s, x, n, (int)c,
                  (const float*)mean, (const float*)invstd, gamma, beta,
                  (flags & OC_FUSE_RELU) ? 1 : 0, y);
  OC_LAUNCH_CHECK();
  return OC_OK;
}

oc_status oc_bn_pool_fwd(const oc_octree* t, int32_t l, int32_t c, const float* z,
                         const float* gamma, const float* beta, float eps, int32_t flags, float* y,
                         uint8_t* sw, float* mean, float* invstd, void* ws, size_t ws_bytes,
                         hipStream_t s) {
  oc_status st = oc::check_tree_level(t, l, 1);
  if (st != OC_OK) return st;
  if (c < 1 || c > 65536) return oc::fail(OC_ERR_ARG, "oc_bn_pool_fwd: %d channels", c);
  const int64_t n = t->N[l], np = t->N[l - 1];
  if (np == 0) return OC_OK;
  if (!y || !gamma || !beta || !mean || !invstd || (n > 0 && (!z || !sw)))
    return oc::fail(OC_ERR_ARG, "oc_bn_pool_fwd: NULL buffer");
  if (!(eps > 0.f)) return oc::fail(OC_ERR_ARG, "oc_bn_pool_fwd: eps must be positive");
  if (n == 0) return oc::fail(OC_ERR_ARG, "oc_bn_pool_fwd: depth %d has no octant", l);
  if (!ws || ws_bytes < oc_bn_workspace(n, c))
    return oc::fail(OC_ERR_ARG, "oc_bn_pool_fwd: workspace %zu bytes < %zu", ws ? ws_bytes : 0,
                    oc_bn_workspace(n, c));
  bn_stats(n, c, z, eps, mean, invstd, (double*)ws, s);
  oc::launch_main(k_bn_pool, dim3(grid_for(np * c)), dim3(TB), s, z,
                  (const int32_t*)t->labels[l - 1], np, (int)c, (const float*)mean,
                  (const float*)invstd, gamma, beta, (flags & OC_FUSE_RELU) ? 1 : 0, y, sw);
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
  oc::launch(k_bn_partial, dim3(nb), dim3(TB), 0, s, x, dy, n, (int)c, mean, invstd, part);
  oc::launch(k_bn_final, dim3((unsigned)c), dim3(TB), 0, s, (const double*)part, nb, (int)c, dbeta,
             dgamma);
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
