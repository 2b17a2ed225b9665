// bf16 octree convolution, stride 1, on the matrix cores
// (v_mfma_f32_16x16x32_bf16: products of bf16 values, fp32 accumulation).
//
// Forward and input gradient (k_conv_bf), the unrolled convolution of
// Sec. 3.2 as an implicit GEMM over sibling groups:
//   out[i][n] = sum_k sum_c x[nb(i,k)][c] W'[k][c][n]
// with W' = W (forward), or W'[k][c][n] = W[K^3-1-k][n][c] and x = dY for the
// input gradient (for stride 1, j is i's neighbour at offset d iff i is j's
// neighbour at -d).  A workgroup takes 8 sibling groups (64 output rows).  The
// eight children of a group read, for every tap, positions of the (K+1)^3
// block around the group (the union neighbourhood of Fig. 4); the block is
// streamed through LDS one x-slab at a time (all channels of a position are
// one 128-byte row, so every gather is whole cache lines).  The taps are
// taken in K phases, one per x-offset dx; phase dx reads the slabs dx+R and
// dx+R+1 (children with x-bit 0 and 1), so a ring of three slab buffers lets
// the slab of the next phase land while the current one is multiplied.
// Eight waves split each phase's (tap, 32-channel half) steps; a wave keeps
// the step's weights (32 channels x 64 output columns) in registers and
// multiplies them with the four 16-row blocks of the tile, so one 16-byte
// LDS read feeds four MFMAs.  The waves' partial tiles are added through LDS
// in a fixed order at the end.
//
// Weight gradient (k_conv_bf_dw):
//   dW[k][c][n] = sum_g sum_j x[pos(g, j, k)][c] dY[8g + j][n]
// is a GEMM with M = input channels, N = output channels and the octants as
// the reduction.  The MFMA wants eight consecutive octants of one channel
// per lane; the transposing LDS load ds_read_b64_tr_b16 gives exactly that
// from row-major tiles (lane i of a 16-lane group receives element i % 4 of
// the 8-byte rows read by lanes 4r + i / 4, r = 0..3), so the staged x
// positions and dY rows keep the layout of HBM.  A workgroup owns the taps
// of one x-offset and two (K = 5) or three (K = 3) y-offsets for every input
// channel block,
// the waves split those (tap, channel block) pairs and keep their dW blocks
// in registers, and the workgroup streams a range of sibling groups, four
// per step.  Ranges write partial sums that a second kernel adds in a fixed
// order, so results do not depend on scheduling.
//
// LDS layouts place the 16-byte pieces (8 channels) of a position or row at
// piece index o ^ f(position): the eight children of a group (forward), or
// the four rows of a transposing load (weight gradient), then fall on
// distinct banks.
#include "conv_bf16.h"

#include <algorithm>

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) void* lptr_t;

constexpr int TB = 256;

__device__ __forceinline__ uint32_t lds_addr(const void* lds) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lptr_t)lds);
}
// Direct global->LDS load of 16 bytes per lane: lane i's bytes land at LDS
// byte address lds + 16 i (lds uniform over the wave).  Inline assembly, so
// the compiler's wait counting stays exact for the code around it; the
// caller waits for completion (vm_wait0) before other waves read the data.
__device__ __forceinline__ void lds_load16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(src)
               : "memory", "m0");
}
// s_waitcnt vmcnt(0): all of this wave's vector memory operations are done.
__device__ __forceinline__ void vm_wait0() { __builtin_amdgcn_s_waitcnt(0x0F70); }

__device__ __forceinline__ v4f mfma_bf(v4u a, v4u b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a),
                                                  __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
}

// Transposing LDS load at byte offset off of the LDS array base.
__device__ __forceinline__ v4s lds_tr16(const void* base, int off) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)((lds_char*)base + off));
}
__device__ __forceinline__ v4u join(v4s lo, v4s hi) {
  const uint64_t a = __builtin_bit_cast(uint64_t, lo), b = __builtin_bit_cast(uint64_t, hi);
  return v4u{(uint32_t)a, (uint32_t)(a >> 32), (uint32_t)b, (uint32_t)(b >> 32)};
}

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint32_t f2bf(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u) return (u >> 16) | ((u & 0xffffu) ? 0x40u : 0u);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// Neighbour row of tile position (px, py, pz) of group g (positions are
// offsets +R from the group's first child, per axis in [0, K]), or -1.
template <int R>
__device__ __forceinline__ int32_t tile_row(const int32_t* __restrict__ nbr, int64_t g, int px,
                                            int py, int pz) {
  const int ux = px - R, uy = py - R, uz = pz - R;
  const int32_t b = nbr[27 * g + ((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1)];
  return b < 0 ? -1 : b + 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1);
}

// ---------------------------------------------------------------------------
// Weights in MFMA order: wp[o][t][n][e] = W'[t][8o + e][n] for reduction
// channel octet o, tap t, output channel n (16 bytes per (o, t, n)).
// flip: W'[t][c][n] = W[K3-1-t][n][c] (input gradient; kk = cout, nn = cin).
__global__ __launch_bounds__(TB) void k_bf_wprep(const uint16_t* __restrict__ w, int K3, int kk,
                                                 int nn, int flip, uint16_t* __restrict__ wp) {
  const int64_t i = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (i >= (int64_t)kk * K3 * nn) return;
  const int e = (int)(i & 7);
  int64_t r = i >> 3;
  const int n = (int)(r % nn);
  r /= nn;
  const int t = (int)(r % K3), o = (int)(r / K3);
  const int c = 8 * o + e;
  wp[i] = flip ? w[((int64_t)(K3 - 1 - t) * nn + n) * kk + c] : w[((int64_t)t * kk + c) * nn + n];
}

// out[e] = bf16(ym ? (ym[e] > 0 ? in[e] : 0) : in[e]), four entries per thread.
__global__ __launch_bounds__(TB) void k_bf_cvt(const float* __restrict__ in,
                                               const float* __restrict__ ym, int64_t n, int vec,
                                               uint16_t* __restrict__ out) {
  const int64_t e = 4 * ((int64_t)blockIdx.x * TB + threadIdx.x);
  if (e >= n) return;
  if (vec && e + 4 <= n) {
    float4 v = *reinterpret_cast<const float4*>(in + e);
    if (ym) {
      const float4 y = *reinterpret_cast<const float4*>(ym + e);
      v = float4{y.x > 0.f ? v.x : 0.f, y.y > 0.f ? v.y : 0.f, y.z > 0.f ? v.z : 0.f,
                 y.w > 0.f ? v.w : 0.f};
    }
    *reinterpret_cast<uint2*>(out + e) =
        uint2{f2bf(v.x) | (f2bf(v.y) << 16), f2bf(v.z) | (f2bf(v.w) << 16)};
  } else {
    for (int64_t i = e; i < n && i < e + 4; ++i)
      out[i] = (uint16_t)f2bf(ym && !(ym[i] > 0.f) ? 0.f : in[i]);
  }
}

// out[e] = sum_{r < nparts} part[r][e] in the order r = 0, 1, ... (n % 4 == 0).
__global__ __launch_bounds__(TB) void k_bf_sum(const float* __restrict__ part, int nparts,
                                               int64_t n, float* __restrict__ out) {
  const int64_t e = 4 * ((int64_t)blockIdx.x * TB + threadIdx.x);
  if (e >= n) return;
  v4f s = {0.f, 0.f, 0.f, 0.f};
  for (int r = 0; r < nparts; ++r) s += *reinterpret_cast<const v4f*>(part + r * n + e);
  *reinterpret_cast<v4f*>(out + e) = s;
}

// ---------------------------------------------------------------------------
// Forward / input gradient.  x [8 ngroups][kk] bf16 (kk % 8 == 0), wp as
// produced by k_bf_wprep, out [8 ngroups][nn] fp32 (nn % 16 == 0).
// Grid: x = tiles of 8 groups, y = blocks of 64 output channels; 512 threads.
// Slab j of channel chunk c (64 channels) is global slab G = c S + j and
// lives in ring buffer G % 3: 8 groups x S^2 positions x 8 pieces, piece o
// of position (j, py, pz) at o ^ ((j&1) << 2 | (py&1) << 1 | (pz&1)).
// FLIP only names the pass (the weights decide what is computed).
template <int K, bool FLIP>
__global__ __launch_bounds__(512) void k_conv_bf(const int32_t* __restrict__ nbr, int64_t ngroups,
                                                  const uint16_t* __restrict__ x, int kk,
                                                  const uint16_t* __restrict__ wp, int nn,
                                                  float* __restrict__ out, int relu) {
  constexpr int R = (K - 1) / 2, S = K + 1, S2 = S * S, K2 = K * K, K3 = K2 * K;
  constexpr int GT = 8, NW = 8;
  constexpr int SLAB = GT * S2 * 8;  // 16-byte pieces of one slab buffer
  constexpr int RS = 68;             // floats per row of a reduction slot
  constexpr int RED = NW * 32 * RS;  // floats of one reduction round
  constexpr int NV = (3 * SLAB * 16 > RED * 4 ? 3 * SLAB * 16 : RED * 4) / 16;
  __shared__ __attribute__((aligned(16))) v4u lds[NV];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, q = lane >> 4;
  const int64_t g0 = (int64_t)blockIdx.x * GT;
  const int n0 = blockIdx.y * 64;
  const int KO = kk >> 3;           // channel octets of the reduction
  const int nch = (KO + 7) >> 3;    // chunks of 64 channels

  auto stage = [&](int G) {
    const int c = G / S, j = G - c * S;
    v4u* buf = lds + (G % 3) * SLAB;
    for (int i = wave; i < S2; i += NW) {  // 64 pieces = 8 positions per instruction
      const int s = i * 64 + lane;
      const int pos = s >> 3, g = pos / S2, p = pos - g * S2;
      const int py = p / S, pz = p - py * S;
      const int o = (s & 7) ^ (((j & 1) << 2) | ((py & 1) << 1) | (pz & 1));
      const int oc = 8 * c + o;
      const int64_t gg = g0 + g;
      const int32_t row = gg < ngroups && oc < KO ? tile_row<R>(nbr, gg, j, py, pz) : -1;
      v4u* dst = buf + i * 64;
      if (row >= 0)
        lds_load16(x + (int64_t)row * kk + 8 * oc, lds_addr(dst));
      else
        dst[lane] = v4u{0u, 0u, 0u, 0u};
    }
  };

  // lane (li, q) of row block b supplies row li: child li & 7 of group
  // 2b + (li >> 3), channels 8q..8q+7 of the step's 32
  const int cc = li & 7, cx = cc >> 2, cy = (cc >> 1) & 1, cz = cc & 1, gl = li >> 3;
  auto halves = [&](int c) { return KO - 8 * c > 4 ? 2 : 1; };
  // step e of phase ph (x-offset ph - R) of chunk c: tap (ph, e / hc), half e % hc
  auto load_w = [&](v4u (&wv)[4], int c, int ph, int e) {
    const int hc = halves(c);
    const int tap2 = e / hc, h = e - tap2 * hc;
    const int t = ph * K2 + tap2;
    const int o = 8 * c + 4 * h + q;
#pragma unroll
    for (int nf = 0; nf < 4; ++nf) {
      const int n = n0 + 16 * nf + li;
      wv[nf] = (n < nn && o < KO)
                   ? *reinterpret_cast<const v4u*>(wp + ((int64_t)(o * K3 + t) * nn + n) * 8)
                   : v4u{0u, 0u, 0u, 0u};
    }
  };
  v4f acc[4][4];
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int nf = 0; nf < 4; ++nf) acc[b][nf] = v4f{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const v4u (&wv)[4], int c, int ph, int e) {
    const int hc = halves(c);
    const int tap2 = e / hc, h = e - tap2 * hc;
    const int dyi = tap2 / K, dzi = tap2 - dyi * K;
    const int px = ph + cx, py = dyi + cy, pz = dzi + cz;
    const v4u* buf = lds + ((c * S + px) % 3) * SLAB;
    const int f = ((px & 1) << 2) | ((py & 1) << 1) | (pz & 1);
    const int base = (py * S + pz) * 8 + ((4 * h + q) ^ f);
    v4u a[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) a[b] = buf[(2 * b + gl) * S2 * 8 + base];
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int nf = 0; nf < 4; ++nf) acc[b][nf] = mfma_bf(a[b], wv[nf], acc[b][nf]);
  };
  // the first step of the phase after (c, ph), if any
  auto load_next_phase = [&](v4u (&wv)[4], int c, int ph) {
    if (ph + 1 < K)
      load_w(wv, c, ph + 1, wave);
    else if (c + 1 < nch)
      load_w(wv, c + 1, 0, wave);
  };

  v4u wa[4], wb[4];
  stage(0);
  stage(1);
  load_w(wa, 0, 0, wave);
  for (int c = 0; c < nch; ++c) {
    const int ne = halves(c) * K2;  // steps per phase (> NW)
    for (int ph = 0; ph < K; ++ph) {
      vm_wait0();
      __syncthreads();  // slabs ph and ph+1 have landed; phase ph-1 is done
      if (ph + 2 < S)
        stage(c * S + ph + 2);
      else if (c + 1 < nch)
        stage((c + 1) * S);
      int e = wave;
      for (; e + NW < ne; e += 2 * NW) {
        load_w(wb, c, ph, e + NW);
        compute(wa, c, ph, e);
        if (e + 2 * NW < ne)
          load_w(wa, c, ph, e + 2 * NW);
        else
          load_next_phase(wa, c, ph);
        compute(wb, c, ph, e + NW);
      }
      if (e < ne) {
        load_next_phase(wb, c, ph);
        compute(wa, c, ph, e);
#pragma unroll
        for (int nf = 0; nf < 4; ++nf) wa[nf] = wb[nf];
      }
    }
    if (c + 1 < nch) {
      __syncthreads();  // slab (c, K-1) is no longer read
      stage((c + 1) * S + 1);
    }
  }

  // add the waves' tiles in wave order, 32 rows per round
  __syncthreads();
  float* red = reinterpret_cast<float*>(lds);
  const int64_t nrows = 8 * ngroups;
#pragma unroll
  for (int rd = 0; rd < 2; ++rd) {
#pragma unroll
    for (int bb = 0; bb < 2; ++bb)
#pragma unroll
      for (int nf = 0; nf < 4; ++nf)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          red[(wave * 32 + bb * 16 + 4 * q + j) * RS + 16 * nf + li] = acc[2 * rd + bb][nf][j];
    __syncthreads();
    const int r = tid >> 4, cq = (tid & 15) * 4;
    v4f s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < NW; ++w) s += *reinterpret_cast<const v4f*>(&red[(w * 32 + r) * RS + cq]);
    const int64_t row = 8 * g0 + 32 * rd + r;
    const int n = n0 + cq;
    if (row < nrows && n < nn) {
      if (relu) {
#pragma unroll
        for (int j = 0; j < 4; ++j) s[j] = fmaxf(s[j], 0.f);
      }
      *reinterpret_cast<v4f*>(out + row * nn + n) = s;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Weight gradient.  x [8 ngroups][cin] bf16, dy [8 ngroups][cout] bf16
// (cin, cout % 16 == 0).  Grid: x = units x ranges (unit = x-offset and a
// set of up to three y-offsets, range = a contiguous run of groups), y =
// blocks of 64 output channels, z = blocks of 64 input channels; 256 threads.
// A unit takes the y-offsets [ya, yb) (at most 2 for K = 5, 3 for K = 3).
// Per step of four groups the workgroup stages the x positions its taps read
// (x-slabs dx+R, dx+R+1; y in [ya, yb]; every z) and the 32 dY rows.  x
// piece o of box position (ix, iy, iz) sits at o ^ 2((iz + 2 iy) & 3), dY
// piece o of row r at o ^ 2(r & 3).  part [ranges][K^3][cin][cout].
template <int K, int MAXC>
__global__ __launch_bounds__(TB, 1) void k_conv_bf_dw(const int32_t* __restrict__ nbr,
                                                      int64_t ngroups,
                                                      const uint16_t* __restrict__ x, int cin,
                                                      const uint16_t* __restrict__ dy, int cout,
                                                      int nranges, float* __restrict__ part) {
  constexpr int R = (K - 1) / 2, S = K + 1, K3 = K * K * K;
  constexpr int YR = K == 5 ? 2 : 3;            // y-offsets per unit
  constexpr int NSET = (K + YR - 1) / YR;       // units per x-offset
  constexpr int MAXPOS = 2 * (YR + 1) * S;      // staged positions per group
  constexpr int XP = 4 * MAXPOS * 8;     // pieces of the staged x (four groups)
  constexpr int YP = 32 * 8;             // pieces of the staged dY rows
  constexpr int BUF = XP + YP;
  __shared__ __attribute__((aligned(16))) v4u lds[2 * BUF];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, q = lane >> 4;
  const int unit = blockIdx.x % (K * NSET), range = blockIdx.x / (K * NSET);
  const int dxi = unit / NSET, set = unit % NSET;
  const int ya = YR * set, yb = ya + YR < K ? ya + YR : K;
  const int NY = yb - ya + 1;
  const int npos = 2 * NY * S;
  const int ntap = (yb - ya) * K;
  const int c0 = blockIdx.z * 64, n0 = blockIdx.y * 64;
  const int CB = (cin - c0 < 64 ? cin - c0 : 64) / 16;
  const int ncombo = ntap * CB;
  const int64_t gbeg = ngroups * range / nranges, gend = ngroups * (range + 1) / nranges;
  const int nsteps = (int)((gend - gbeg + 3) / 4);

  auto stage = [&](int st, v4u* buf) {
    const int64_t gs = gbeg + 4 * (int64_t)st;
    const int nxi = npos / 2;  // instructions of 64 pieces for the x positions
    for (int i = wave; i < nxi + 4; i += 4) {
      if (i < nxi) {
        const int s = i * 64 + lane;
        const int pos = s >> 3, g = pos / npos, p = pos - g * npos;
        const int ix = p / (NY * S), rem = p - ix * (NY * S), iy = rem / S, iz = rem - iy * S;
        const int o = (s & 7) ^ (2 * ((iz + 2 * iy) & 3));
        const int ch = c0 + 8 * o;
        const int64_t gg = gs + g;
        const int32_t row = gg < gend && ch < cin ? tile_row<R>(nbr, gg, dxi + ix, ya + iy, iz) : -1;
        v4u* dst = buf + i * 64;
        if (row >= 0)
          lds_load16(x + (int64_t)row * cin + ch, lds_addr(dst));
        else
          dst[lane] = v4u{0u, 0u, 0u, 0u};
      } else {
        const int s = (i - nxi) * 64 + lane;
        const int rl = s >> 3;
        const int o = (s & 7) ^ (2 * (rl & 3));
        const int co = n0 + 8 * o;
        const int64_t gg = gs + (rl >> 3);
        v4u* dst = buf + XP + (i - nxi) * 64;
        if (gg < gend && co < cout)
          lds_load16(dy + (8 * gg + (rl & 7)) * cout + co, lds_addr(dst));
        else
          dst[lane] = v4u{0u, 0u, 0u, 0u};
      }
    }
  };

  v4f acc[MAXC][4];
#pragma unroll
  for (int m = 0; m < MAXC; ++m)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[m][nb] = v4f{0.f, 0.f, 0.f, 0.f};

  // transposing loads: source lane li reads row 4h + (li >> 2) of its
  // 16-lane group's eight, channels 4 (li & 3).. of the 16-channel block
  const int r4 = li >> 2, tq = li & 3;
  auto compute = [&](const v4u* buf) {
    v4u bfr[4];
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      v4s hv[2];
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int rl = 8 * q + 4 * hh + r4;
        const int o = 2 * nb + (tq >> 1);
        hv[hh] = lds_tr16(buf, (XP + rl * 8 + (o ^ (2 * (rl & 3)))) * 16 + (tq & 1) * 8);
      }
      bfr[nb] = join(hv[0], hv[1]);
    }
#pragma unroll
    for (int mi = 0; mi < MAXC; ++mi) {
      const int m = wave + 4 * mi;
      if (m < ncombo) {
        const int it = m / CB, cb = m - it * CB;
        const int dyl = it / K, dzi = it - dyl * K;
        v4s hv[2];
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {  // child 4 hh + r4 of group q
          const int iy = dyl + (r4 >> 1), iz = dzi + (r4 & 1);
          const int p = (hh * NY + iy) * S + iz;
          const int o = 2 * cb + (tq >> 1);
          hv[hh] = lds_tr16(buf, ((q * npos + p) * 8 + (o ^ (2 * ((iz + 2 * iy) & 3)))) * 16 +
                                     (tq & 1) * 8);
        }
        const v4u a = join(hv[0], hv[1]);
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) acc[mi][nb] = mfma_bf(a, bfr[nb], acc[mi][nb]);
      }
    }
  };

  if (nsteps > 0) stage(0, lds);
  for (int st = 0; st < nsteps; ++st) {
    vm_wait0();
    __syncthreads();  // step st has landed; step st-1 is no longer read
    if (st + 1 < nsteps) stage(st + 1, lds + ((st + 1) & 1) * BUF);
    compute(lds + (st & 1) * BUF);
  }

  // partial dW of this range: lane (li, q), accumulator j holds input channel
  // c0 + 16 cb + 4q + j, output channel n0 + 16 nb + li
#pragma unroll
  for (int mi = 0; mi < MAXC; ++mi) {
    const int m = wave + 4 * mi;
    if (m < ncombo) {
      const int it = m / CB, cb = m - it * CB;
      const int t = (dxi * K + ya + it / K) * K + it % K;
      float* dst = part + ((int64_t)range * K3 + t) * cin * cout;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int n = n0 + 16 * nb + li;
        if (n < cout) {
#pragma unroll
          for (int j = 0; j < 4; ++j) dst[(int64_t)(c0 + 16 * cb + 4 * q + j) * cout + n] = acc[mi][nb][j];
        }
      }
    }
  }
}

inline unsigned blocks(int64_t n, int per) { return (unsigned)oc::cdiv(n, per); }

size_t wp_bytes(int K, int kk, int nn) { return oc::align256((size_t)kk * K * K * K * nn * 2); }

int dw_units(int K) { return K == 5 ? 5 * 3 : 3; }  // x-offsets x sets of y-offsets

int dw_ranges(const oc_octree* t, int l, int K, int cin, int cout) {
  const int64_t G = t->M[l - 1];
  const int per = dw_units(K) * (int)oc::cdiv(cout, 64) * (int)oc::cdiv(cin, 64);
  int64_t r = oc::cdiv(2 * (int64_t)oc::cu_count(), per);
  r = std::min<int64_t>(r, std::max<int64_t>(1, oc::cdiv(G, 16)));  // 16+ groups per range
  return (int)std::max<int64_t>(1, r);
}

void wprep(const uint16_t* w, int K, int kk, int nn, int flip, uint16_t* wp, hipStream_t s) {
  const int K3 = K * K * K;
  hipLaunchKernelGGL(k_bf_wprep, dim3(blocks((int64_t)kk * K3 * nn, TB)), dim3(TB), 0, s, w, K3,
                     kk, nn, flip, wp);
}

template <bool FLIP>
void launch_conv(const oc_octree* t, int l, int K, const uint16_t* x, int kk, const uint16_t* wp,
                 int nn, float* out, int relu, hipStream_t s) {
  const int64_t G = t->M[l - 1];
  const dim3 grid(blocks(G, 8), blocks(nn, 64));
  if (K == 5)
    oc::launch_main(k_conv_bf<5, FLIP>, grid, dim3(512), s, (const int32_t*)t->nbr[l], G, x, kk,
                    wp, nn, out, relu);
  else
    oc::launch_main(k_conv_bf<3, FLIP>, grid, dim3(512), s, (const int32_t*)t->nbr[l], G, x, kk,
                    wp, nn, out, relu);
}

}  // namespace

namespace oc {

bool conv_bf16_supported(int K, int cin, int cout) {
  return (K == 3 || K == 5) && cin % 16 == 0 && cout % 16 == 0;
}

void conv_bf16_kernel_name(int K, int pass, char* buf, size_t n) {
  if (pass == 2)
    snprintf(buf, n, "k_conv_bf_dw<%d, %d>", K, K == 5 ? 10 : 9);
  else
    snprintf(buf, n, "k_conv_bf<%d, %s>", K, pass == 1 ? "true" : "false");
}

size_t conv_bf16_fwd_ws(int K, int cin, int cout) { return wp_bytes(K, cin, cout); }

size_t conv_bf16_bwd_ws(const oc_octree* t, int l, int K, int cin, int cout) {
  const size_t dy16 = align256((size_t)t->N[l] * cout * 2);
  const size_t part =
      align256((size_t)dw_ranges(t, l, K, cin, cout) * K * K * K * cin * cout * sizeof(float));
  return dy16 + wp_bytes(K, cout, cin) + part;
}

void conv_bf16_fwd(const oc_octree* t, int l, int K, const uint16_t* x, int cin,
                   const uint16_t* w, int cout, float* y, int relu, void* ws, hipStream_t s) {
  uint16_t* wp = (uint16_t*)ws;
  wprep(w, K, cin, cout, 0, wp, s);
  launch_conv<false>(t, l, K, x, cin, wp, cout, y, relu, s);
}

void conv_bf16_bwd(const oc_octree* t, int l, int K, const uint16_t* x, int cin,
                   const uint16_t* w, int cout, const float* ym, const float* dy, float* dx,
                   float* dw, void* ws, hipStream_t s) {
  const int64_t N = t->N[l], G = t->M[l - 1];
  char* p = (char*)ws;
  uint16_t* dy16 = (uint16_t*)p;
  p += align256((size_t)N * cout * 2);
  uint16_t* wpf = (uint16_t*)p;
  p += wp_bytes(K, cout, cin);
  float* part = (float*)p;
  const int64_t n = N * cout;
  const int vec = (uintptr_t)dy % 16 == 0 && (!ym || (uintptr_t)ym % 16 == 0);
  hipLaunchKernelGGL(k_bf_cvt, dim3(blocks(n, 4 * TB)), dim3(TB), 0, s, dy, ym, n, vec, dy16);
  if (dx) {
    wprep(w, K, cout, cin, 1, wpf, s);
    launch_conv<true>(t, l, K, dy16, cout, wpf, cin, dx, 0, s);
  }
  if (dw) {
    const int K3 = K * K * K;
    const int nr = dw_ranges(t, l, K, cin, cout);
    const dim3 grid((unsigned)(dw_units(K) * nr), blocks(cout, 64), blocks(cin, 64));
    if (K == 5)
      launch_main(k_conv_bf_dw<5, 10>, grid, dim3(TB), s, (const int32_t*)t->nbr[l], G, x, cin,
                  dy16, cout, nr, part);
    else
      launch_main(k_conv_bf_dw<3, 9>, grid, dim3(TB), s, (const int32_t*)t->nbr[l], G, x, cin,
                  dy16, cout, nr, part);
    const int64_t E = (int64_t)K3 * cin * cout;
    hipLaunchKernelGGL(k_bf_sum, dim3(blocks(E, 4 * TB)), dim3(TB), 0, s, part, nr, E, dw);
  }
}

}  // namespace oc
