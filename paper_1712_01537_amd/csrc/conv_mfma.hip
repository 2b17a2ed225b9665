// fp32 octree convolution on the matrix cores (v_mfma_f32_16x16x4_f32).
//
// Stride-1 forward and input gradient share one implicit-GEMM kernel that
// works on sibling groups.  The eight children of a group sit at the corners
// of a 2x2x2 block; every tap of every child reads a position of the
// (K+1)^3 block around it (Sec. 3.2, Fig. 4: the siblings share one union
// neighbourhood).  A workgroup gathers that dense (K+1)^3 x channel tile of
// each of its groups into LDS once per channel chunk (rows of absent
// neighbours are zero), and the tap loop then reads fixed tile positions:
// output child c, tap d reads tile position c + d + r, with no indirection.
//
//   forward      out[i][n] = sum_k sum_c x[nb(i,k)][c] W[k][c][n]
//   input grad   the same with x = dY (optionally masked by [y > 0]) and
//                W'[k][c][n] = W[K^3-1-k][n][c]: for stride 1 the
//                neighbour relation is symmetric under d -> -d.
//
// MFMA operand layout (16x16x4, fp32): lane l supplies A[l%16][l/16] and
// B[l/16][l%16] and receives D[4(l/16)+j][l%16] in accumulator j.  Rows of
// A are 16 output octants (two sibling groups), columns of B 16 output
// channels.  With V = 4, lane group q supplies reduction channels 4q..4q+3
// of a 16-channel block to four consecutive MFMAs (channel 4q+s to the s-th),
// so one 16-byte LDS read per lane feeds four MFMAs.
//
// The weight gradient dW[k][c][n] = sum_i x[nb(i,k)][c] dY[i][n] is a GEMM
// with M = (tap, channel) pairs, N = output channels and the octants as the
// reduction.  Each wave owns an MT x NT block tile of dW and streams a chunk
// of sibling groups (four octants per MFMA step), gathering its A values
// straight from global memory: a 16-lane slice reads 16 consecutive channels
// of one row.  Chunks write partial sums that a second kernel adds in a fixed
// order, so results do not depend on scheduling.
#include "conv_mfma.h"

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int TB = 256;
constexpr int WAVES = TB / 64;

__device__ __forceinline__ v4f mfma4(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Row at depth l of tile position (px,py,pz) of a group whose 27-entry
// parent-neighbour row is nb, or -1.  Positions are offsets +R from the
// group's first child, per axis in [-R, 1+R].
template <int R>
__device__ __forceinline__ int32_t tile_src(const int32_t* __restrict__ nb, int px, int py,
                                            int pz) {
  const int ux = px - R, uy = py - R, uz = pz - R;
  const int32_t base = nb[((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1)];
  return base < 0 ? -1 : base + 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1);
}

// ---------------------------------------------------------------------------
// Stride-1 implicit GEMM over group tiles.
//   K   kernel size (3 or 5);  V  channels per lane per LDS read (1 or 4);
//   MR, NR  16-row / 16-column MFMA blocks per wave;  WM  waves along rows
//   (WAVES / WM along columns);  FLIP  false: forward, W[k][c][n] at
//   (k*kk + c)*nn + n;  true: input gradient, W'[k][c][n] = W[K3-1-k][n][c].
// A workgroup computes BM = 16 WM MR rows (BM / 8 sibling groups) by
// BN = 16 (WAVES/WM) NR columns.  Per chunk of CC reduction channels it
// gathers the groups' (K+1)^3 tiles into LDS, then walks the taps in slabs
// of TSL taps, staging each slab's weights as Bt[tap][n][c] so that a lane
// reads its V channels with one LDS load.  Group tiles are stored with two
// padding rows per x-slab and rows of RS = CC + 4 floats, which puts the
// eight children of a group (and 16 consecutive weight columns) on distinct
// LDS banks.
// Grid: x = ceil(groups / (BM/8)), y = ceil(nn / BN), z = splits of the
// reduction channels, cps chunks each.  With one split the result (ReLU
// applied if relu) goes to out; otherwise split z writes its partial sum to
// part[z][row][n] and k_sum_split finishes.
template <int K, int V, int MR, int NR, int WM, bool FLIP>
__global__ __launch_bounds__(TB) void k_conv_tile(const int32_t* __restrict__ nbr, int64_t ngroups,
                                                  const float* __restrict__ x,
                                                  const float* __restrict__ xmask, int kk,
                                                  const float* __restrict__ w, int nn,
                                                  float* __restrict__ out, int relu, int cps,
                                                  float* __restrict__ part) {
  constexpr int WN = WAVES / WM;
  constexpr int R = (K - 1) / 2, S = K + 1, K2 = K * K, K3 = K2 * K, S3 = S * S * S;
  constexpr int PX = S * S + 2;  // tile rows per x-slab (two padding rows)
  constexpr int P3 = S * PX;     // tile rows per group
  constexpr int CC = 4 * V;
  constexpr int RS = V == 4 ? CC + 4 : CC;
  constexpr int BM = WM * MR * 16, BN = WN * NR * 16, GPB = BM / 8;
  constexpr int TSL = (V == 1 && K == 3) ? K3 : K2;  // taps per weight slab
  __shared__ __attribute__((aligned(16))) float At[GPB * P3 * RS];
  __shared__ __attribute__((aligned(16))) float Bt[TSL * BN * RS];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int li = lane & 15, q = lane >> 4;
  const int wm = wave % WM, wn = wave / WM;
  const int64_t g0 = (int64_t)blockIdx.x * GPB;
  const int n0 = blockIdx.y * BN;
  const int cb = blockIdx.z * cps * CC;
  const int ce = cb + cps * CC < kk ? cb + cps * CC : kk;

  const int c = li & 7;
  const int cx = c >> 2, cy = (c >> 1) & 1, cz = c & 1;
  int tbase[MR];  // tile row of this lane's child at tap offset -R on every axis
#pragma unroll
  for (int mr = 0; mr < MR; ++mr)
    tbase[mr] = ((wm * MR + mr) * 2 + (li >> 3)) * P3 + cx * PX + cy * S + cz;
  int bcol[NR];  // this lane's column within the workgroup's BN
#pragma unroll
  for (int nr = 0; nr < NR; ++nr) bcol[nr] = (wn * NR + nr) * 16 + li;

  v4f acc[MR][NR];
#pragma unroll
  for (int mr = 0; mr < MR; ++mr)
#pragma unroll
    for (int nr = 0; nr < NR; ++nr) acc[mr][nr] = v4f{0.f, 0.f, 0.f, 0.f};

  for (int c0 = cb; c0 < ce; c0 += CC) {
    __syncthreads();
    // gather the group tiles of this channel chunk: one thread per (position, 4 channels)
    constexpr int F4 = CC / 4;
    for (int e = tid; e < GPB * S3 * F4; e += TB) {
      const int rp = e / F4, f = e - rp * F4;
      const int gl = rp / S3, p = rp - gl * S3;
      const int px = p / (S * S), py = (p / S) % S, pz = p % S;
      const int64_t g = g0 + gl;
      v4f v = {0.f, 0.f, 0.f, 0.f};
      if (g < ngroups) {
        const int32_t src = tile_src<R>(nbr + 27 * g, px, py, pz);
        if (src >= 0) {
          const int ch = c0 + 4 * f;
          const float* xr = x + (int64_t)src * kk;
          if (ch + 4 <= kk && (kk & 3) == 0) {
            v = *reinterpret_cast<const v4f*>(xr + ch);
            if (xmask) {
              const v4f m = *reinterpret_cast<const v4f*>(xmask + (int64_t)src * kk + ch);
#pragma unroll
              for (int j = 0; j < 4; ++j) v[j] = m[j] > 0.f ? v[j] : 0.f;
            }
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j)
              if (ch + j < kk) {
                float a = xr[ch + j];
                if (xmask && !(xmask[(int64_t)src * kk + ch + j] > 0.f)) a = 0.f;
                v[j] = a;
              }
          }
        }
      }
      *reinterpret_cast<v4f*>(&At[(gl * P3 + px * PX + py * S + pz) * RS + 4 * f]) = v;
    }

    for (int k0 = 0; k0 < K3; k0 += TSL) {
      if (k0 > 0) __syncthreads();  // previous slab consumed
      // stage the weights of taps k0 .. k0+TSL-1 as Bt[t][n][c]
      if constexpr (FLIP) {
        for (int e = tid; e < TSL * BN * F4; e += TB) {
          const int f = e % F4, tn = e / F4, n = tn % BN, t = tn / BN;
          const int gn = n0 + n, ch = c0 + 4 * f;
          v4f v = {0.f, 0.f, 0.f, 0.f};
          if (gn < nn) {
            const float* wr = w + ((int64_t)(K3 - 1 - (k0 + t)) * nn + gn) * kk;
            if (ch + 4 <= kk && (kk & 3) == 0) {
              v = *reinterpret_cast<const v4f*>(wr + ch);
            } else {
#pragma unroll
              for (int j = 0; j < 4; ++j)
                if (ch + j < kk) v[j] = wr[ch + j];
            }
          }
          *reinterpret_cast<v4f*>(&Bt[(t * BN + n) * RS + 4 * f]) = v;
        }
      } else {
        for (int e = tid; e < TSL * CC * BN; e += TB) {
          const int n = e % BN, tc = e / BN, cc = tc % CC, t = tc / CC;
          const int gn = n0 + n, ch = c0 + cc;
          float v = 0.f;
          if (gn < nn && ch < kk) v = w[((int64_t)(k0 + t) * kk + ch) * nn + gn];
          Bt[(t * BN + n) * RS + cc] = v;
        }
      }
      __syncthreads();

#pragma unroll 3
      for (int t = 0; t < TSL; ++t) {
        const int k = k0 + t;
        const int toff = (k / K2) * PX + ((k / K) % K) * S + k % K;
        float a[MR][V], b[NR][V];
#pragma unroll
        for (int mr = 0; mr < MR; ++mr) {
          const float* tp = &At[(tbase[mr] + toff) * RS + V * q];
          if constexpr (V == 4) {
            const v4f u = *reinterpret_cast<const v4f*>(tp);
#pragma unroll
            for (int j = 0; j < 4; ++j) a[mr][j] = u[j];
          } else {
            a[mr][0] = tp[0];
          }
        }
#pragma unroll
        for (int nr = 0; nr < NR; ++nr) {
          const float* bp = &Bt[(t * BN + bcol[nr]) * RS + V * q];
          if constexpr (V == 4) {
            const v4f u = *reinterpret_cast<const v4f*>(bp);
#pragma unroll
            for (int j = 0; j < 4; ++j) b[nr][j] = u[j];
          } else {
            b[nr][0] = bp[0];
          }
        }
#pragma unroll
        for (int j = 0; j < V; ++j)
#pragma unroll
          for (int mr = 0; mr < MR; ++mr)
#pragma unroll
            for (int nr = 0; nr < NR; ++nr) acc[mr][nr] = mfma4(a[mr][j], b[nr][j], acc[mr][nr]);
      }
    }
  }

  // epilogue: accumulator j of lane l is row 4(l/16)+j, column l%16
  const int64_t nrows = 8 * ngroups;
  const bool split = gridDim.z > 1;
  float* dst = split ? part + (int64_t)blockIdx.z * nrows * nn : out;
#pragma unroll
  for (int mr = 0; mr < MR; ++mr) {
    const int64_t rbase = 8 * g0 + (wm * MR + mr) * 16 + 4 * q;
#pragma unroll
    for (int nr = 0; nr < NR; ++nr) {
      const int n = n0 + bcol[nr];
      if (n >= nn) continue;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t row = rbase + j;
        if (row < nrows) {
          const float v = acc[mr][nr][j];
          dst[row * nn + n] = (!split && relu) ? fmaxf(v, 0.f) : v;
        }
      }
    }
  }
}

// out[e] = sum over splits of part[z][e] (in split order), ReLU if relu.
__global__ __launch_bounds__(TB) void k_sum_split(const float* __restrict__ part, int splits,
                                                  int64_t n, float* __restrict__ out, int relu) {
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e >= n) return;
  float s = 0.f;
  for (int z = 0; z < splits; ++z) s += part[(int64_t)z * n + e];
  out[e] = relu ? fmaxf(s, 0.f) : s;
}

// ---------------------------------------------------------------------------
// Weight gradient partial sums, stride 1.
//   Tile: MT blocks of 16 (tap, channel) pairs x NT blocks of 16 output
//   channels, one per workgroup (grid y).  Grid x: chunks of gchunk groups;
//   wave w of the workgroup takes groups gb + w, gb + w + WAVES, ... and the
//   four waves' sums are added through LDS in wave order before the chunk's
//   partial is written: part[chunk][(k*cin + c)*cout + n].
template <int K, int MT, int NT>
__global__ __launch_bounds__(TB) void k_conv_dw(const int32_t* __restrict__ nbr, int64_t ngroups,
                                                int64_t gchunk, const float* __restrict__ x,
                                                int cin, const float* __restrict__ dy,
                                                const float* __restrict__ ymask, int cout,
                                                float* __restrict__ part) {
  constexpr int R = (K - 1) / 2, K3 = K * K * K;
  constexpr int NACC = MT * NT * 4;
  __shared__ float red[(WAVES - 1) * NACC * 64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int li = lane & 15, q = lane >> 4;
  const int mtot = K3 * cin;
  const int tiles_m = (mtot + 16 * MT - 1) / (16 * MT);
  const int tm = blockIdx.y % tiles_m, tn = blockIdx.y / tiles_m;

  // this lane's (tap, channel) pair in each M block
  int ach[MT], aox[MT], aoy[MT], aoz[MT];
  bool aval[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int m = (tm * MT + mt) * 16 + li;
    aval[mt] = m < mtot;
    const int k = aval[mt] ? m / cin : 0;
    ach[mt] = aval[mt] ? m - k * cin : 0;
    aox[mt] = k / (K * K);  // tap offset + R per axis
    aoy[mt] = (k / K) % K;
    aoz[mt] = k % K;
  }
  int bcol[NT];
#pragma unroll
  for (int nt = 0; nt < NT; ++nt) bcol[nt] = (tn * NT + nt) * 16 + li;

  v4f acc[MT][NT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = v4f{0.f, 0.f, 0.f, 0.f};

  const int64_t gb = (int64_t)blockIdx.x * gchunk;
  const int64_t ge = gb + gchunk < ngroups ? gb + gchunk : ngroups;
  for (int64_t g = gb + wave; g < ge; g += WAVES) {
    const int32_t* nb = nbr + 27 * g;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = 4 * h + q;  // this lane's octant of the reduction step
      const int cx = c >> 2, cy = (c >> 1) & 1, cz = c & 1;
      float a[MT], b[NT];
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        float v = 0.f;
        if (aval[mt]) {
          const int32_t src = tile_src<R>(nb, cx + aox[mt], cy + aoy[mt], cz + aoz[mt]);
          if (src >= 0) v = x[(int64_t)src * cin + ach[mt]];
        }
        a[mt] = v;
      }
      const int64_t orow = 8 * g + c;
#pragma unroll
      for (int nt = 0; nt < NT; ++nt) {
        float v = 0.f;
        if (bcol[nt] < cout) {
          const int64_t idx = orow * cout + bcol[nt];
          v = dy[idx];
          if (ymask && !(ymask[idx] > 0.f)) v = 0.f;
        }
        b[nt] = v;
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) acc[mt][nt] = mfma4(a[mt], b[nt], acc[mt][nt]);
    }
  }

  // wave-ordered sum of the four waves' tiles
  if (wave > 0) {
    float* r = red + (wave - 1) * NACC * 64;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int j = 0; j < 4; ++j) r[((mt * NT + nt) * 4 + j) * 64 + lane] = acc[mt][nt][j];
  }
  __syncthreads();
  if (wave != 0) return;
  float* pp = part + (int64_t)blockIdx.x * ((int64_t)mtot * cout);
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
      const int n = bcol[nt];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float v = acc[mt][nt][j];
#pragma unroll
        for (int w = 0; w < WAVES - 1; ++w) v += red[(w * NACC + (mt * NT + nt) * 4 + j) * 64 + lane];
        const int m = (tm * MT + mt) * 16 + 4 * q + j;
        if (n < cout && m < mtot) pp[(int64_t)m * cout + n] = v;
      }
    }
}

// Fixed-order sum of the chunk partials.
__global__ __launch_bounds__(TB) void k_sum_parts(const float* __restrict__ part, int nparts,
                                                  int64_t entries, float* __restrict__ out) {
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e >= entries) return;
  float s = 0.f;
  for (int p = 0; p < nparts; ++p) s += part[(int64_t)p * entries + e];
  out[e] = s;
}

// ---------------------------------------------------------------------------
// Launch-shape selection.

struct TileCfg {
  int V, MR, NR, WM, splits, cps;
};

// Workgroup tile and split of the reduction for a stride-1 layer of G groups.
TileCfg pick_tile(int K, int64_t G, int kk, int nn) {
  TileCfg c;
  c.V = (K == 3 && kk >= 16) ? 4 : 1;
  if (nn <= 16) {
    c.WM = 4, c.MR = 1, c.NR = 1;  // 64 x 16
  } else if (nn <= 32) {
    c.WM = 2, c.MR = 2, c.NR = 1;  // 64 x 32
  } else {
    c.WM = 2, c.MR = 2, c.NR = 2;  // 64 x 64
  }
  const int BM = 16 * c.WM * c.MR, BN = 16 * (WAVES / c.WM) * c.NR;
  const int64_t tiles = oc::cdiv(G, BM / 8) * oc::cdiv(nn, BN);
  const int chunks = (int)oc::cdiv(kk, 4 * c.V);
  int splits = 1;
  while (tiles * splits < 512 && splits * 2 <= chunks) splits *= 2;
  c.cps = (int)oc::cdiv(chunks, splits);
  c.splits = (int)oc::cdiv(chunks, c.cps);
  return c;
}

template <int K, int V, int MR, int NR, int WM, bool FLIP>
void launch_tile(const oc_octree* t, int l, const TileCfg& c, const float* x, const float* xmask,
                 int kk, const float* w, int nn, float* out, int relu, float* part,
                 hipStream_t s) {
  const int64_t G = t->M[l - 1];
  constexpr int BM = 16 * WM * MR, BN = 16 * (WAVES / WM) * NR;
  dim3 grid((unsigned)oc::cdiv(G, BM / 8), (unsigned)oc::cdiv(nn, BN), (unsigned)c.splits);
  hipLaunchKernelGGL((k_conv_tile<K, V, MR, NR, WM, FLIP>), grid, dim3(TB), 0, s,
                     (const int32_t*)t->nbr[l], G, x, xmask, kk, w, nn, out, relu, c.cps, part);
  if (c.splits > 1) {
    const int64_t n = t->N[l] * (int64_t)nn;
    hipLaunchKernelGGL(k_sum_split, dim3((unsigned)oc::cdiv(n, TB)), dim3(TB), 0, s,
                       (const float*)part, c.splits, n, out, relu);
  }
}

template <bool FLIP>
void dispatch_tile(const oc_octree* t, int l, int K, const float* x, const float* xmask, int kk,
                   const float* w, int nn, float* out, int relu, float* part, hipStream_t s) {
  const TileCfg c = pick_tile(K, t->M[l - 1], kk, nn);
#define OC_TILE(K_, V_, MR_, NR_, WM_)                                                     \
  if (K == K_ && c.V == V_ && c.MR == MR_ && c.NR == NR_ && c.WM == WM_) {                 \
    launch_tile<K_, V_, MR_, NR_, WM_, FLIP>(t, l, c, x, xmask, kk, w, nn, out, relu, part, s); \
    return;                                                                                \
  }
  OC_TILE(3, 4, 1, 1, 4) OC_TILE(3, 4, 2, 1, 2) OC_TILE(3, 4, 2, 2, 2)
  OC_TILE(3, 1, 1, 1, 4) OC_TILE(3, 1, 2, 1, 2) OC_TILE(3, 1, 2, 2, 2)
  OC_TILE(5, 1, 1, 1, 4) OC_TILE(5, 1, 2, 1, 2) OC_TILE(5, 1, 2, 2, 2)
#undef OC_TILE
}

struct DwCfg {
  int MT, NT, tiles;
  int64_t gchunk, nchunks;
};

DwCfg pick_dw(int K, int64_t G, int cin, int cout) {
  DwCfg c;
  const int64_t entries = (int64_t)K * K * K * cin * cout;
  const int mblocks = (int)oc::cdiv((int64_t)K * K * K * cin, 16);
  const int nblocks = (int)oc::cdiv(cout, 16);
  c.NT = nblocks >= 4 ? 4 : nblocks >= 2 ? 2 : 1;
  c.MT = mblocks >= 4 ? 4 : 2;
  c.tiles = (int)(oc::cdiv(mblocks, c.MT) * oc::cdiv(nblocks, c.NT));
  // about 512 workgroups, partial sums capped at 4M floats
  int64_t chunks = std::max<int64_t>(1, oc::cdiv(512, c.tiles));
  chunks = std::min<int64_t>(chunks, std::max<int64_t>(1, (int64_t(4) << 20) / entries));
  c.gchunk = std::max<int64_t>(WAVES, oc::cdiv(std::max<int64_t>(G, 1), chunks));
  c.nchunks = std::max<int64_t>(1, oc::cdiv(G, c.gchunk));
  return c;
}

template <int K, int MT, int NT>
void launch_dw(const oc_octree* t, int l, const DwCfg& c, const float* x, int cin,
               const float* dy, const float* ym, int cout, float* part, hipStream_t s) {
  dim3 grid((unsigned)c.nchunks, (unsigned)c.tiles);
  hipLaunchKernelGGL((k_conv_dw<K, MT, NT>), grid, dim3(TB), 0, s, (const int32_t*)t->nbr[l],
                     t->M[l - 1], c.gchunk, x, cin, dy, ym, cout, part);
}

}  // namespace

namespace oc {

size_t conv_s1_tile_ws(const oc_octree* t, int l, int K, int kk, int nn) {
  const TileCfg c = pick_tile(K, t->M[l - 1], kk, nn);
  return c.splits > 1 ? (size_t)c.splits * t->N[l] * nn * sizeof(float) : 0;
}

void conv_s1_fwd_f32(const oc_octree* t, int l, int K, const float* x, int cin, const float* w,
                     int cout, float* y, int relu, float* ws, hipStream_t s) {
  dispatch_tile<false>(t, l, K, x, nullptr, cin, w, cout, y, relu, ws, s);
}

void conv_s1_bwd_data_f32(const oc_octree* t, int l, int K, const float* dy, const float* ymask,
                          int cout, const float* w, int cin, float* dx, float* ws, hipStream_t s) {
  dispatch_tile<true>(t, l, K, dy, ymask, cout, w, cin, dx, 0, ws, s);
}

size_t conv_s1_dw_parts(const oc_octree* t, int l, int K, int cin, int cout) {
  const DwCfg c = pick_dw(K, t->M[l - 1], cin, cout);
  return (size_t)c.nchunks;
}

void conv_s1_bwd_weight_f32(const oc_octree* t, int l, int K, const float* x, int cin,
                            const float* dy, const float* ymask, int cout, float* dw, float* part,
                            hipStream_t s) {
  const DwCfg c = pick_dw(K, t->M[l - 1], cin, cout);
#define OC_DW(K_, MT_, NT_)                                                \
  if (K == K_ && c.MT == MT_ && c.NT == NT_) {                             \
    launch_dw<K_, MT_, NT_>(t, l, c, x, cin, dy, ymask, cout, part, s);    \
  } else
  OC_DW(3, 2, 1) OC_DW(3, 2, 2) OC_DW(3, 2, 4) OC_DW(3, 4, 1) OC_DW(3, 4, 2) OC_DW(3, 4, 4)
  OC_DW(5, 2, 1) OC_DW(5, 2, 2) OC_DW(5, 2, 4) OC_DW(5, 4, 1) OC_DW(5, 4, 2) OC_DW(5, 4, 4) {}
#undef OC_DW
  const int64_t entries = (int64_t)K * K * K * cin * cout;
  hipLaunchKernelGGL(k_sum_parts, dim3((unsigned)oc::cdiv(entries, TB)), dim3(TB), 0, s,
                     (const float*)part, (int)c.nchunks, entries, dw);
}

}  // namespace oc
