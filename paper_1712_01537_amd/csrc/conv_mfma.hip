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
//   MR  16-row blocks per wave (2 MR groups);  NR  16-column blocks per wave;
//   FLIP  false: forward, W[k][c][n] at (k*kk + c)*nn + n;
//         true : input gradient, W'[k][c][n] = W[K3-1-k][n][c].
// Grid: x = ceil(groups / (WAVES*2*MR)), y = ceil(nn / (16*NR)).
template <int K, int V, int MR, int NR, bool FLIP>
__global__ __launch_bounds__(TB) void k_conv_tile(const int32_t* __restrict__ nbr, int64_t ngroups,
                                                  const float* __restrict__ x,
                                                  const float* __restrict__ xmask, int kk,
                                                  const float* __restrict__ w, int nn,
                                                  float* __restrict__ out, int relu) {
  constexpr int R = (K - 1) / 2, S = K + 1, P3 = S * S * S, K3 = K * K * K;
  constexpr int CC = 4 * V;                  // channels per LDS fill
  constexpr int CCP = V == 4 ? CC + 4 : CC;  // padded tile row (floats)
  constexpr int GPW = 2 * MR;                // groups per wave
  constexpr int GPB = GPW * WAVES;           // groups per workgroup
  __shared__ __attribute__((aligned(16))) float tile[GPB * P3 * CCP];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int li = lane & 15, q = lane >> 4;
  const int64_t g0 = (int64_t)blockIdx.x * GPB;
  const int n0 = blockIdx.y * (16 * NR);

  // this lane's output child (row of A) within each of its row blocks
  const int c = li & 7;
  const int cx = c >> 2, cy = (c >> 1) & 1, cz = c & 1;
  int tbase[MR];  // tile row of this lane's child at tap offset -R (all axes)
#pragma unroll
  for (int mr = 0; mr < MR; ++mr) {
    const int gl = wave * GPW + 2 * mr + (li >> 3);
    tbase[mr] = gl * P3 + (cx * S + cy) * S + cz;
  }

  v4f acc[MR][NR];
#pragma unroll
  for (int mr = 0; mr < MR; ++mr)
#pragma unroll
    for (int nr = 0; nr < NR; ++nr) acc[mr][nr] = v4f{0.f, 0.f, 0.f, 0.f};

  for (int c0 = 0; c0 < kk; c0 += CC) {
    __syncthreads();
    // gather the tiles of this channel chunk: one thread per (row, 4 channels)
    constexpr int F4 = CC / 4;
    for (int e = tid; e < GPB * P3 * F4; e += TB) {
      const int row = e / F4, f = e - row * F4;
      const int gl = row / P3, p = row - gl * P3;
      const int64_t g = g0 + gl;
      v4f v = {0.f, 0.f, 0.f, 0.f};
      if (g < ngroups) {
        const int32_t src = tile_src<R>(nbr + 27 * g, p / (S * S), (p / S) % S, p % S);
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
      *reinterpret_cast<v4f*>(&tile[row * CCP + 4 * f]) = v;
    }
    __syncthreads();

    // B operand of tap k: reduction channel c0 + V q + s, column n0 + 16 nr + li
    auto load_b = [&](int k, float (&b)[NR][V]) {
#pragma unroll
      for (int nr = 0; nr < NR; ++nr) {
        const int n = n0 + 16 * nr + li;
#pragma unroll
        for (int s = 0; s < V; ++s) {
          const int ch = c0 + V * q + s;
          float v = 0.f;
          if (n < nn && ch < kk)
            v = FLIP ? w[((int64_t)(K3 - 1 - k) * nn + n) * kk + ch]
                     : w[((int64_t)k * kk + ch) * nn + n];
          b[nr][s] = v;
        }
      }
    };
    float bc[NR][V], bn[NR][V];
    load_b(0, bc);
#pragma unroll 1
    for (int k = 0; k < K3; ++k) {
      if (k + 1 < K3) load_b(k + 1, bn);
      const int dx = k / (K * K), dy = (k / K) % K, dz = k % K;  // tap offset + R
      const int toff = (dx * S + dy) * S + dz;
      float a[MR][V];
#pragma unroll
      for (int mr = 0; mr < MR; ++mr) {
        const float* tp = &tile[(tbase[mr] + toff) * CCP + V * q];
        if constexpr (V == 4) {
          const v4f t = *reinterpret_cast<const v4f*>(tp);
#pragma unroll
          for (int s = 0; s < 4; ++s) a[mr][s] = t[s];
        } else {
          a[mr][0] = tp[0];
        }
      }
#pragma unroll
      for (int s = 0; s < V; ++s)
#pragma unroll
        for (int mr = 0; mr < MR; ++mr)
#pragma unroll
          for (int nr = 0; nr < NR; ++nr) acc[mr][nr] = mfma4(a[mr][s], bc[nr][s], acc[mr][nr]);
#pragma unroll
      for (int nr = 0; nr < NR; ++nr)
#pragma unroll
        for (int s = 0; s < V; ++s) bc[nr][s] = bn[nr][s];
    }
  }

  // epilogue: accumulator j of lane l is row 4(l/16)+j, column l%16
  const int64_t nrows = 8 * ngroups;
#pragma unroll
  for (int mr = 0; mr < MR; ++mr) {
    const int64_t rbase = 8 * (g0 + wave * GPW + 2 * mr) + 4 * q;
#pragma unroll
    for (int nr = 0; nr < NR; ++nr) {
      const int n = n0 + 16 * nr + li;
      if (n >= nn) continue;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t row = rbase + j;
        if (row < nrows) {
          float v = acc[mr][nr][j];
          out[row * nn + n] = relu ? fmaxf(v, 0.f) : v;
        }
      }
    }
  }
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
  int V, MR, NR;
};

TileCfg pick_tile(int K, int kk, int nn) {
  TileCfg c;
  c.V = (K == 3 && kk >= 16) ? 4 : 1;
  c.MR = 1;
  c.NR = nn <= 16 ? 1 : nn <= 32 ? 2 : 4;
  return c;
}

template <int K, int V, int MR, int NR, bool FLIP>
void launch_tile(const oc_octree* t, int l, const float* x, const float* xmask, int kk,
                 const float* w, int nn, float* out, int relu, hipStream_t s) {
  const int64_t G = t->M[l - 1];
  constexpr int GPB = 2 * MR * WAVES;
  dim3 grid((unsigned)oc::cdiv(G, GPB), (unsigned)oc::cdiv(nn, 16 * NR));
  hipLaunchKernelGGL((k_conv_tile<K, V, MR, NR, FLIP>), grid, dim3(TB), 0, s,
                     (const int32_t*)t->nbr[l], G, x, xmask, kk, w, nn, out, relu);
}

template <bool FLIP>
void dispatch_tile(const oc_octree* t, int l, int K, const float* x, const float* xmask, int kk,
                   const float* w, int nn, float* out, int relu, hipStream_t s) {
  const TileCfg c = pick_tile(K, kk, nn);
#define OC_TILE(K_, V_, NR_)                                                     \
  if (K == K_ && c.V == V_ && c.NR == NR_) {                                     \
    launch_tile<K_, V_, 1, NR_, FLIP>(t, l, x, xmask, kk, w, nn, out, relu, s); \
    return;                                                                      \
  }
  OC_TILE(3, 4, 1) OC_TILE(3, 4, 2) OC_TILE(3, 4, 4)
  OC_TILE(3, 1, 1) OC_TILE(3, 1, 2) OC_TILE(3, 1, 4)
  OC_TILE(5, 1, 1) OC_TILE(5, 1, 2) OC_TILE(5, 1, 4)
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

void conv_s1_fwd_f32(const oc_octree* t, int l, int K, const float* x, int cin, const float* w,
                     int cout, float* y, int relu, hipStream_t s) {
  dispatch_tile<false>(t, l, K, x, nullptr, cin, w, cout, y, relu, s);
}

void conv_s1_bwd_data_f32(const oc_octree* t, int l, int K, const float* dy, const float* ymask,
                          int cout, const float* w, int cin, float* dx, hipStream_t s) {
  dispatch_tile<true>(t, l, K, dy, ymask, cout, w, cin, dx, 0, s);
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
