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
//   input grad   the same with x = dY and W'[k][c][n] = W[K^3-1-k][n][c]:
//                for stride 1 the neighbour relation is symmetric under
//                d -> -d.
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
#include "pool_fuse.h"

#include "conv_cin.h"

#include <algorithm>
#include <cmath>
#include <type_traits>

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int TB = 256;
constexpr int WAVES = TB / 64;

typedef __attribute__((address_space(3))) void* lptr_t;  // LDS

// Direct global->LDS load of 16 bytes per lane: lane i's bytes land at LDS
// byte address lds + 16 i (lds uniform over the wave).  Written as inline
// assembly so that the compiler's wait insertion, which does not know the
// instruction, keeps exact LDS counters for the surrounding code; the caller
// waits for completion itself (vm_wait0) before other waves read the data.
// LDS byte address of a wave-uniform LDS pointer, in a scalar register.
__device__ __forceinline__ uint32_t lds_addr(const void* lds) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lptr_t)lds);
}
__device__ __forceinline__ void lds_load16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(src)
               : "memory", "m0");
}
// The same for 12 bytes per lane (the lane stride in LDS stays 16 bytes).
__device__ __forceinline__ void lds_load12(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx3 %1, off" ::"s"(lds), "v"(src)
               : "memory", "m0");
}
// A 16x16 MFMA result held as D[4(l/16)+j][l%16] in lane l (j = 0..3) is
// handed over so that lane l holds D[4(l%4)+j][l/4]: with rows l%16 of the
// result as output rows, consecutive lanes then store consecutive 16 bytes.
__device__ __forceinline__ v4f store_order(v4f d, int lane) {
  const int src = (((lane & 3) << 4) + (lane >> 2)) << 2;  // byte lane index
  v4f r;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    r[j] = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(d[j])));
  return r;
}

// s_waitcnt vmcnt(0): all of this wave's vector memory operations are done.
__device__ __forceinline__ void vm_wait0() { __builtin_amdgcn_s_waitcnt(0x0F70); }

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
// Workgroups are persistent over a contiguous range of row tiles.  The loads
// of the next step (the next weight slab; at the end of a chunk also the next
// chunk's or the next tile's group tiles) are issued before each step's
// MFMAs, the neighbour entries a whole tile ahead.  Every prefetch writes the
// same registers on one straight-line path: addresses are clamped to valid
// memory and out-of-range elements are zeroed when the registers are stored
// to LDS, so no load result is copied (and waited for) before the MFMAs.
// VEC: kk and nn are multiples of 4, so rows of x and W are read as float4.
// Grid: x = persistent workgroups, y = ceil(nn / BN), z = splits of the
// reduction channels, cps chunks each.  With one split the result (ReLU
// applied if relu) goes to out; otherwise split z writes its partial sum to
// part[z][row][n] and k_sum_split finishes.
template <int K, int V, int MR, int NR, int WM, bool FLIP, bool VEC>
__global__ __launch_bounds__(TB) void k_conv_tile(const int32_t* __restrict__ nbr, int64_t ngroups,
                                                  const float* __restrict__ x, int kk,
                                                  const float* __restrict__ w, int nn,
                                                  float* __restrict__ out, int relu, int cps,
                                                  float* __restrict__ part) {
  constexpr int WN = WAVES / WM;
  constexpr int R = (K - 1) / 2, S = K + 1, K2 = K * K, K3 = K2 * K, S3 = S * S * S;
  constexpr int PX = S * S + 2;  // tile rows per x-slab (two padding rows)
  constexpr int P3 = S * PX;     // tile rows per group
  constexpr int CC = 4 * V;
  constexpr int F4 = CC / 4;
  constexpr int RS = V == 4 ? CC + 4 : CC;
  constexpr int BM = WM * MR * 16, BN = WN * NR * 16, GPB = BM / 8;
  constexpr int TSL = (V == 1 && K == 3) ? K3 : K2;  // taps per weight slab
  constexpr int NSL = K3 / TSL;                     // slabs per channel chunk
  // Staging of the next step's global loads in registers.  Tile: each pass
  // covers GPP groups, thread -> fixed (group of the pass, position, channel
  // quad); NA passes.  Weight slab: (tap, column, channel quad) elements,
  // float4 along the contiguous axis of W; NB passes.
  constexpr int GPP = TB / (S3 * F4) > 0 ? TB / (S3 * F4) : 1;
  constexpr int NA = GPB / GPP;
  constexpr int NB = (TSL * BN * F4 + TB - 1) / TB;
  static_assert(S3 * F4 <= TB && GPB % GPP == 0, "tile staging must cover every position");
  static_assert(NA <= 32 && NB <= 32, "validity bits fit a word");
  __shared__ __attribute__((aligned(16))) float At[GPB * P3 * RS];
  __shared__ __attribute__((aligned(16))) float Bt[TSL * BN * RS];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int li = lane & 15, q = lane >> 4;
  const int wm = wave % WM, wn = wave / WM;
  const int n0 = blockIdx.y * BN;
  const int cb = blockIdx.z * cps * CC;
  const int ce = cb + cps * CC < kk ? cb + cps * CC : kk;
  const int nchunk = cb < ce ? (ce - cb + CC - 1) / CC : 0;
  // Row tiles, a contiguous range per workgroup.  The workgroup of linear
  // index b runs on XCD b % 8, so the ranges are handed out XCD by XCD:
  // neighbouring tiles, whose gathers share halo rows, then run under the
  // same L2 (gridDim.x is a multiple of 8 when it is >= 8).
  const int64_t ntile = (ngroups + GPB - 1) / GPB;
  const int nx = gridDim.x, bx = blockIdx.x;
  const int lb = nx >= 8 ? (bx % 8) * (nx / 8) + bx / 8 : bx;
  const int64_t tile0 = ntile * lb / nx, mytiles = ntile * (lb + 1) / nx - tile0;
  if (mytiles <= 0 || nchunk <= 0) return;  // uniform over the workgroup

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

  // this thread's tile element: group a_g + GPP i, position a_p, channels 4 a_f..
  const bool a_on = tid < GPP * S3 * F4;
  const int a_g = tid / (S3 * F4), a_p = (tid / F4) % S3, a_f = tid % F4;
  const int a_px = a_p / (S * S), a_py = (a_p / S) % S, a_pz = a_p % S;
  const int a_lds = (a_g * P3 + a_px * PX + a_py * S + a_pz) * RS + 4 * a_f;
  // the position's parent-offset slot in the 27-entry neighbour row, and child
  const int a_ux = a_px - R, a_uy = a_py - R, a_uz = a_pz - R;
  const int a_slot = ((a_ux >> 1) + 1) * 9 + ((a_uy >> 1) + 1) * 3 + ((a_uz >> 1) + 1);
  const int a_coff = 4 * (a_ux & 1) + 2 * (a_uy & 1) + (a_uz & 1);

  // neighbour entries of this thread's positions: nbc for the tile being
  // gathered, nbn for the one after; entries of groups past the end read
  // entry 0 and are flagged -1 when used
  int32_t nbc[NA], nbn[NA];
  uint32_t okc = 0, okn = 0;
  auto load_nb = [&](int64_t t, int32_t (&v)[NA], uint32_t& ok) {
    const int64_t g0 = (tile0 + t) * GPB;
    ok = 0;
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int64_t g = g0 + a_g + GPP * i;
      const bool live = a_on && t < mytiles && g < ngroups;
      v[i] = nbr[live ? 27 * g + a_slot : 0];
      ok |= (uint32_t)live << i;
    }
  };

  // global -> registers: the tile of channel chunk c0
  v4f ra[NA];
  uint32_t aok = 0;
  int a_c0 = 0;
  auto load_a = [&](int c0) {
    const int ch = c0 + 4 * a_f;
    a_c0 = c0;
    aok = 0;
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const bool live = ((okc >> i) & 1) && nbc[i] >= 0 && ch < kk;
      const int64_t off = live ? (int64_t)(nbc[i] + a_coff) * kk + ch : 0;
      if constexpr (VEC) {
        ra[i] = *reinterpret_cast<const v4f*>(x + off);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) ra[i][j] = x[off + (live && ch + j < kk ? j : 0)];
      }
      aok |= (uint32_t)live << i;
    }
  };
  auto store_a = [&]() {
    if (!a_on) return;
    const int ch = a_c0 + 4 * a_f;
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      v4f v = ra[i];
      const bool live = (aok >> i) & 1;
#pragma unroll
      for (int j = 0; j < 4; ++j) v[j] = live && ch + j < kk ? v[j] : 0.f;
      *reinterpret_cast<v4f*>(&At[a_lds + i * GPP * P3 * RS]) = v;
    }
  };

  // weight slab element of this thread, pass i
  float4 rb[NB];
  uint32_t bok = 0;
  int b_c0 = 0;
  auto load_b = [&](int c0, int k0) {
    b_c0 = c0;
    bok = 0;
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int e = tid + i * TB;
      if constexpr (FLIP) {  // (t, n, f): 4 consecutive channels of W[K3-1-k][n]
        const int f = e % F4, n = (e / F4) % BN, t = e / (F4 * BN);
        const int gn = n0 + n, ch = c0 + 4 * f;
        const bool live = t < TSL && gn < nn && ch < kk;
        const int64_t off = live ? ((int64_t)(K3 - 1 - (k0 + t)) * nn + gn) * kk + ch : 0;
        if constexpr (VEC) {
          rb[i] = *reinterpret_cast<const float4*>(w + off);
        } else {
          rb[i].x = w[off];
          rb[i].y = w[off + (live && ch + 1 < kk ? 1 : 0)];
          rb[i].z = w[off + (live && ch + 2 < kk ? 2 : 0)];
          rb[i].w = w[off + (live && ch + 3 < kk ? 3 : 0)];
        }
        bok |= (uint32_t)live << i;
      } else {  // (t, cc, n4): 4 consecutive columns of W[k][ch]
        const int n4 = e % (BN / 4), cc = (e / (BN / 4)) % CC, t = e / (BN / 4 * CC);
        const int gn = n0 + 4 * n4, ch = c0 + cc;
        const bool live = t < TSL && ch < kk && gn < nn;
        const int64_t off = live ? ((int64_t)(k0 + t) * kk + ch) * nn + gn : 0;
        if constexpr (VEC) {
          rb[i] = *reinterpret_cast<const float4*>(w + off);
        } else {
          rb[i].x = w[off];
          rb[i].y = w[off + (live && gn + 1 < nn ? 1 : 0)];
          rb[i].z = w[off + (live && gn + 2 < nn ? 2 : 0)];
          rb[i].w = w[off + (live && gn + 3 < nn ? 3 : 0)];
        }
        bok |= (uint32_t)live << i;
      }
    }
  };
  auto store_b = [&]() {
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int e = tid + i * TB;
      const bool live = (bok >> i) & 1;
      if constexpr (FLIP) {
        const int f = e % F4, n = (e / F4) % BN, t = e / (F4 * BN);
        const int ch = b_c0 + 4 * f;
        if (t < TSL) {
          const float4 v = rb[i];
          *reinterpret_cast<float4*>(&Bt[(t * BN + n) * RS + 4 * f]) =
              float4{live ? v.x : 0.f, live && ch + 1 < kk ? v.y : 0.f,
                     live && ch + 2 < kk ? v.z : 0.f, live && ch + 3 < kk ? v.w : 0.f};
        }
      } else {
        const int n4 = e % (BN / 4), cc = (e / (BN / 4)) % CC, t = e / (BN / 4 * CC);
        const int gn = n0 + 4 * n4;
        if (t < TSL) {
          float* d = &Bt[(t * BN + 4 * n4) * RS + cc];
          d[0] = live ? rb[i].x : 0.f;
          d[RS] = live && gn + 1 < nn ? rb[i].y : 0.f;
          d[2 * RS] = live && gn + 2 < nn ? rb[i].z : 0.f;
          d[3 * RS] = live && gn + 3 < nn ? rb[i].w : 0.f;
        }
      }
    }
  };

  auto compute = [&](int k0) {
#pragma unroll 3
    for (int tp = 0; tp < TSL; ++tp) {
      const int k = k0 + tp;
      const int toff = (k / K2) * PX + ((k / K) % K) * S + k % K;
      float a[MR][V], b[NR][V];
#pragma unroll
      for (int mr = 0; mr < MR; ++mr) {
        const float* tpp = &At[(tbase[mr] + toff) * RS + V * q];
        if constexpr (V == 4) {
          const v4f u = *reinterpret_cast<const v4f*>(tpp);
#pragma unroll
          for (int j = 0; j < 4; ++j) a[mr][j] = u[j];
        } else {
          a[mr][0] = tpp[0];
        }
      }
#pragma unroll
      for (int nr = 0; nr < NR; ++nr) {
        const float* bp = &Bt[(tp * BN + bcol[nr]) * RS + V * q];
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
  };

  load_nb(0, nbc, okc);
  load_nb(1, nbn, okn);
  load_a(cb);
  load_b(cb, 0);
  for (int64_t t = 0; t < mytiles; ++t) {
    for (int ci = 0; ci < nchunk; ++ci) {
      const int c0 = cb + ci * CC;
      const bool last = ci + 1 == nchunk;
#pragma unroll
      for (int sl = 0; sl < NSL; ++sl) {
        __syncthreads();  // the previous step's LDS reads are done
        if (sl == 0) store_a();
        store_b();
        __syncthreads();
        if (sl + 1 < NSL) {
          load_b(c0, (sl + 1) * TSL);
        } else {  // the next chunk of this tile, or the first chunk of the next tile
#pragma unroll
          for (int i = 0; i < NA; ++i) nbc[i] = last ? nbn[i] : nbc[i];
          okc = last ? okn : okc;
          load_nb(last ? t + 2 : t + 1, nbn, okn);
          const int nc0 = last ? cb : c0 + CC;
          load_a(nc0);
          load_b(nc0, 0);
        }
        compute(sl * TSL);
      }
    }
    // the tile is complete: accumulator j of lane l is row 4(l/16)+j, column l%16
    const int64_t g0 = (tile0 + t) * GPB;
    const int64_t nrows = 8 * ngroups;
    const bool split = gridDim.z > 1;
    float* dst = split ? part + (int64_t)blockIdx.z * nrows * nn : out;
#pragma unroll
    for (int mr = 0; mr < MR; ++mr) {
      const int64_t rbase = 8 * g0 + (wm * MR + mr) * 16 + 4 * q;
#pragma unroll
      for (int nr = 0; nr < NR; ++nr) {
        const int n = n0 + bcol[nr];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int64_t row = rbase + j;
          if (n < nn && row < nrows) {
            const float v = acc[mr][nr][j];
            dst[row * nn + n] = (!split && relu) ? fmaxf(v, 0.f) : v;
          }
        }
        acc[mr][nr] = v4f{0.f, 0.f, 0.f, 0.f};
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Stride-1, K = 3 convolution, weights in registers (k_conv_tile3):
// out[i][n] = sum_k sum_c x[nb(i,k)][c] W'[k][c][n] for the 16-channel chunk
// c0 = 16 blockIdx.z of the reduction (partial sums when there are several).
// The MFMA computes out^T: A = W'^T (16 output channels x 4 reduction
// channels), B = the gathered rows (4 channels x 16 octants).  Each wave
// keeps the chunk's weights of its 16 output channels in registers for the
// whole launch (27 taps x 4 channels per lane), so the only LDS traffic is
// the group tiles: one 16-byte read per lane feeds four MFMAs.
// Workgroups (two or three per CU) are persistent over a contiguous range of
// sibling groups, taken in tiles of GPB groups (GPB/2 blocks of 16 rows).
// Wave w takes output channels 16 (w % WN).. and row blocks RB (w / WN) + r,
// r < RB; in the range's last tile, which may be partial, the live row
// blocks are dealt round the WM waves of a column instead.  The
// (K+1)^3 x 16-channel group tiles are streamed with direct global->LDS
// loads into two static buffers: tile t+1 lands while tile t is multiplied,
// with one barrier per tile.  Absent neighbours and channels past kk read a
// zero row.
// Group tile layout, in 16-byte chunks: group g at 280 g, x-slab at 68 x,
// position (y, z) at slot 4y + z, channel quad f stored at f ^ ((y + 2z) & 3).
// A read of one tap by 8 (or 16) lanes touches 2 slabs x 2 y x 2 z positions
// (of 1 or 2 groups) at one quad; the quad swizzle and the strides (68 = 4
// mod 8, 280 = 8 mod 16) put them on distinct banks whether the LDS serves 8
// lanes from 32 banks or 16 lanes from 64.  Each x-slab of a group (16
// positions x 4 quads) is one wave's load instruction.
// FLIP: input gradient, W'[k][c][n] = W[26-k][n][c].
// POOL (forward only, one reduction chunk): the 2x2x2 max-pool follows the
// (ReLU'd) output in the epilogue, through a small LDS area per wave; out
// is then the pooled map [npar][nn] of depth l-1 (row prow[g] for group g,
// loaded a tile ahead), psw the switches [ngroups][nn], and the workgroups
// of column block 0 zero an equal share of the rows of empty depth-(l-1)
// octants (plab[i] == 0).
template <int WN, int GPB, bool FLIP, bool POOL>
__global__ __launch_bounds__(TB) __attribute__((amdgpu_waves_per_eu(2))) void k_conv_tile3(const int32_t* __restrict__ nbr,
                                                   int64_t ngroups, const float* __restrict__ x,
                                                   int kk, const float* __restrict__ w, int nn,
                                                   float* __restrict__ out, int relu,
                                                   float* __restrict__ part,
                                                   const int32_t* __restrict__ prow,
                                                   const int32_t* __restrict__ plab, int64_t npar,
                                                   uint8_t* __restrict__ psw) {
  constexpr int K3 = 27, BN = 16 * WN, WM = WAVES / WN;
  constexpr int RB = GPB / 2 / WM;  // row blocks per wave
  static_assert(RB >= 1 && RB * WM * 2 == GPB, "every row block has one wave");
  constexpr int GSTR = 280, XSTR = 68, BUFC = GPB * GSTR;  // in 16-byte chunks
  __shared__ __attribute__((aligned(16))) v4f X0[BUFC];
  __shared__ __attribute__((aligned(16))) v4f X1[BUFC];
  __shared__ __attribute__((aligned(16))) float PS[WAVES][POOL ? oc::kPoolLdsFloats : 4];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, q = lane >> 4;
  const int wn = wave % WN, wm = wave / WN;
  const int n0 = blockIdx.y * BN + 16 * wn, c0 = 16 * blockIdx.z;
  const int nx = gridDim.x, bx = blockIdx.x;
  const int lb = nx >= 8 ? (bx % 8) * (nx / 8) + bx / 8 : bx;  // XCD-contiguous ranges
  const int64_t g0 = ngroups * lb / nx, g1 = ngroups * (lb + 1) / nx;  // groups [g0, g1)
  const int T = (int)((g1 - g0 + GPB - 1) / GPB);
  if constexpr (POOL) {
    if (blockIdx.y == 0) {  // rows of empty depth-(l-1) octants
      const int64_t r0 = npar * lb / nx, r1 = npar * (lb + 1) / nx;
      const int c4 = nn / 4, cnt = (int)(r1 - r0) * c4;
      for (int e = tid; e < cnt; e += TB) {
        const int64_t i = r0 + e / c4;
        if (plab[i] == 0)
          *reinterpret_cast<v4f*>(out + i * nn + 4 * (e % c4)) = v4f{0.f, 0.f, 0.f, 0.f};
      }
    }
  }
  if (T <= 0) return;  // uniform over the workgroup
  // pooled forward: the depth-(l-1) output row of this lane's group in each
  // of its row blocks, loaded a tile ahead of the epilogue that stores it
  int32_t prq[RB];
  auto load_pr = [&](int t) {
    if constexpr (POOL) {
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        const int64_t g = g0 + (int64_t)t * GPB + 2 * (wm * RB + r) + ((lane >> 4) & 1);
        prq[r] = g < g1 ? prow[g] : -1;
      }
    }
  };

  // loads: wave w fills x-slab w of every group; lane -> chunk (slot 4y + z,
  // stored quad), holding channel quad (stored ^ ((y + 2z) & 3))
  const int py = lane >> 4, pz = (lane >> 2) & 3, px = wave;
  const int f_ = (lane & 3) ^ ((py + 2 * pz) & 3);
  const int ux = px - 1, uy = py - 1, uz = pz - 1;
  const int l_slot = ((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1);
  const int l_coff = 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1);
  const int l_ch = c0 + 4 * f_;
  int32_t nbc[GPB], nbn[GPB];
  uint32_t okc = 0, okn = 0;
  auto load_nb = [&](int t, int32_t (&v)[GPB], uint32_t& ok) {
    ok = 0;
#pragma unroll
    for (int i = 0; i < GPB; ++i) {
      const int64_t g = g0 + (int64_t)t * GPB + i;
      const bool live = t < T && g < g1;
      v[i] = nbr[live ? 27 * g + l_slot : 0];
      ok |= (uint32_t)live << i;
    }
  };
  // lanes of absent rows write their zeros themselves (a shared zero row
  // would put every absent lane of the grid on one cache line)
  auto dma = [&](v4f* buf) {
#pragma unroll
    for (int i = 0; i < GPB; ++i) {
      const bool live = ((okc >> i) & 1) && nbc[i] >= 0 && l_ch < kk;
      v4f* blk = buf + i * GSTR + px * XSTR;
      const uint32_t a = lds_addr(blk);
      if (live)
        lds_load16(x + (int64_t)(nbc[i] + l_coff) * kk + l_ch, a);
      else
        blk[lane] = v4f{0.f, 0.f, 0.f, 0.f};
    }
  };

  // reads: lane (li, q) supplies row li of row block rb: child li & 7 of
  // group 2 rb + (li >> 3), channels 4q..4q+3
  int aoff[9];
  {
    const int g = 2 * (wm * RB) + (li >> 3), c = li & 7;
    const int cx = c >> 2, cy = (c >> 1) & 1, cz = c & 1;
#pragma unroll
    for (int j = 0; j < 9; ++j) {
      const int y = cy + j / 3, z = cz + j % 3;
      aoff[j] = g * GSTR + cx * XSTR + 4 * (4 * y + z) + (q ^ ((y + 2 * z) & 3));
    }
  }

  v4f acc0[RB], acc1[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) acc0[r] = acc1[r] = v4f{0.f, 0.f, 0.f, 0.f};
  v4f wr[K3];  // this lane's weights: wr[k][s] = W'[k][c0 + 4q + s][n0 + li]
  constexpr int KLO = 13;
  auto load_w = [&](bool hi) {  // taps k < KLO, or k >= KLO
    const int n = n0 + li, c = c0 + 4 * q;
    const bool ok = n < nn && c < kk;
#pragma unroll
    for (int k = 0; k < K3; ++k) {
      if ((k >= KLO) != hi) continue;
      v4f v = {0.f, 0.f, 0.f, 0.f};
      if (ok) {
        if constexpr (FLIP) {
          v = *reinterpret_cast<const v4f*>(w + ((int64_t)(K3 - 1 - k) * nn + n) * kk + c);
        } else {
#pragma unroll
          for (int s = 0; s < 4; ++s) v[s] = w[((int64_t)k * kk + c + s) * nn + n];
        }
      }
      wr[k] = v;
    }
  };

  // the rows of tap k+1 are read before the MFMAs of tap k
  auto compute = [&](const v4f* buf, v4f (&acc)[RB]) {
    v4f b[2][RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) b[0][r] = buf[aoff[0] + 2 * r * GSTR];
#pragma unroll
    for (int k = 0; k < K3; ++k) {
      const int cu = k & 1, nx2 = cu ^ 1;
      if (k + 1 < K3) {
#pragma unroll
        for (int r = 0; r < RB; ++r)
          b[nx2][r] = buf[aoff[(k + 1) % 9] + ((k + 1) / 9) * XSTR + 2 * r * GSTR];
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int r = 0; r < RB; ++r) acc[r] = mfma4(wr[k][s], b[cu][r][s], acc[r]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  // one row block rb of the tile (the partial last tile), into acc
  auto compute1 = [&](const v4f* buf, int rb, v4f& acc) {
    const v4f* bb = buf + 2 * (rb - wm * RB) * GSTR;
    v4f b[2];
    b[0] = bb[aoff[0]];
#pragma unroll
    for (int k = 0; k < K3; ++k) {
      const int cu = k & 1, nx2 = cu ^ 1;
      if (k + 1 < K3) b[nx2] = bb[aoff[(k + 1) % 9] + ((k + 1) / 9) * XSTR];
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int s = 0; s < 4; ++s) acc = mfma4(wr[k][s], b[cu][s], acc);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  const int64_t nrows = 8 * ngroups;
  const bool split = gridDim.z > 1;
  float* dst = split ? part + (int64_t)blockIdx.z * nrows * nn : out;
  // accumulator j of lane l: output channel 4(l/16) + j, row l % 16; stored
  // after store_order: lane l writes row l/4, channels 4(l%4)..
  const int64_t rowe = 8 * g1;  // rows past the range are not stored
  // pr: the pooled forward's output row of this lane's group
  auto store_rb = [&](int t, int rb, const v4f& acc, int32_t pr) {
    if constexpr (POOL) {
      // through the wave's LDS area: lane o < 32 pools group o/16 of the
      // row block in channel n0 + o%16
      v4f v = acc;
      if (relu) {
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = fmaxf(v[j], 0.f);
      }
      float* ps = &PS[wave][0];
      oc::pool_put(ps, v, lane);
      uint32_t sw;
      const float m = oc::pool_scan(ps, lane, sw);
      const int c = n0 + (lane & 15);
      const int64_t g = g0 + (int64_t)t * GPB + 2 * rb + ((lane >> 4) & 1);
      if (lane < 32 && c < nn && g < g1) {
        out[(int64_t)pr * nn + c] = m;
        psw[g * nn + c] = (uint8_t)sw;
      }
      return;
    }
    const int n = n0 + 4 * (lane & 3);
    const int64_t row = 8 * (g0 + (int64_t)t * GPB) + 16 * rb + (lane >> 2);
    const v4f sv = store_order(acc, lane);
    if (n < nn && row < rowe) {
      v4f v = sv;
      if (!split && relu) {
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = fmaxf(v[j], 0.f);
      }
      *reinterpret_cast<v4f*>(dst + row * nn + n) = v;
    }
  };
  auto epilogue = [&](int t, v4f (&acc)[RB]) {
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      store_rb(t, wm * RB + r, acc[r], POOL ? prq[r] : 0);
      acc[r] = v4f{0.f, 0.f, 0.f, 0.f};
    }
  };
  // tile t: wait for its loads everywhere (and for tile t-1's reads), write
  // tile t-1, start tile t+1's loads, multiply tile t
  auto step = [&](int t, const v4f* cur, v4f* nxt, v4f (&accc)[RB], v4f (&accp)[RB],
                  bool first) {
    vm_wait0();  // this wave's loads into cur have landed
    __syncthreads();
    if (t > 0) epilogue(t - 1, accp);
    load_pr(t);  // lands during tile t's MFMAs
#pragma unroll
    for (int i = 0; i < GPB; ++i) nbc[i] = nbn[i];
    okc = okn;
    if (t + 1 < T) {
      load_nb(t + 2, nbn, okn);
      dma(nxt);
    }
    if (first) load_w(true);  // the later taps' weights land during tile 0
    __builtin_amdgcn_sched_barrier(0);
    compute(cur, accc);
  };

  // the first tile's neighbour entries, the first KLO taps' weights and the
  // first tile's rows are in flight together; the other taps' weights are
  // loaded at the start of tile 0 and waited for tap by tap
  load_nb(0, nbc, okc);
  load_w(false);
  dma(X0);
  load_nb(1, nbn, okn);

  // tiles 0 .. T-2 (tile 0 apart, with the rest of the weights), then the
  // last one (in X0 when T-1 is even)
  if (T > 1) step(0, X0, X1, acc0, acc1, true);
  for (int t = 1; t + 1 < T; t += 2) {
    step(t, X1, X0, acc1, acc0, false);
    if (t + 2 < T) step(t + 1, X0, X1, acc0, acc1, false);
  }
  const bool last0 = (T - 1) % 2 == 0;
  vm_wait0();
  __syncthreads();
  if (T > 1) {
    if (last0)
      epilogue(T - 2, acc1);
    else
      epilogue(T - 2, acc0);
  }
  if (T == 1) load_w(true);
  // live row blocks of the last tile, rb = wm + WM i
  const int rbl = (int)((g1 - g0 - (int64_t)(T - 1) * GPB + 1) / 2);
  for (int rb = wm; rb < rbl; rb += WM) {
    int32_t pr = 0;
    if constexpr (POOL) {
      const int64_t g = g0 + (int64_t)(T - 1) * GPB + 2 * rb + ((lane >> 4) & 1);
      pr = g < g1 ? prow[g] : -1;
    }
    v4f a = v4f{0.f, 0.f, 0.f, 0.f};
    compute1(last0 ? X0 : X1, rb, a);
    store_rb(T - 1, rb, a, pr);
  }
}

// ---------------------------------------------------------------------------
// Stride-1, K = 3 forward for Cin = 3 or 4 (k_conv_cin): the first layer,
// whose rows are too short for the channel-quad kernels.  MFMA step s is tap
// s; within it, lane group q supplies input channel q (a zero weight when
// q >= Cin), so a row block of 16 octants takes 27 MFMAs and every operand
// read is one base register plus a compile-time offset.  The MFMA computes
// out^T: A = W^T (16 output channels x 4 channels of tap s), B = the gathered
// rows (4 channels x 16 octants).
// A workgroup takes 8 sibling groups (64 rows, one block of 16 per wave) and
// 16 output channels (blockIdx.y).  Each group's (K+1)^3 tile is one wave
// load instruction (direct global->LDS, 12 or 16 bytes per position at a
// 16-byte lane stride), position (x, y, z) in slot 16x + 4y + z.  The weight
// block goes through LDS with 16-byte loads.
template <int CIN>
__global__ __launch_bounds__(TB) void k_conv_cin(const int32_t* __restrict__ nbr, int64_t ngroups,
                                                 const float* __restrict__ x,
                                                 const float* __restrict__ w, int nn,
                                                 float* __restrict__ out, int relu) {
  constexpr int K3 = 27, GPB = 8;
  constexpr int GSTR = 64 * 4 + 8;  // floats per group tile; 8 mod 32 separates the two groups' banks
  constexpr int NW4 = K3 * 4 * 4;   // float4 elements of the weight block [27][4][16]
  __shared__ __attribute__((aligned(16))) float Xs[GPB * GSTR];
  __shared__ __attribute__((aligned(16))) v4f Ws[NW4];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, q = lane >> 4;
  const int n0 = blockIdx.y * 16;
  const int64_t g0 = (int64_t)blockIdx.x * GPB;

  // loads: wave w fills the tiles of groups 2w and 2w+1, lane = slot
  {
    const int px = lane >> 4, py = (lane >> 2) & 3, pz = lane & 3;
    const int ux = px - 1, uy = py - 1, uz = pz - 1;
    const int slot = ((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1);
    const int coff = 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1);
    int32_t nb[2];
#pragma unroll
    for (int gg = 0; gg < 2; ++gg) {
      const int64_t g = g0 + 2 * wave + gg;
      nb[gg] = g < ngroups ? nbr[27 * g + slot] : -1;
    }
#pragma unroll
    for (int gg = 0; gg < 2; ++gg) {
      float* dst = Xs + (2 * wave + gg) * GSTR;
      const uint32_t a = lds_addr(dst);
      if (nb[gg] >= 0) {  // absent rows: the lane writes zeros itself
        const float* src = x + (int64_t)(nb[gg] + coff) * CIN;
        if constexpr (CIN == 4) {
          lds_load16(src, a);
        } else {
          lds_load12(src, a);
        }
      } else {
        *reinterpret_cast<v4f*>(dst + 4 * lane) = v4f{0.f, 0.f, 0.f, 0.f};
      }
    }
  }
  // the weight block: Ws[(k * 4 + c) * 4 + f] = W[k][c][n0 + 4f..] (zero for
  // c >= Cin or past nn), 16-byte loads
#pragma unroll
  for (int i = 0; i < (NW4 + TB - 1) / TB; ++i) {
    const int e = tid + i * TB;
    if (e < NW4) {
      const int f = e & 3, c = (e >> 2) & 3, k = e >> 4, n = n0 + 4 * f;
      Ws[e] = c < CIN && n < nn ? *reinterpret_cast<const v4f*>(w + ((int64_t)k * CIN + c) * nn + n)
                                : v4f{0.f, 0.f, 0.f, 0.f};
    }
  }
  vm_wait0();  // this wave's tile loads have landed
  __syncthreads();
  // lane (li, q): row li of the wave's block (child li & 7 of group
  // 2 wave + (li >> 3)), input channel q (channel 0 with weight 0 past Cin)
  const int c = li & 7;
  const float* xb = Xs + (2 * wave + (li >> 3)) * GSTR +
                    4 * (16 * (c >> 2) + 4 * ((c >> 1) & 1) + (c & 1)) + (q < CIN ? q : 0);
  const float* wb = reinterpret_cast<const float*>(Ws) + q * 16 + li;
  v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int k = 0; k < K3; ++k)
    acc = mfma4(wb[k * 64], xb[4 * (16 * (k / 9) + 4 * ((k / 3) % 3) + k % 3)], acc);
  // accumulator j of lane l: output channel n0 + 4(l/16) + j, row l % 16;
  // after store_order lane l writes row l/4, channels n0 + 4(l%4)..
  acc = store_order(acc, lane);
  const int64_t row = 8 * g0 + 16 * wave + (lane >> 2);
  const int n = n0 + 4 * (lane & 3);
  if (row < 8 * ngroups && n < nn) {
    if (relu) {
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] = fmaxf(acc[j], 0.f);
    }
    *reinterpret_cast<v4f*>(out + row * nn + n) = acc;
  }
}

// out[e] = sum over splits of part[z][e] (in split order), ReLU if relu.
// Four consecutive entries per thread (16-byte loads when vec, i.e. n is a
// multiple of 4 and the buffers are 16-byte aligned), four splits in flight.
__global__ __launch_bounds__(TB) void k_sum_split(const float* __restrict__ part, int splits,
                                                  int64_t n, float* __restrict__ out, int relu,
                                                  int vec) {
  const int64_t e = 4 * ((int64_t)blockIdx.x * TB + threadIdx.x);
  if (e >= n) return;
  if (vec) {
    const v4f* p = reinterpret_cast<const v4f*>(part + e);
    const int64_t n4 = n / 4;
    v4f s = {0.f, 0.f, 0.f, 0.f};
    int z = 0;
    for (; z + 4 <= splits; z += 4) {
      const v4f a = p[z * n4], b = p[(z + 1) * n4], c = p[(z + 2) * n4], d = p[(z + 3) * n4];
      s += a;
      s += b;
      s += c;
      s += d;
    }
    for (; z < splits; ++z) s += p[z * n4];
    if (relu) {
#pragma unroll
      for (int j = 0; j < 4; ++j) s[j] = fmaxf(s[j], 0.f);
    }
    *reinterpret_cast<v4f*>(out + e) = s;
    return;
  }
  for (int64_t i = e; i < e + 4 && i < n; ++i) {
    float s = 0.f;
    for (int z = 0; z < splits; ++z) s += part[(int64_t)z * n + i];
    out[i] = relu ? fmaxf(s, 0.f) : s;
  }
}

// k_sum_split followed by the 2x2x2 max-pool (the conv + pool forward with a
// split reduction).  Thread (i, channel quad) has two independent jobs, so
// that no load waits for another: as depth-(l-1) octant i, it writes a zero
// row when i is empty (labels[i] == 0); as sibling group i (i < ngroups), it
// forms the eight children's sums in k_sum_split's order, ReLU'd when relu,
// and writes their maximum (the first over children 0..7 wins, strict '>')
// to the row of group i's parent, rows[i], with its switches.  nn a
// multiple of 4; part, y 16-byte and sw 4-byte aligned.
__global__ __launch_bounds__(TB) void k_sum_split_pool(const float* __restrict__ part, int splits,
                                                       int64_t n, const int32_t* __restrict__ labels,
                                                       const int32_t* __restrict__ rows,
                                                       int64_t npar, int64_t ngroups, int cv,
                                                       int relu, float* __restrict__ y,
                                                       uint8_t* __restrict__ sw) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= npar * cv) return;
  const int64_t i = t / cv;
  const int cc = (int)(t - i * cv);
  if (labels[i] == 0) reinterpret_cast<v4f*>(y)[t] = v4f{0.f, 0.f, 0.f, 0.f};
  if (i >= ngroups) return;
  const int64_t g = i, n4 = n / 4;
  const int64_t prow = rows[g];
  const v4f* p = reinterpret_cast<const v4f*>(part) + 8 * g * cv + cc;
  v4f sk[8];  // the eight children's sums, their loads of one split in flight together
#pragma unroll
  for (int k = 0; k < 8; ++k) sk[k] = v4f{0.f, 0.f, 0.f, 0.f};
  for (int z = 0; z < splits; ++z) {
#pragma unroll
    for (int k = 0; k < 8; ++k) sk[k] += p[z * n4 + (int64_t)k * cv];
  }
  v4f best = {0.f, 0.f, 0.f, 0.f};
  uint32_t arg = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    v4f s = sk[k];
    if (relu) {
#pragma unroll
      for (int j = 0; j < 4; ++j) s[j] = fmaxf(s[j], 0.f);
    }
    if (k == 0) {
      best = s;
      continue;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (s[j] > best[j]) {
        best[j] = s[j];
        arg = (arg & ~(0xffu << (8 * j))) | ((uint32_t)k << (8 * j));
      }
  }
  reinterpret_cast<v4f*>(y)[prow * cv + cc] = best;
  reinterpret_cast<uint32_t*>(sw)[g * cv + cc] = arg;
}

// Launch of k_sum_split over n entries.
void sum_split(const float* part, int splits, int64_t n, float* out, int relu, hipStream_t s) {
  const int vec = n % 4 == 0 && (uintptr_t)part % 16 == 0 && (uintptr_t)out % 16 == 0;
  oc::launch(k_sum_split, dim3((unsigned)oc::cdiv(n, 4 * TB)), dim3(TB), 0, s, part, splits,
                     n, out, relu, vec);
}

// Max-pool backward (Sec. 3.2 "Pooling") of an input gradient that is still
// held as the split partial sums of its reduction: thread (g, quad) forms the
// gradient of group g's parent row rows[g] (depth l) in channels 4 quad ..
// 4 quad + 3 (splits > 1: the sum over part[z] in k_sum_split's order; 1: the
// gradient itself) and writes the eight child rows 8g .. 8g+7 (depth l+1):
// the gradient in the child the switch names where the pooled value mask is
// > 0 (no mask: NULL), zero elsewhere.  The depth-l gradient is never
// stored; the result equals k_sum_split followed by the pool backward.
// pn: floats per split (N_l * cin); cv = cin / 4.
__global__ __launch_bounds__(TB) void k_route_parts(const float* __restrict__ part, int splits,
                                                    int64_t pn, const float* __restrict__ mask,
                                                    const uint8_t* __restrict__ sw,
                                                    const int32_t* __restrict__ rows,
                                                    int64_t ngroups, int cv,
                                                    float* __restrict__ out) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ngroups * cv) return;
  const int64_t g = t / cv;
  const int cc = (int)(t - g * cv);
  const uint32_t sv = reinterpret_cast<const uint32_t*>(sw)[t];
  const int64_t src = (int64_t)rows[g] * cv + cc;
  const v4f* p = reinterpret_cast<const v4f*>(part) + src;
  v4f v;
  if (splits == 1) {
    v = p[0];
  } else {
    const int64_t n4 = pn / 4;
    v = v4f{0.f, 0.f, 0.f, 0.f};
    for (int z = 0; z < splits; ++z) v += p[z * n4];
  }
  v4f m = {1.f, 1.f, 1.f, 1.f};
  if (mask) m = reinterpret_cast<const v4f*>(mask)[src];
  v4f* dst = reinterpret_cast<v4f*>(out) + 8 * g * cv + cc;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    v4f o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = ((sv >> (8 * e)) & 0xffu) == (uint32_t)k && m[e] > 0.f ? v[e] : 0.f;
    dst[(int64_t)k * cv] = o;
  }
}

// Routing of a depth-l input gradient through the 2x2x2 max-pool from depth
// l+1 (see k_route_parts).
struct RouteOut {
  const float* mask;  // pooled values [N_l][cin], or NULL
  const uint8_t* sw;  // switches [M_l][cin]
  float* out;         // [N_{l+1}][cin]
};

void route_parts(const oc_octree* t, int l, const float* part, int splits, int cin,
                 const RouteOut& ro, hipStream_t s) {
  const int64_t G = t->M[l];
  const int cv = cin / 4;
  if (G == 0) return;
  oc::launch(k_route_parts, dim3((unsigned)oc::cdiv(G * cv, TB)), dim3(TB), 0, s, part, splits,
             t->N[l] * (int64_t)cin, ro.mask, ro.sw, (const int32_t*)t->rows[l], G, cv, ro.out);
}

// ---------------------------------------------------------------------------
// Weight gradient partial sums, stride 1:
//   dW[k][c][n] = sum over octants i of x[nb(i,k)][c] * dY[i][n], an M x N =
//   (tap, channel) x (output channel) GEMM whose reduction runs over the octants, four per MFMA step: the
//   children 4h + q (q = lane / 16) of one sibling group.
// Operand loads go straight to global memory, where one 16-lane slice reads
// one row: with VA > 1 lane i loads channels VA i .. VA i + VA - 1 of it in one
// vector load and feeds them to VA MFMAs (M row i of MFMA s is channel
// VA i + s); likewise VB for the output channels of dY.  A wave owns TT taps x
// 16 VA channels x 16 VB output channels (PERM mode) or, for cin < 16, MB
// blocks of 16 consecutive flattened (tap, channel) pairs x 16 VB output
// channels (FLAT mode, MB > 0), and walks the groups of its workgroup's chunk
// with the neighbour entries two groups and the operands one group ahead.
// A workgroup holds WT tiles; the WAVES / WT waves of a tile interleave over
// the groups of the chunk and their sums are added in wave order through LDS.
// Grid: x = chunk of gchunk groups, y = ceil(tiles / WT);
// part[chunk][(k*cin + c)*cout + n].
template <int V>
__device__ __forceinline__ void ldv(const float* p, int valid, float (&v)[V]) {
  if constexpr (V == 4) {
    if (valid >= 4) {
      const float4 t = *reinterpret_cast<const float4*>(p);
      v[0] = t.x, v[1] = t.y, v[2] = t.z, v[3] = t.w;
      return;
    }
  } else if constexpr (V == 2) {
    if (valid >= 2) {
      const float2 t = *reinterpret_cast<const float2*>(p);
      v[0] = t.x, v[1] = t.y;
      return;
    }
  }
#pragma unroll
  for (int s = 0; s < V; ++s) v[s] = s < valid ? p[s] : 0.f;
}

template <int K, int VA, int VB, int TT, int MB, int WT>
__global__ __launch_bounds__(TB) void k_conv_dw(const int32_t* __restrict__ nbr, int64_t ngroups,
                                                int64_t gchunk, const float* __restrict__ x,
                                                int cin, const float* __restrict__ dy, int cout,
                                                float* __restrict__ part) {
  constexpr int R = (K - 1) / 2, K3 = K * K * K;
  constexpr bool FLAT = MB > 0;
  constexpr int NA = FLAT ? MB : TT;  // A operands per reduction step
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int li = lane & 15, q = lane >> 4;
  const int mtot = K3 * cin;
  const int tiles_n = (cout + 16 * VB - 1) / (16 * VB);
  const int tiles_m = FLAT ? (mtot + 16 * MB - 1) / (16 * MB)
                           : (K3 / TT) * ((cin + 16 * VA - 1) / (16 * VA));
  constexpr int WPT = WAVES / WT;  // waves per tile
  const int wt = wave % WT, gp = wave / WT;
  const int tile = blockIdx.y * WT + wt;
  const bool on = tile < tiles_m * tiles_n;  // idle waves still reach the barrier
  const int tm = on ? tile % tiles_m : 0, tn = on ? tile / tiles_m : 0;

  // per-lane operand geometry: parent-offset slot and child offset of each
  // (half, operand), the channel and its count of valid lanes
  int slot[2][NA], coff[2][NA], ach[NA], aval[NA];
#pragma unroll
  for (int a = 0; a < NA; ++a) {
    int k, c0;
    if constexpr (FLAT) {
      const int m = (tm * MB + a) * 16 + li;
      k = m < mtot ? m / cin : 0;
      c0 = m - k * cin;
      aval[a] = m < mtot ? 1 : 0;
    } else {
      const int tg = tm % (K3 / TT), cb = tm / (K3 / TT);
      k = tg * TT + a;
      c0 = cb * 16 * VA + VA * li;
      aval[a] = cin - c0;
    }
    ach[a] = c0;
    const int ox = k / (K * K), oy = (k / K) % K, oz = k % K;  // tap offset + R
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int c = 4 * h + q;
      const int ux = (c >> 2) + ox - R, uy = ((c >> 1) & 1) + oy - R, uz = (c & 1) + oz - R;
      slot[h][a] = ((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1);
      coff[h][a] = 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1);
    }
  }
  const int n0 = tn * 16 * VB + VB * li;
  const int nval = cout - n0;

  v4f acc[NA][FLAT ? 1 : VA][VB];
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int sa = 0; sa < (FLAT ? 1 : VA); ++sa)
#pragma unroll
      for (int sb = 0; sb < VB; ++sb) acc[a][sa][sb] = v4f{0.f, 0.f, 0.f, 0.f};

  // the waves of a tile take groups gb + gp, gb + gp + WPT, ...
  const int64_t gb = (int64_t)blockIdx.x * gchunk;
  const int64_t ge = !on ? gb : gb + gchunk < ngroups ? gb + gchunk : ngroups;

  constexpr int WA = FLAT ? 1 : VA;
  int32_t nbc[2][NA], nbn[2][NA];
  float ac[2][NA][WA], an[2][NA][WA], bc[2][VB], bn[2][VB];
  auto load_nb = [&](int64_t g, int32_t (&v)[2][NA]) {
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int a = 0; a < NA; ++a) v[h][a] = g < ge ? nbr[27 * g + slot[h][a]] : -1;
  };
  auto load_ops = [&](int64_t g, const int32_t (&v)[2][NA], float (&A)[2][NA][WA],
                      float (&Bv)[2][VB]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int64_t orow = 8 * g + 4 * h + q;
      float b[VB];
      ldv<VB>(dy + orow * cout + n0, g < ge ? nval : 0, b);
#pragma unroll
      for (int s = 0; s < VB; ++s) Bv[h][s] = b[s];
#pragma unroll
      for (int a = 0; a < NA; ++a) {
        const int32_t src = v[h][a] < 0 ? -1 : v[h][a] + coff[h][a];
        float t[WA];
        ldv<WA>(x + (int64_t)(src < 0 ? 0 : src) * cin + ach[a], src < 0 ? 0 : aval[a], t);
#pragma unroll
        for (int s = 0; s < WA; ++s) A[h][a][s] = t[s];
      }
    }
  };

  load_nb(gb + gp, nbc);
  load_ops(gb + gp, nbc, ac, bc);
  load_nb(gb + gp + WPT, nbn);
  for (int64_t g = gb + gp; g < ge; g += WPT) {
    load_ops(g + WPT, nbn, an, bn);
    load_nb(g + 2 * WPT, nbn);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int sa = 0; sa < WA; ++sa)
#pragma unroll
          for (int sb = 0; sb < VB; ++sb)
            acc[a][sa][sb] = mfma4(ac[h][a][sa], bc[h][sb], acc[a][sa][sb]);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int s = 0; s < WA; ++s) ac[h][a][s] = an[h][a][s];
#pragma unroll
      for (int s = 0; s < VB; ++s) bc[h][s] = bn[h][s];
    }
  }

  // the sums of a tile's waves, added in wave order through LDS
  constexpr int NACC = NA * WA * VB * 4;
  if constexpr (WPT > 1) {
    __shared__ float red[WT * (WPT - 1) * NACC * 64];
    if (gp > 0) {
      float* r = red + (wt * (WPT - 1) + gp - 1) * NACC * 64;
#pragma unroll
      for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int sa = 0; sa < WA; ++sa)
#pragma unroll
          for (int sb = 0; sb < VB; ++sb)
#pragma unroll
            for (int j = 0; j < 4; ++j)
              r[(((a * WA + sa) * VB + sb) * 4 + j) * 64 + lane] = acc[a][sa][sb][j];
    }
    __syncthreads();
    if (gp != 0) return;
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
      for (int sa = 0; sa < WA; ++sa)
#pragma unroll
        for (int sb = 0; sb < VB; ++sb)
#pragma unroll
          for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int w = 0; w < WPT - 1; ++w)
              acc[a][sa][sb][j] +=
                  red[((wt * (WPT - 1) + w) * NACC + ((a * WA + sa) * VB + sb) * 4 + j) * 64 + lane];
  }
  if (!on) return;

  // accumulator r of lane l: M row 4(l/16)+r, N column l%16
  float* pp = part + (int64_t)blockIdx.x * ((int64_t)mtot * cout);
#pragma unroll
  for (int a = 0; a < NA; ++a)
#pragma unroll
    for (int sa = 0; sa < WA; ++sa)
#pragma unroll
      for (int sb = 0; sb < VB; ++sb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = 4 * q + r;
          const int n = tn * 16 * VB + VB * li + sb;
          int m;
          if constexpr (FLAT) {
            m = (tm * MB + a) * 16 + i;
          } else {
            const int tg = tm % (K3 / TT), cb = tm / (K3 / TT);
            const int ch = cb * 16 * VA + VA * i + sa;
            m = ch < cin ? (tg * TT + a) * cin + ch : mtot;
          }
          if (m < mtot && n < cout) pp[(int64_t)m * cout + n] = acc[a][sa][sb][r];
        }
}

// ---------------------------------------------------------------------------
// Weight gradient through LDS, K = 3:
//   dW[k][c][n] = sum over octants i of x[nb(i,k)][c] * dY[i][n]
// A workgroup takes a chunk of sibling groups and, GS groups at a time,
// stages their (K+1)^3 x CW tiles of x and their 8 GS rows x BN columns of dY
// in LDS (register-staged one stage ahead, the neighbour entries two).  The
// MFMA reduction index is the octant: the children 4h + q (q = lane / 16) of
// a group, so lane l supplies A[c = l%16][child] from the tile position of
// that child's tap and B[child][n = l%16] from the dY rows; one staged dY
// value feeds the MFMAs of every tap.
// Tiled mode (cin >= 16): the workgroup owns channels 16 cbk.. 16 cbk+15 and
// columns BN nbk..; wave w takes taps w, w+4, ... (NJ at most).
// FLAT mode (cin < 16): M runs over (tap, channel) pairs m = tap cin + c,
// which is the row of dW itself; blocks of 16 pairs are dealt to the waves
// (rotated by workgroup so that no SIMD always gets the short share).
// HV = 2 (tiled mode only): the workgroup is two such 4-wave halves that
// take alternate stages of the chunk, each with its own staging buffers; at
// the end they add their accumulators through LDS (half 0 keeps the first
// ceil(NJ/2) blocks, half 1 the rest), so a workgroup holds twice the
// octants per partial and the partial traffic halves.
// Workgroup (chunk, tile) writes part[chunk][K3 cin][cout] for its block of
// dW (every entry of the block, zeros included); a second kernel adds the
// chunks in a fixed order.  XV: cin is a multiple of 4 (x rows read as
// float4); cout must be a multiple of 4.
template <bool FLAT, int CW, int NBN, int GS, bool XV, int HV>
__global__ __launch_bounds__(TB * HV) void k_conv_dwt(const int32_t* __restrict__ nbr,
                                                      int64_t ngroups, int64_t gchunk,
                                                      const float* __restrict__ x, int cin,
                                                      const float* __restrict__ dy, int cout,
                                                      float* __restrict__ part) {
  static_assert(HV == 1 || (HV == 2 && !FLAT), "two halves in tiled mode only");
  constexpr int R = 1, S = 4, K3 = 27, S3 = 64;
  // M blocks per wave at most: 27 taps, or ceil(27 cin / 16) <= 7, 14, 27 pairs
  constexpr int NJ = !FLAT ? 7 : CW == 4 ? 2 : CW == 8 ? 4 : 7;
  constexpr int SY = S + 2, PX = S * SY, P3 = S * PX;  // tile row of (px,py,pz): px PX + py SY + pz
  constexpr int RS = CW, F4 = CW / 4;
  constexpr int BN = 16 * NBN;
  constexpr int BNS = (BN % 32 == 0) ? BN + 16 : BN;  // dY rows of 4 children on distinct banks
  constexpr int GPP = TB / (S3 * F4);                 // groups per staging pass
  constexpr int NX = GS / GPP;
  constexpr int NYE = 8 * GS * (BN / 4);  // float4 elements of a dY stage
  constexpr int NY = (NYE + TB - 1) / TB;
  static_assert(TB % (S3 * F4) == 0 && GS % GPP == 0, "x staging covers the stage");
  static_assert(NX <= 32 && NY <= 32, "validity bits fit a word");
  constexpr int NA = GS * P3 * RS, NB = 8 * GS * BNS;      // floats of one half's buffers
  constexpr int NRED = HV == 2 ? NJ * NBN * WAVES * 64 * 4 : 0;  // floats of the reduction
  constexpr int NSM = HV * (NA + NB) > NRED ? HV * (NA + NB) : NRED;
  __shared__ __attribute__((aligned(16))) float smem[NSM];

  const int tid = threadIdx.x & (TB - 1), lane = tid & 63;
  const int half = HV == 1 ? 0 : __builtin_amdgcn_readfirstlane(threadIdx.x >> 8);
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar branches
  float* const At = smem + half * (NA + NB);
  float* const Bt = At + NA;
  const int li = lane & 15, q = lane >> 4;
  const int nCB = FLAT ? 1 : (cin + 15) / 16;
  const int cbk = (int)(blockIdx.y % nCB), nbk = (int)(blockIdx.y / nCB);
  const int c0 = FLAT ? 0 : 16 * cbk, n0 = BN * nbk;
  const int64_t gb = (int64_t)blockIdx.x * gchunk;
  const int64_t ge = gb + gchunk < ngroups ? gb + gchunk : ngroups;
  // stages of GS groups; half h takes stages h, h + HV, ...
  const int nsub = gb < ge ? (int)((ge - gb + GS * HV - 1) / (GS * HV)) : 0;
  const int nmb = FLAT ? (K3 * cin + 15) / 16 : K3;  // M blocks (taps when tiled)
  const int rot = FLAT ? (int)(blockIdx.x % WAVES) : 0;
  const int mb0 = (wave + rot) % WAVES;
  const int njw = nmb > mb0 ? (nmb - mb0 + WAVES - 1) / WAVES : 0;  // blocks of this wave

  // M blocks of this wave: block mb[j] = 4 j + mb0; the lane's LDS offset
  // (tap position and channel) and, in FLAT mode, validity
  int aoff[NJ];
  bool alive[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int mb = 4 * j + mb0;
    int tap, ch;
    if constexpr (FLAT) {
      const int m = 16 * mb + li;
      alive[j] = m < K3 * cin;
      tap = alive[j] ? m / cin : 0;
      ch = alive[j] ? m - tap * cin : 0;
    } else {
      alive[j] = mb < K3;
      tap = alive[j] ? mb : 0;
      ch = li;
    }
    aoff[j] = ((tap / 9) * PX + ((tap / 3) % 3) * SY + tap % 3) * RS + ch;
  }
  // tile row of child 4h + q at tap offset -R on every axis: h PX + (q>>1) SY + (q&1)
  const int hoff = ((q >> 1) * SY + (q & 1)) * RS;

  v4f acc[NJ][NBN];
#pragma unroll
  for (int j = 0; j < NJ; ++j)
#pragma unroll
    for (int nb = 0; nb < NBN; ++nb) acc[j][nb] = v4f{0.f, 0.f, 0.f, 0.f};

  // x staging: thread -> (group a_g + GPP i, position a_p, channel quad a_f)
  const int a_g = tid / (S3 * F4), a_p = (tid / F4) % S3, a_f = tid % F4;
  const int a_px = a_p / 16, a_py = (a_p / 4) % 4, a_pz = a_p % 4;
  const int a_lds = (a_g * P3 + a_px * PX + a_py * SY + a_pz) * RS + 4 * a_f;
  const int a_ux = a_px - R, a_uy = a_py - R, a_uz = a_pz - R;
  const int a_slot = ((a_ux >> 1) + 1) * 9 + ((a_uy >> 1) + 1) * 3 + ((a_uz >> 1) + 1);
  const int a_coff = 4 * (a_ux & 1) + 2 * (a_uy & 1) + (a_uz & 1);
  const int a_ch = c0 + 4 * a_f;

  int32_t nbc[NX], nbn[NX];
  uint32_t okc = 0, okn = 0;
  auto load_nb = [&](int s, int32_t (&v)[NX], uint32_t& ok) {
    ok = 0;
#pragma unroll
    for (int i = 0; i < NX; ++i) {
      const int64_t g = gb + (int64_t)(HV * s + half) * GS + a_g + GPP * i;
      const bool live = g < ge;
      v[i] = nbr[live ? 27 * g + a_slot : 0];
      ok |= (uint32_t)live << i;
    }
  };
  v4f rx[NX];
  uint32_t xok = 0;
  auto load_x = [&]() {
    xok = 0;
#pragma unroll
    for (int i = 0; i < NX; ++i) {
      const bool live = ((okc >> i) & 1) && nbc[i] >= 0 && a_ch < cin;
      const int64_t off = live ? (int64_t)(nbc[i] + a_coff) * cin + a_ch : 0;
      if constexpr (XV) {
        rx[i] = *reinterpret_cast<const v4f*>(x + off);
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j) rx[i][j] = x[off + (live && a_ch + j < cin ? j : 0)];
      }
      xok |= (uint32_t)live << i;
    }
  };
  auto store_x = [&]() {
#pragma unroll
    for (int i = 0; i < NX; ++i) {
      const bool live = (xok >> i) & 1;
      v4f v = rx[i];
#pragma unroll
      for (int j = 0; j < 4; ++j) v[j] = live && a_ch + j < cin ? v[j] : 0.f;
      *reinterpret_cast<v4f*>(&At[a_lds + i * GPP * P3 * RS]) = v;
    }
  };
  // dY staging: element e = tid + i TB -> stage row e / (BN/4), columns 4 (e % (BN/4))..
  v4f ry[NY];
  uint32_t yok = 0;
  auto load_dy = [&](int s) {
    yok = 0;
#pragma unroll
    for (int i = 0; i < NY; ++i) {
      const int e = tid + i * TB;
      const int r = e / (BN / 4), gn = n0 + 4 * (e % (BN / 4));
      const int64_t g0 = gb + (int64_t)(HV * s + half) * GS;
      const bool live = e < NYE && g0 + r / 8 < ge && gn < cout;
      const int64_t off = live ? (8 * g0 + r) * cout + gn : 0;
      ry[i] = *reinterpret_cast<const v4f*>(dy + off);
      yok |= (uint32_t)live << i;
    }
  };
  auto store_dy = [&]() {
#pragma unroll
    for (int i = 0; i < NY; ++i) {
      const int e = tid + i * TB;
      if (NYE % TB == 0 || e < NYE) {
        const int r = e / (BN / 4), f = e % (BN / 4);
        const bool live = (yok >> i) & 1;
        const v4f v = ry[i];
        *reinterpret_cast<v4f*>(&Bt[r * BNS + 4 * f]) =
            v4f{live ? v[0] : 0.f, live ? v[1] : 0.f, live ? v[2] : 0.f, live ? v[3] : 0.f};
      }
    }
  };

  load_nb(0, nbc, okc);
  load_nb(1, nbn, okn);
  load_x();
  load_dy(0);
  for (int s = 0; s < nsub; ++s) {
    __syncthreads();  // the previous stage's LDS reads are done
    store_x();
    store_dy();
    __syncthreads();
#pragma unroll
    for (int i = 0; i < NX; ++i) nbc[i] = nbn[i];
    okc = okn;
    load_nb(s + 2, nbn, okn);
    load_x();
    load_dy(s + 1);
    // operands of step st = (group st/2, children 4(st%2)+q), one step ahead
    // of the MFMAs; blocks past the wave's share multiply zeros (the longest
    // share sets the pace anyway)
    float a[2][NJ], b[2][NBN];
    auto rd = [&](int st, float (&av)[NJ], float (&bv)[NBN]) {
      const int g = st >> 1, h = st & 1;
#pragma unroll
      for (int nb = 0; nb < NBN; ++nb) bv[nb] = Bt[(8 * g + 4 * h + q) * BNS + 16 * nb + li];
      const float* ag = &At[g * P3 * RS + h * PX * RS + hoff];
#pragma unroll
      for (int j = 0; j < NJ; ++j) av[j] = ag[aoff[j]];
    };
    rd(0, a[0], b[0]);
#pragma unroll
    for (int st = 0; st < 2 * GS; ++st) {
      const int cu = st & 1, nx = cu ^ 1;
      if (st + 1 < 2 * GS) rd(st + 1, a[nx], b[nx]);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const float av = alive[j] ? a[cu][j] : 0.f;
#pragma unroll
        for (int nb = 0; nb < NBN; ++nb) acc[j][nb] = mfma4(av, b[cu][nb], acc[j][nb]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // halves add their accumulators: block j goes to half j < JH ? 0 : 1
  constexpr int JH = (NJ + 1) / 2;
  if constexpr (HV == 2) {
    v4f* red = reinterpret_cast<v4f*>(smem);
    __syncthreads();  // the last stage's LDS reads are done
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if ((j < JH) != (half == 0))
#pragma unroll
        for (int nb = 0; nb < NBN; ++nb) red[((j * NBN + nb) * WAVES + wave) * 64 + lane] = acc[j][nb];
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      if ((j < JH) == (half == 0))
#pragma unroll
        for (int nb = 0; nb < NBN; ++nb) {
          const v4f o = red[((j * NBN + nb) * WAVES + wave) * 64 + lane];
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[j][nb][r] += o[r];
        }
  }

  // accumulator r of lane l: M row 4(l/16) + r, column l % 16
  const int64_t entries = (int64_t)K3 * cin * cout;
  float* pp = part + (int64_t)blockIdx.x * entries;
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int mb = 4 * j + mb0;
    if (j >= njw || (HV == 2 && (j < JH) != (half == 0))) continue;
#pragma unroll
    for (int nb = 0; nb < NBN; ++nb) {
      const int n = n0 + 16 * nb + li;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int i = 4 * q + r;
        int m;
        bool ok;
        if constexpr (FLAT) {
          m = 16 * mb + i;
          ok = m < K3 * cin;
        } else {
          ok = c0 + i < cin;
          m = mb * cin + c0 + i;
        }
        if (ok && n < cout) pp[(int64_t)m * cout + n] = acc[j][nb][r];
      }
    }
  }
}

// Fixed-order sum of np partials of n entries in one pass, for buffers that
// k_sum_parts_multi cannot take (not 16-byte aligned, or n not a multiple of
// 4): a workgroup takes TB / SUB entry slots (four consecutive entries each
// when V = 4), and thread (slot, k) adds partials k, k + SUB, k + 2 SUB, ...
// in order, four loads in flight; the SUB sub-sums of a slot are then added
// in k order.  SUB = 64 gives small n enough threads.
template <int SUB, int V>
__global__ __launch_bounds__(TB) void k_sum_parts(const float* __restrict__ part, int np,
                                                  int64_t n, float* __restrict__ out) {
  using vec = std::conditional_t<V == 4, v4f, float>;
  constexpr int SLOTS = TB / SUB;
  __shared__ vec r[SUB][SLOTS];
  const int el = threadIdx.x % SLOTS, sg = threadIdx.x / SLOTS;
  const int64_t nv = n / V, e = (int64_t)blockIdx.x * SLOTS + el;
  const vec* pv = reinterpret_cast<const vec*>(part);
  vec acc = {};
  if (e < nv) {
    int p = sg;
    for (; p + 3 * SUB < np; p += 4 * SUB) {  // four independent loads in flight
      const vec a = pv[(int64_t)p * nv + e], b = pv[(int64_t)(p + SUB) * nv + e];
      const vec c = pv[(int64_t)(p + 2 * SUB) * nv + e], d = pv[(int64_t)(p + 3 * SUB) * nv + e];
      acc += a;
      acc += b;
      acc += c;
      acc += d;
    }
    for (; p < np; p += SUB) acc += pv[(int64_t)p * nv + e];
  }
  r[sg][el] = acc;
  __syncthreads();
  if (sg == 0 && e < nv) {
    vec t = r[0][el];
#pragma unroll 8
    for (int k = 1; k < SUB; ++k) t += r[k][el];
    reinterpret_cast<vec*>(out)[e] = t;
  }
}

// Sub-sums per entry slot of k_sum_parts_multi for np partials: the power of
// two nearest below np / 8 (about eight loads per thread), 1 to 64.
int sum_sub(int np) {
  int sub = 1;
  while (sub < 64 && 16 * sub <= np) sub *= 2;
  return sub;
}

// Fixed-order sums of several sets of partials in one launch: workgroups
// [first[i], first[i + 1]) add set i.  A workgroup takes TB / SUB entry
// slots of four consecutive entries; thread (slot, k) adds partials k,
// k + SUB, k + 2 SUB, ... in order, four loads in flight, and the SUB
// sub-sums of a slot are then added pairwise in LDS (k + SUB/2 into k, then
// k + SUB/4, ...).  The order depends only on the set's partial count, so
// every entry's bits are the same in any batch.  Every set's count a
// multiple of 4, 16-byte aligned buffers.
struct PartSet {
  const float* part;
  float* out;
  int64_t n;
  int np, sub, first;
};
constexpr int MAX_SETS = 8;
struct PartSets {
  PartSet s[MAX_SETS];
  int n;
};

__global__ __launch_bounds__(TB) void k_sum_parts_multi(PartSets sets) {
  __shared__ v4f r[TB];
  int i = 0;
  while (i + 1 < sets.n && (int)blockIdx.x >= sets.s[i + 1].first) ++i;
  const PartSet& d = sets.s[i];
  const int SUB = d.sub, SLOTS = TB / SUB;
  const int el = threadIdx.x % SLOTS, sg = threadIdx.x / SLOTS;  // slot, sub-sum
  const int64_t nv = d.n / 4, e = (int64_t)((int)blockIdx.x - d.first) * SLOTS + el;
  const v4f* pv = reinterpret_cast<const v4f*>(d.part);
  const int np = d.np;
  v4f acc = {};
  if (e < nv) {
    int p = sg;
    for (; p + 3 * SUB < np; p += 4 * SUB) {  // four independent loads in flight
      const v4f a = pv[(int64_t)p * nv + e], b = pv[(int64_t)(p + SUB) * nv + e];
      const v4f c = pv[(int64_t)(p + 2 * SUB) * nv + e], f = pv[(int64_t)(p + 3 * SUB) * nv + e];
      acc += a;
      acc += b;
      acc += c;
      acc += f;
    }
    for (; p < np; p += SUB) acc += pv[(int64_t)p * nv + e];
  }
  r[sg * SLOTS + el] = acc;
  for (int h = SUB / 2; h >= 1; h /= 2) {
    __syncthreads();
    if (sg < h) r[sg * SLOTS + el] += r[(sg + h) * SLOTS + el];
  }
  if (sg == 0 && e < nv) reinterpret_cast<v4f*>(d.out)[e] = r[el];
}

void sum_parts(const float* part, int np, int64_t n, float* out, hipStream_t s) {
  const bool v4 = n % 4 == 0 && (uintptr_t)part % 16 == 0 && (uintptr_t)out % 16 == 0;
  if (v4) {  // the batched kernel with one set: the same bits as in a batch
    oc::sum_partials_multi(1, &part, &np, &n, &out, s);
    return;
  }
  // unaligned or ragged: one entry per slot
  const bool wide = oc::cdiv(n, TB / 16) >= 2 * (int64_t)oc::cu_count();
  const unsigned grid = (unsigned)oc::cdiv(n, TB / (wide ? 16 : 64));
  if (wide)
    oc::launch((k_sum_parts<16, 1>), dim3(grid), dim3(TB), 0, s, part, np, n, out);
  else
    oc::launch((k_sum_parts<64, 1>), dim3(grid), dim3(TB), 0, s, part, np, n, out);
}

// ---------------------------------------------------------------------------
// Launch-shape selection.

struct TileCfg {
  int V, MR, NR, WM, splits, cps;
  bool VEC;
  bool v2;  // k_conv_tile3: K = 3, 16-channel chunks, one chunk per split
  int gpb;  // k_conv_tile3: sibling groups per tile
};

// Workgroup tile and split of the reduction for a stride-1 layer of G groups
// (chosen from measurements of the depth-2..6 layers of the 32-shape batch).
TileCfg pick_tile(int K, int64_t G, int kk, int nn) {
  TileCfg c;
  c.VEC = kk % 4 == 0 && nn % 4 == 0;
  c.v2 = K == 3 && c.VEC && kk >= 16;
  if (c.v2) {
    c.V = 4, c.MR = 1, c.WM = 4;
    c.NR = nn <= 16 ? 1 : nn <= 32 ? 2 : 4;  // column blocks per workgroup (WN)
    c.cps = 1;
    c.splits = (int)oc::cdiv(kk, 16);
    // tile size: the least time for the longest range of groups (two
    // workgroups per CU), counting a wave's row blocks plus a fixed cost per
    // tile (barrier, loads, stores) of about 3/4 of a row block
    const int64_t slots = 2 * (int64_t)oc::cu_count();
    const int64_t gyz = oc::cdiv(nn, 16 * c.NR) * c.splits;
    const int64_t ng = oc::cdiv(G, std::max<int64_t>(1, slots / gyz));
    const int wm = WAVES / c.NR;
    double best = 1e30;
    c.gpb = 8;
    for (int gpb = 8; gpb >= 2; gpb /= 2) {
      if (gpb / 2 < wm) break;  // a row block for every wave
      const int rb = gpb / 2 / wm;
      const int64_t full = ng / gpb, tail = ng - full * gpb;
      const double cost = full * (rb + 0.75) +
                          (tail > 0 ? (double)oc::cdiv(oc::cdiv(tail, 2), wm) + 0.75 : 0.0);
      if (cost < best - 1e-9) best = cost, c.gpb = gpb;
    }
    return c;
  }
  c.V = (K == 3 && kk >= 16 && c.VEC) ? 4 : 1;
  c.WM = 4;
  if (c.V == 1 && K == 3) {
    c.MR = 2, c.NR = 1;  // 128 x 16
  } else {
    c.MR = 1, c.NR = nn <= 16 ? 1 : 2;  // 64 x 16 or 64 x 32
  }
  const int BM = 16 * c.WM * c.MR, BN = 16 * (WAVES / c.WM) * c.NR;
  const int64_t tiles = oc::cdiv(G, BM / 8) * oc::cdiv(nn, BN);
  const int chunks = (int)oc::cdiv(kk, 4 * c.V);
  int splits = 1;
  while (tiles * splits < 2048 && splits * 2 <= chunks) splits *= 2;
  c.cps = (int)oc::cdiv(chunks, splits);
  c.splits = (int)oc::cdiv(chunks, c.cps);
  return c;
}

template <int K, int V, int MR, int NR, int WM, bool FLIP, bool VEC>
void launch_tile(const oc_octree* t, int l, const TileCfg& c, const float* x, int kk,
                 const float* w, int nn, float* out, int relu, float* part, hipStream_t s,
                 const RouteOut* ro = nullptr) {
  const auto kernel = k_conv_tile<K, V, MR, NR, WM, FLIP, VEC>;
  static const int occ = [&] {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, TB, 0) != hipSuccess || n < 1)
      n = 1;
    return n;
  }();
  const int64_t G = t->M[l - 1];
  constexpr int BM = 16 * WM * MR, BN = 16 * (WAVES / WM) * NR;
  const int64_t ntile = oc::cdiv(G, BM / 8);
  const int64_t gyz = oc::cdiv(nn, BN) * c.splits;
  // one resident wave of workgroups, each over a contiguous range of tiles
  int64_t px = std::min<int64_t>(ntile, std::max<int64_t>(1, (int64_t)oc::cu_count() * occ / gyz));
  if (px >= 8) px -= px % 8;
  dim3 grid((unsigned)px, (unsigned)oc::cdiv(nn, BN), (unsigned)c.splits);
  oc::launch_main(kernel, grid, dim3(TB), s, (const int32_t*)t->nbr[l], G, x, kk, w, nn, out, relu,
                  c.cps, part);
  if (ro) {  // input gradient routed on (relu is 0)
    route_parts(t, l, c.splits > 1 ? part : out, c.splits, nn, *ro, s);
  } else if (c.splits > 1) {
    sum_split(part, c.splits, t->N[l] * (int64_t)nn, out, relu, s);
  }
}

// Destination of a pooled forward (conv + ReLU + 2x2x2 max-pool): the
// pooled rows of depth l-1 and the switches.
struct PoolOut {
  float* y;
  uint8_t* sw;
};

template <int NR, int GPB, bool FLIP>
void launch_tile2(const oc_octree* t, int l, const TileCfg& c, const float* x, int kk,
                  const float* w, int nn, float* out, int relu, float* part, hipStream_t s,
                  const PoolOut* po = nullptr, const RouteOut* ro = nullptr) {
  const auto plain = k_conv_tile3<NR, GPB, FLIP, false>;
  const auto pooled = k_conv_tile3<NR, GPB, FLIP, true>;
  const bool fuse = !FLIP && po && c.splits == 1;
  const auto kernel = fuse ? pooled : plain;
  static const int occ = [&] {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, plain, TB, 0) != hipSuccess || n < 1)
      n = 1;
    return n;
  }();
  const int64_t G = t->M[l - 1];
  const int64_t gy = oc::cdiv(nn, 16 * NR), gyz = gy * c.splits;
  // one resident workgroup per slot, each over a contiguous range of groups
  int64_t px = std::min<int64_t>(G, std::max<int64_t>(1, (int64_t)oc::cu_count() * occ / gyz));
  if (px >= 8) px -= px % 8;
  dim3 grid((unsigned)px, (unsigned)gy, (unsigned)c.splits);
  if (fuse) {
    oc::launch_main(kernel, grid, dim3(TB), s, (const int32_t*)t->nbr[l], G, x, kk, w, nn, po->y,
                    relu, part, (const int32_t*)t->rows[l - 1], (const int32_t*)t->labels[l - 1],
                    t->N[l - 1], po->sw);
    return;
  }
  oc::launch_main(kernel, grid, dim3(TB), s, (const int32_t*)t->nbr[l], G, x, kk, w, nn, out,
                  relu, part, (const int32_t*)nullptr, (const int32_t*)nullptr, (int64_t)0,
                  (uint8_t*)nullptr);
  if (ro) {  // input gradient routed on (relu is 0)
    route_parts(t, l, c.splits > 1 ? part : out, c.splits, nn, *ro, s);
    return;
  }
  if (c.splits > 1) {
    if (po) {
      const int cv = nn / 4;
      const int64_t npar = t->N[l - 1];
      oc::launch(k_sum_split_pool, dim3((unsigned)oc::cdiv(npar * cv, TB)), dim3(TB), 0, s,
                 (const float*)part, c.splits, t->N[l] * (int64_t)nn,
                 (const int32_t*)t->labels[l - 1], (const int32_t*)t->rows[l - 1], npar,
                 t->M[l - 1], cv, relu, po->y, po->sw);
    } else {
      sum_split(part, c.splits, t->N[l] * (int64_t)nn, out, relu, s);
    }
  }
}

template <bool FLIP>
void dispatch_tile(const oc_octree* t, int l, int K, const float* x, int kk, const float* w,
                   int nn, float* out, int relu, float* part, hipStream_t s,
                   const RouteOut* ro = nullptr) {
  const TileCfg c = pick_tile(K, t->M[l - 1], kk, nn);
  if (c.v2) {
#define OC_T3(NR_, GPB_)                                                                 \
  if (c.NR == NR_ && c.gpb == GPB_) {                                                    \
    launch_tile2<NR_, GPB_, FLIP>(t, l, c, x, kk, w, nn, out, relu, part, s, nullptr, ro); \
    return;                                                                              \
  }
    OC_T3(1, 8) OC_T3(2, 8) OC_T3(2, 4) OC_T3(4, 8) OC_T3(4, 4) OC_T3(4, 2)
#undef OC_T3
    return;
  }
#define OC_TILE(K_, V_, MR_, NR_, WM_, VEC_)                                                    \
  if (K == K_ && c.V == V_ && c.MR == MR_ && c.NR == NR_ && c.WM == WM_ && c.VEC == VEC_) {     \
    launch_tile<K_, V_, MR_, NR_, WM_, FLIP, VEC_>(t, l, c, x, kk, w, nn, out, relu, part, s, ro); \
    return;                                                                                     \
  }
  OC_TILE(3, 4, 1, 1, 4, true) OC_TILE(3, 4, 1, 2, 4, true)
  OC_TILE(3, 1, 2, 1, 4, true) OC_TILE(3, 1, 2, 1, 4, false)
  OC_TILE(5, 1, 1, 1, 4, true) OC_TILE(5, 1, 1, 1, 4, false)
  OC_TILE(5, 1, 1, 2, 4, true) OC_TILE(5, 1, 1, 2, 4, false)
#undef OC_TILE
}

// Weight gradient through LDS (k_conv_dwt): K = 3 with cout a multiple of 4,
// and cin a multiple of 4 when cin >= 16.
struct DwtCfg {
  bool flat, xv;
  int CW, NBN, GS, HV, tiles;
  int64_t gchunk, nchunks;
};

int dwt_occupancy(const DwtCfg& c);

bool pick_dwt(int K, int64_t G, int cin, int cout, DwtCfg* c) {
  if (K != 3 || cout % 4 != 0) return false;
  c->flat = cin < 16;
  c->xv = cin % 4 == 0;
  if (!c->flat && !c->xv) return false;
  if (c->flat) {
    c->CW = cin <= 4 ? 4 : cin <= 8 ? 8 : 16;
    c->GS = 64 / c->CW;
    c->NBN = cout <= 16 ? 1 : 2;
  } else {
    c->CW = 16, c->GS = 4;
    // 32 output channels per workgroup: 64 writes twice the partial sums (one
    // per resident workgroup) and 16 stages x twice as often; both were
    // measured slower on the depth-2..5 layers of the 32-shape batch
    c->NBN = cout >= 32 ? 2 : 1;
  }
  c->HV = c->flat ? 1 : 2;
  const int nCB = c->flat ? 1 : (int)oc::cdiv(cin, 16);
  c->tiles = nCB * (int)oc::cdiv(cout, 16 * c->NBN);
  const int64_t entries = (int64_t)27 * cin * cout;
  // one round of resident workgroups (at least one stage of groups each),
  // partial sums capped at 16M floats
  const int64_t slots = (int64_t)oc::cu_count() * dwt_occupancy(*c);
  int64_t chunks = std::max<int64_t>(1, slots / c->tiles);
  chunks = std::min<int64_t>(chunks, std::max<int64_t>(1, (int64_t(16) << 20) / entries));
  c->gchunk = std::max<int64_t>(c->GS, oc::cdiv(std::max<int64_t>(G, 1), chunks));
  c->nchunks = std::max<int64_t>(1, oc::cdiv(G, c->gchunk));
  return true;
}

template <bool FLAT, int CW, int NBN, int GS, bool XV, int HV>
void launch_dwt(const oc_octree* t, int l, const DwtCfg& c, const float* x, int cin,
                const float* dy, int cout, float* part, hipStream_t s) {
  dim3 grid((unsigned)c.nchunks, (unsigned)c.tiles);
  oc::launch_main(k_conv_dwt<FLAT, CW, NBN, GS, XV, HV>, grid, dim3(TB * HV), s, (const int32_t*)t->nbr[l],
                  t->M[l - 1], c.gchunk, x, cin, dy, cout, part);
}

// Resident workgroups per CU of the configuration's kernel (cached).
template <bool FLAT, int CW, int NBN, int GS, bool XV, int HV>
int dwt_occ() {
  static const int occ = [] {
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_conv_dwt<FLAT, CW, NBN, GS, XV, HV>, TB * HV, 0) !=
            hipSuccess ||
        n < 1)
      n = 1;
    return n;
  }();
  return occ;
}

#define OC_DWT_LIST(X)                                                                       \
  X(false, 16, 1, 4, true, 2) X(false, 16, 2, 4, true, 2) X(false, 16, 4, 4, true, 2)       \
  X(true, 4, 1, 16, true, 1) X(true, 4, 2, 16, true, 1) X(true, 4, 1, 16, false, 1)          \
  X(true, 4, 2, 16, false, 1) X(true, 8, 1, 8, true, 1) X(true, 8, 2, 8, true, 1)            \
  X(true, 8, 1, 8, false, 1) X(true, 8, 2, 8, false, 1) X(true, 16, 1, 4, true, 1)           \
  X(true, 16, 2, 4, true, 1) X(true, 16, 1, 4, false, 1) X(true, 16, 2, 4, false, 1)

int dwt_occupancy(const DwtCfg& c) {
#define OC_DWT_OCC(FLAT_, CW_, NBN_, GS_, XV_, HV_)                                         \
  if (c.flat == FLAT_ && c.CW == CW_ && c.NBN == NBN_ && c.GS == GS_ && c.xv == XV_ &&      \
      c.HV == HV_)                                                                          \
    return dwt_occ<FLAT_, CW_, NBN_, GS_, XV_, HV_>();
  OC_DWT_LIST(OC_DWT_OCC)
#undef OC_DWT_OCC
  return 1;
}

bool dispatch_dwt(const oc_octree* t, int l, const DwtCfg& c, const float* x, int cin,
                  const float* dy, int cout, float* part, hipStream_t s) {
#define OC_DWT(FLAT_, CW_, NBN_, GS_, XV_, HV_)                                             \
  if (c.flat == FLAT_ && c.CW == CW_ && c.NBN == NBN_ && c.GS == GS_ && c.xv == XV_ &&    \
      c.HV == HV_) {                                                                        \
    launch_dwt<FLAT_, CW_, NBN_, GS_, XV_, HV_>(t, l, c, x, cin, dy, cout, part, s);      \
    return true;                                                                          \
  }
  OC_DWT_LIST(OC_DWT)
#undef OC_DWT
  return false;
}

struct DwCfg {
  int VA, VB, TT, MB, WT, tiles;
  int64_t gchunk, nchunks;
};

// Wave tile, chunking and partial-sum count of the weight gradient.
DwCfg pick_dw(int K, int64_t G, int cin, int cout) {
  DwCfg c;
  const int K3 = K * K * K;
  const int64_t entries = (int64_t)K3 * cin * cout;
  // vector widths need rows whose length they divide
  c.VB = (cout >= 64 && cout % 4 == 0) ? 4 : (cout >= 32 && cout % 2 == 0) ? 2 : 1;
  const int tiles_n = (int)oc::cdiv(cout, 16 * c.VB);
  int tiles_m;
  if (cin < 16) {
    c.VA = 1, c.TT = 1;
    c.MB = (int)std::min<int64_t>(8, oc::cdiv((int64_t)K3 * cin, 16));
    tiles_m = (int)oc::cdiv((int64_t)K3 * cin, 16 * c.MB);
  } else {
    c.MB = 0;
    c.VA = (cin >= 64 && cin % 4 == 0) ? 4 : (cin >= 32 && cin % 2 == 0) ? 2 : 1;
    const int per = c.VA * c.VB;  // MFMAs per operand and reduction step
    c.TT = per >= 8 ? 1 : per >= 2 ? 3 : (K == 3 ? 9 : 5);
    if (K == 5 && c.TT == 3) c.TT = 5;
    tiles_m = (K3 / c.TT) * (int)oc::cdiv(cin, 16 * c.VA);
  }
  c.tiles = tiles_m * tiles_n;
  // many tiles: the waves of a workgroup share groups (L1 reuse); few: they
  // share a tile and split the groups
  c.WT = c.tiles >= 32 ? 4 : 1;
  // measured on the depth-2..6 layers of the 32-shape batch: about 2048
  // waves with WT = 4, 8192 with WT = 1; partial sums capped at 16M floats
  const int64_t target = c.WT == 4 ? 2048 : 8192;
  int64_t chunks = std::max<int64_t>(1, oc::cdiv(target, (int64_t)c.tiles * (WAVES / c.WT)));
  chunks = std::min<int64_t>(chunks, std::max<int64_t>(1, (int64_t(16) << 20) / entries));
  c.gchunk = std::max<int64_t>(8, oc::cdiv(std::max<int64_t>(G, 1), chunks));
  c.nchunks = std::max<int64_t>(1, oc::cdiv(G, c.gchunk));
  return c;
}

template <int K, int VA, int VB, int TT, int MB>
void launch_dw(const oc_octree* t, int l, const DwCfg& c, const float* x, int cin,
               const float* dy, int cout, float* part, hipStream_t s) {
  if (c.WT == 4) {
    dim3 grid((unsigned)c.nchunks, (unsigned)oc::cdiv(c.tiles, 4));
    oc::launch_main(k_conv_dw<K, VA, VB, TT, MB, 4>, grid, dim3(TB), s,
                    (const int32_t*)t->nbr[l], t->M[l - 1], c.gchunk, x, cin, dy, cout, part);
    return;
  }
  dim3 grid((unsigned)c.nchunks, (unsigned)c.tiles);
  oc::launch_main(k_conv_dw<K, VA, VB, TT, MB, 1>, grid, dim3(TB), s,
                     (const int32_t*)t->nbr[l], t->M[l - 1], c.gchunk, x, cin, dy, cout, part);
}

// Forward of a 3- or 4-channel input (the first layer): k_conv_cin.
inline bool use_cin_kernel(int K, int cin, int cout) {
  return K == 3 && (cin == 3 || cin == 4) && cout % 4 == 0;
}

}  // namespace

namespace oc {

void conv_s1_kernel_name(const oc_octree* t, int l, int K, int cin, int cout, int pass, char* buf,
                         size_t n) {
  const bool pooled = pass == 3;  // the conv + pool forward (its convolution kernel)
  if (pooled) pass = 0;
  if (pass != 1 && conv_cin_supported(K, cin, cout)) {
    conv_cin_kernel_name(cin, pooled ? 3 : pass, buf, n);
    return;
  }
  if (pass == 2) {
    DwtCfg d;
    if (pick_dwt(K, t->M[l - 1], cin, cout, &d)) {
      snprintf(buf, n, "k_conv_dwt<%s, %d, %d, %d, %s, %d>", d.flat ? "true" : "false", d.CW,
               d.NBN, d.GS, d.xv ? "true" : "false", d.HV);
      return;
    }
    const DwCfg c = pick_dw(K, t->M[l - 1], cin, cout);
    snprintf(buf, n, "k_conv_dw<%d, %d, %d, %d, %d, %d>", K, c.VA, c.VB, c.TT, c.MB, c.WT);
    return;
  }
  if (pass == 0 && use_cin_kernel(K, cin, cout)) {
    snprintf(buf, n, "k_conv_cin<%d>", cin);
    return;
  }
  const int kk = pass == 0 ? cin : cout, nn = pass == 0 ? cout : cin;
  const TileCfg c = pick_tile(K, t->M[l - 1], kk, nn);
  if (c.v2) {
    snprintf(buf, n, "k_conv_tile3<%d, %d, %s, %s>", c.NR, c.gpb, pass == 0 ? "false" : "true",
             pooled && c.splits == 1 ? "true" : "false");
    return;
  }
  snprintf(buf, n, "k_conv_tile<%d, %d, %d, %d, %d, %s, %s>", K, c.V, c.MR, c.NR, c.WM,
           pass == 0 ? "false" : "true", c.VEC ? "true" : "false");
}

size_t conv_s1_tile_ws(const oc_octree* t, int l, int K, int kk, int nn) {
  const TileCfg c = pick_tile(K, t->M[l - 1], kk, nn);
  return c.splits > 1 ? (size_t)c.splits * t->N[l] * nn * sizeof(float) : 0;
}

void conv_s1_fwd_f32(const oc_octree* t, int l, int K, const float* x, int cin, const float* w,
                     int cout, float* y, int relu, float* ws, hipStream_t s) {
  if (conv_cin_supported(K, cin, cout)) {
    conv_cin_fwd(t, l, x, cin, w, cout, y, relu, s);
    return;
  }
  if (use_cin_kernel(K, cin, cout)) {
    const int64_t G = t->M[l - 1];
    const dim3 grid((unsigned)oc::cdiv(G, 8), (unsigned)oc::cdiv(cout, 16));
    if (cin == 3)
      oc::launch_main(k_conv_cin<3>, grid, dim3(TB), s, (const int32_t*)t->nbr[l], G, x, w, cout,
                      y, relu);
    else
      oc::launch_main(k_conv_cin<4>, grid, dim3(TB), s, (const int32_t*)t->nbr[l], G, x, w, cout,
                      y, relu);
    return;
  }
  dispatch_tile<false>(t, l, K, x, cin, w, cout, y, relu, ws, s);
}

bool conv_s1_pool_fused(const oc_octree* t, int l, int K, int cin, int cout) {
  if (conv_cin_supported(K, cin, cout)) return true;
  if (use_cin_kernel(K, cin, cout)) return false;
  return pick_tile(K, t->M[l - 1], cin, cout).v2;
}

void conv_s1_pool_fwd_f32(const oc_octree* t, int l, int K, const float* x, int cin,
                          const float* w, int cout, float* yp, uint8_t* sw, int relu, float* ws,
                          hipStream_t s) {
  if (conv_cin_supported(K, cin, cout)) {
    conv_cin_pool_fwd(t, l, x, cin, w, cout, yp, sw, relu, s);
    return;
  }
  const TileCfg c = pick_tile(K, t->M[l - 1], cin, cout);
  const PoolOut po{yp, sw};
#define OC_T3(NR_, GPB_)                                                              \
  if (c.NR == NR_ && c.gpb == GPB_) {                                                 \
    launch_tile2<NR_, GPB_, false>(t, l, c, x, cin, w, cout, nullptr, relu, ws, s, &po); \
    return;                                                                           \
  }
  OC_T3(1, 8) OC_T3(2, 8) OC_T3(2, 4) OC_T3(4, 8) OC_T3(4, 4) OC_T3(4, 2)
#undef OC_T3
  oc::set_error("no pooled kernel for cin=%d cout=%d", cin, cout);
}

void conv_s1_bwd_data_f32(const oc_octree* t, int l, int K, const float* dy, int cout,
                          const float* w, int cin, float* dx, float* ws, hipStream_t s) {
  dispatch_tile<true>(t, l, K, dy, cout, w, cin, dx, 0, ws, s);
}

void conv_s1_bwd_data_pool_f32(const oc_octree* t, int l, int K, const float* dy, int cout,
                               const float* w, int cin, float* dx, const float* mask,
                               const uint8_t* sw, float* dxf, float* ws, hipStream_t s) {
  const RouteOut ro{mask, sw, dxf};
  dispatch_tile<true>(t, l, K, dy, cout, w, cin, dx, 0, ws, s, &ro);
}

size_t conv_s1_dw_parts(const oc_octree* t, int l, int K, int cin, int cout) {
  if (conv_cin_supported(K, cin, cout)) return conv_cin_dw_parts(t, l, cin, cout);
  DwtCfg d;
  int64_t np;
  if (pick_dwt(K, t->M[l - 1], cin, cout, &d)) {
    np = d.nchunks;
  } else {
    np = pick_dw(K, t->M[l - 1], cin, cout).nchunks;
  }
  return (size_t)np;
}

void conv_s1_bwd_weight_f32(const oc_octree* t, int l, int K, const float* x, int cin,
                            const float* dy, int cout, float* dw, float* part,
                            hipStream_t s, bool defer) {
  const int64_t entries = (int64_t)K * K * K * cin * cout;
  if (conv_cin_supported(K, cin, cout)) {
    conv_cin_dw(t, l, x, cin, dy, cout, dw, part, s, defer);
    return;
  }
  DwtCfg d;
  if (pick_dwt(K, t->M[l - 1], cin, cout, &d)) {
    if (dispatch_dwt(t, l, d, x, cin, dy, cout, part, s)) {
      if (!defer) sum_parts(part, (int)d.nchunks, entries, dw, s);
    } else {
      oc::set_error("no weight-gradient kernel for cin=%d cout=%d", cin, cout);
    }
    return;
  }
  const DwCfg c = pick_dw(K, t->M[l - 1], cin, cout);
#define OC_DW(K_, VA_, VB_, TT_, MB_)                                                       \
  if (K == K_ && c.VA == VA_ && c.VB == VB_ && c.TT == TT_ && c.MB == MB_) {               \
    launch_dw<K_, VA_, VB_, TT_, MB_>(t, l, c, x, cin, dy, cout, part, s);                 \
  } else
  // PERM mode, K = 3
  OC_DW(3, 4, 4, 1, 0) OC_DW(3, 4, 2, 1, 0) OC_DW(3, 2, 4, 1, 0) OC_DW(3, 4, 1, 3, 0)
  OC_DW(3, 1, 4, 3, 0) OC_DW(3, 2, 2, 3, 0) OC_DW(3, 2, 1, 3, 0) OC_DW(3, 1, 2, 3, 0)
  OC_DW(3, 1, 1, 9, 0)
  // FLAT mode (cin < 16), K = 3: MB = ceil(27 cin / 16) capped at 8
  OC_DW(3, 1, 1, 1, 2) OC_DW(3, 1, 2, 1, 2) OC_DW(3, 1, 4, 1, 2)
  OC_DW(3, 1, 1, 1, 4) OC_DW(3, 1, 2, 1, 4) OC_DW(3, 1, 4, 1, 4)
  OC_DW(3, 1, 1, 1, 6) OC_DW(3, 1, 2, 1, 6) OC_DW(3, 1, 4, 1, 6)
  OC_DW(3, 1, 1, 1, 7) OC_DW(3, 1, 2, 1, 7) OC_DW(3, 1, 4, 1, 7)
  OC_DW(3, 1, 1, 1, 8) OC_DW(3, 1, 2, 1, 8) OC_DW(3, 1, 4, 1, 8)
  // K = 5
  OC_DW(5, 4, 4, 1, 0) OC_DW(5, 4, 2, 1, 0) OC_DW(5, 2, 4, 1, 0) OC_DW(5, 4, 1, 5, 0)
  OC_DW(5, 1, 4, 5, 0) OC_DW(5, 2, 2, 5, 0) OC_DW(5, 2, 1, 5, 0) OC_DW(5, 1, 2, 5, 0)
  OC_DW(5, 1, 1, 5, 0)
  OC_DW(5, 1, 1, 1, 8) OC_DW(5, 1, 2, 1, 8) OC_DW(5, 1, 4, 1, 8) {
    oc::set_error("no weight-gradient kernel for K=%d cin=%d cout=%d", K, cin, cout);
  }
#undef OC_DW
  if (!defer) sum_parts(part, (int)c.nchunks, entries, dw, s);
}

void sum_partials(const float* part, int np, int64_t n, float* out, hipStream_t s) {
  sum_parts(part, np, n, out, s);
}

void sum_partials_multi(int n, const float* const* parts, const int* nparts,
                        const int64_t* counts, float* const* outs, hipStream_t s) {
  PartSets sets{};
  int blocks = 0;
  for (int i = 0; i < n; ++i) {
    const bool v4 = counts[i] % 4 == 0 && (uintptr_t)parts[i] % 16 == 0 &&
                    (uintptr_t)outs[i] % 16 == 0;
    if (!v4 || nparts[i] < 1 || counts[i] == 0) {  // not for the batch: alone
      if (counts[i] > 0 && nparts[i] >= 1) sum_parts(parts[i], nparts[i], counts[i], outs[i], s);
      continue;
    }
    if (sets.n == MAX_SETS) {  // a full batch goes now
      oc::launch(k_sum_parts_multi, dim3((unsigned)blocks), dim3(TB), 0, s, sets);
      sets.n = 0;
      blocks = 0;
    }
    const int64_t nv = counts[i] / 4;
    const int sub = sum_sub(nparts[i]);
    sets.s[sets.n++] = PartSet{parts[i], outs[i], counts[i], nparts[i], sub, blocks};
    blocks += (int)oc::cdiv(nv, TB / sub);
  }
  if (sets.n > 0) oc::launch(k_sum_parts_multi, dim3((unsigned)blocks), dim3(TB), 0, s, sets);
}

}  // namespace oc
