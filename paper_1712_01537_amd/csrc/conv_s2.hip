// Stride-2 octree convolution, K = 3 (Sec. 3.2 of O-CNN, Fig. 2): the output
// of sibling group g is the convolution evaluated at its first child (child
// 0), written to the row of g's parent at depth l-1 (rows of empty parents
// are 0).  The fp32 forward with channel counts that are multiples of 16 is
// one implicit-GEMM kernel (k_s2_fwd, below).  Everything else follows the
// paper's im2col + GEMM:
// a gather kernel builds the column buffer Col[g][k][c] = x[n(8g, k)][c]
// (0 for an absent neighbour; only parent offsets {-1,0}^3 are reached from
// child 0), a library GEMM multiplies it by W viewed as [27 Cin][Cout], and
// a second kernel moves each group's row to its parent's row.
//   weight gradient: dW = Col^T dY_g (GEMMs over runs of groups into eight
//     partial sums, added in a fixed order);
//   input gradient: input row 8h + c (child c of group h) is read by the
//     groups at parent offsets o in {0,1}^3 from h's parent with o_a = 0
//     where c_a = 0, through tap d = c - 2o.  So the eight rows of group h
//     are one product: dX[8h..8h+7] = D[h] Wx with D[h][o][:] = dY_g of the
//     group at offset o (0 if absent) and the expanded weight
//     Wx[o][co][c][ci] = W[c - 2o][ci][co] (0 where c - 2o leaves {-1,0,1}^3):
//     a gather and one GEMM whose output is dX itself, no atomics.
// dY_g[g] = dY[row of g's parent], masked by [y > 0] when the forward applied
// a ReLU.  bf16: every GEMM multiplies bf16 operands with fp32 accumulation;
// the backward's dY_g is rounded to bf16 (nearest even), like the stride-1
// backward.  GEMM atomics are disabled, so results are bit-for-bit
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

// fp32 -> bf16, round to nearest even (NaN stays NaN).
__device__ __forceinline__ uint16_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// Row of x that tap k of group g reads (child 0 + d), or -1.
__device__ __forceinline__ int32_t s2_src(const int32_t* __restrict__ nbr, int64_t g, int k) {
  const int dx = k / 9 - 1, dy = (k / 3) % 3 - 1, dz = k % 3 - 1;
  const int32_t base = nbr[27 * g + ((dx >> 1) + 1) * 9 + ((dy >> 1) + 1) * 3 + ((dz >> 1) + 1)];
  return base < 0 ? -1 : base + 4 * (dx & 1) + 2 * (dy & 1) + (dz & 1);
}

// Stride 4 (Sec. 3.2, stride 2^r with r = 2): row of x that tap k of
// output p reads, or -1.  Output p (the p-th non-empty octant of depth l-2)
// sits at depth-l position 4p; tap offset d reaches 4p + d = 2 (2p + a) +
// (d & 1) with a = d >> 1 in {-1, 0}: the depth-(l-1) octant at 2p + a is
// child (a & 1) of p's neighbour at offset a (through nbr1 = the depth-(l-1)
// group table, whose group p holds p's children), and the depth-l octant is
// child (d & 1) of it, when it is non-empty (lab1 = the depth-(l-1) labels).
__device__ __forceinline__ int32_t s4_src(const int32_t* __restrict__ nbr1,
                                          const int32_t* __restrict__ lab1, int64_t p, int k) {
  const int dx = k / 9 - 1, dy = (k / 3) % 3 - 1, dz = k % 3 - 1;
  const int ax = dx >> 1, ay = dy >> 1, az = dz >> 1;
  const int32_t f = nbr1[27 * p + (ax + 1) * 9 + (ay + 1) * 3 + (az + 1)];
  if (f < 0) return -1;
  const int32_t L = lab1[f + 4 * (ax & 1) + 2 * (ay & 1) + (az & 1)];
  return L <= 0 ? -1 : 8 * (L - 1) + 4 * (dx & 1) + 2 * (dy & 1) + (dz & 1);
}

// Source row of tap k of output g at stride 2^RR (RR = 1: nbr = the depth-l
// table; RR = 2: nbr = the depth-(l-1) table, lab = the depth-(l-1) labels).
template <int RR>
__device__ __forceinline__ int32_t sr_src(const int32_t* __restrict__ nbr,
                                          const int32_t* __restrict__ lab, int64_t g, int k) {
  if constexpr (RR == 1)
    return s2_src(nbr, g, k);
  else
    return s4_src(nbr, lab, g, k);
}

// Column buffer of groups g0 .. g0+ng-1: col[g-g0][k][:] = x[src][:] (T = fp32
// or bf16), one 16-byte piece per thread; rows of rb bytes, rb % 16 == 0.
template <typename T, int RR>
__global__ __launch_bounds__(TB) void k_s2_col(const int32_t* __restrict__ nbr,
                                               const int32_t* __restrict__ lab, int64_t g0,
                                               int64_t ng, const T* __restrict__ x, int rb,
                                               T* __restrict__ col) {
  const int np = rb / 16;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ng * 27 * np) return;
  const int pc = (int)(t % np);
  const int64_t gk = t / np;  // (g - g0) * 27 + k
  const int32_t src = sr_src<RR>(nbr, lab, g0 + gk / 27, (int)(gk % 27));
  uint4 v = {0u, 0u, 0u, 0u};
  if (src >= 0) v = *reinterpret_cast<const uint4*>((const char*)x + (int64_t)src * rb + 16 * pc);
  *reinterpret_cast<uint4*>((char*)col + gk * rb + 16 * pc) = v;
}

// Element-wise fallback for rows that are not a multiple of 16 bytes.
template <typename T, int RR>
__global__ __launch_bounds__(TB) void k_s2_col1(const int32_t* __restrict__ nbr,
                                                const int32_t* __restrict__ lab, int64_t g0,
                                                int64_t ng, const T* __restrict__ x, int cin,
                                                T* __restrict__ col) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ng * 27 * cin) return;
  const int c = (int)(t % cin);
  const int64_t gk = t / cin;
  const int32_t src = sr_src<RR>(nbr, lab, g0 + gk / 27, (int)(gk % 27));
  col[t] = src < 0 ? T(0) : x[(int64_t)src * cin + c];
}

// y[i] (depth l-1) = label L > 0 ? yg[L-1] : 0, ReLU applied if relu; four
// channels per thread (cout % 4 == 0).
__global__ __launch_bounds__(TB) void k_s2_rows_out(const int32_t* __restrict__ labels,
                                                    int64_t n_out, const float* __restrict__ yg,
                                                    int cout, int relu, float* __restrict__ y) {
  const int c4n = cout / 4;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_out * c4n) return;
  const int64_t i = t / c4n;
  const int c = 4 * (int)(t - i * c4n);
  const int32_t L = labels[i];
  float4 v = {0.f, 0.f, 0.f, 0.f};
  if (L > 0) v = *reinterpret_cast<const float4*>(yg + (int64_t)(L - 1) * cout + c);
  if (relu) v = float4{fmaxf(v.x, 0.f), fmaxf(v.y, 0.f), fmaxf(v.z, 0.f), fmaxf(v.w, 0.f)};
  *reinterpret_cast<float4*>(y + i * cout + c) = v;
}

// dyg[g] = dy[rows[g]], zero where ym[rows[g]] <= 0 (ym: the forward output
// through a fused ReLU, or null); T = bf16 rounds to nearest even.  Four
// channels per thread (cout % 4 == 0).
template <typename T>
__global__ __launch_bounds__(TB) void k_s2_dy_rows(const int32_t* __restrict__ rows, int64_t ng,
                                                   const float* __restrict__ dy,
                                                   const float* __restrict__ ym, int cout,
                                                   T* __restrict__ dyg) {
  const int c4n = cout / 4;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ng * c4n) return;
  const int64_t g = t / c4n;
  const int c = 4 * (int)(t - g * c4n);
  const int64_t src = (int64_t)rows[g] * cout + c;
  float4 v = *reinterpret_cast<const float4*>(dy + src);
  if (ym) {
    const float4 m = *reinterpret_cast<const float4*>(ym + src);
    v = float4{m.x > 0.f ? v.x : 0.f, m.y > 0.f ? v.y : 0.f, m.z > 0.f ? v.z : 0.f,
               m.w > 0.f ? v.w : 0.f};
  }
  T* o = dyg + g * cout + c;
  if constexpr (sizeof(T) == 2) {
    *reinterpret_cast<uint2*>(o) = uint2{bf16_rne(v.x) | ((uint32_t)bf16_rne(v.y) << 16),
                                         bf16_rne(v.z) | ((uint32_t)bf16_rne(v.w) << 16)};
  } else {
    *reinterpret_cast<float4*>(o) = v;
  }
}

// Expanded weight of the input gradient: wx[(o cout + co) 8 cin + c cin + ci]
// = W[c - 2o][ci][co] where c - 2o lies in {-1,0,1}^3 per axis, else 0
// (o, c: parent offset and child, x-bit 4, y-bit 2, z-bit 1).
template <typename T>
__global__ __launch_bounds__(TB) void k_s2_wx(const T* __restrict__ w, int cin, int cout,
                                              T* __restrict__ wx) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  const int64_t n = (int64_t)64 * cin * cout;
  if (t >= n) return;
  const int ci = (int)(t % cin);
  const int c = (int)((t / cin) % 8);
  const int co = (int)((t / (8 * cin)) % cout);
  const int o = (int)(t / ((int64_t)8 * cin * cout));
  int k = 0;
  bool ok = true;
#pragma unroll
  for (int a = 2; a >= 0; --a) {
    const int d = ((c >> a) & 1) - 2 * ((o >> a) & 1);
    ok = ok && d >= -1;
    k = 3 * k + (d + 1);
  }
  wx[t] = ok ? w[((int64_t)k * cin + ci) * cout + co] : T(0);
}

// D[h][o][:] = dyg[group of the parent neighbour at offset o in {0,1}^3] (0
// if absent), one 16-byte piece per thread; rows of rb bytes, rb % 16 == 0.
template <typename T>
__global__ __launch_bounds__(TB) void k_s2_dgather(const int32_t* __restrict__ nbr, int64_t G,
                                                   const T* __restrict__ dyg, int rb,
                                                   T* __restrict__ D) {
  const int np = rb / 16;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= G * 8 * np) return;
  const int pc = (int)(t % np);
  const int64_t ho = t / np;
  const int64_t h = ho / 8;
  const int o = (int)(ho % 8);
  const int32_t f = nbr[27 * h + ((o >> 2) + 1) * 9 + (((o >> 1) & 1) + 1) * 3 + ((o & 1) + 1)];
  uint4 v = {0u, 0u, 0u, 0u};
  if (f >= 0) v = *reinterpret_cast<const uint4*>((const char*)dyg + (int64_t)(f >> 3) * rb + 16 * pc);
  *reinterpret_cast<uint4*>((char*)D + ho * rb + 16 * pc) = v;
}

// Element-wise forms of k_s2_rows_out, k_s2_dy_rows and k_s2_dgather for
// channel counts or pointers that do not allow 16-byte accesses.
__global__ __launch_bounds__(TB) void k_s2_rows_out1(const int32_t* __restrict__ labels,
                                                     int64_t n_out, const float* __restrict__ yg,
                                                     int cout, int relu, float* __restrict__ y) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_out * cout) return;
  const int64_t i = t / cout;
  const int c = (int)(t - i * cout);
  const int32_t L = labels[i];
  const float v = L > 0 ? yg[(int64_t)(L - 1) * cout + c] : 0.f;
  y[t] = relu ? fmaxf(v, 0.f) : v;
}

template <typename T>
__global__ __launch_bounds__(TB) void k_s2_dy_rows1(const int32_t* __restrict__ rows, int64_t ng,
                                                    const float* __restrict__ dy,
                                                    const float* __restrict__ ym, int cout,
                                                    T* __restrict__ dyg) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ng * cout) return;
  const int64_t g = t / cout;
  const int c = (int)(t - g * cout);
  const int64_t src = (int64_t)rows[g] * cout + c;
  const float v = (ym && !(ym[src] > 0.f)) ? 0.f : dy[src];
  if constexpr (sizeof(T) == 2)
    dyg[t] = bf16_rne(v);
  else
    dyg[t] = v;
}

template <typename T>
__global__ __launch_bounds__(TB) void k_s2_dgather1(const int32_t* __restrict__ nbr, int64_t G,
                                                    const T* __restrict__ dyg, int cout,
                                                    T* __restrict__ D) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= G * 8 * cout) return;
  const int c = (int)(t % cout);
  const int64_t ho = t / cout;
  const int64_t h = ho / 8;
  const int o = (int)(ho % 8);
  const int32_t f = nbr[27 * h + ((o >> 2) + 1) * 9 + (((o >> 1) & 1) + 1) * 3 + ((o & 1) + 1)];
  D[t] = f >= 0 ? dyg[(int64_t)(f >> 3) * cout + c] : T(0);
}

// ---------------------------------------------------------------------------
// fp32 forward as an implicit GEMM on the matrix cores (k_s2_fwd), for cin
// and cout multiples of 16: no column buffer.  The MFMA computes the output
// transposed: A = W^T (16 output channels x reduction), B = the gathered
// inputs (reduction x 16 sibling groups), so lane (i, q) (i = lane % 16,
// q = lane / 16) supplies group i's input row at one tap, channels
// c0 + 4q .. c0 + 4q + 3, from one 16-byte load to four consecutive
// 16x16x4 MFMAs (channel 4q + s to the s-th), and holds the chunk's weights
// W[k][c][n0 + i] of its channel slots for all 27 taps in registers (read
// from a transposed copy wt[k][n][c], 16 bytes per tap).
// Child 0 of group g reaches, per axis, offset -1 (child 1 of the parent
// neighbour at -1), 0 and +1 (children 0 and 1 of its own parent's column),
// so the 27 taps read the children of the 8 parent neighbours at offsets
// {-1,0}^3; a lane keeps those 8 first-child rows of its group per row block
// and every tap is then a compile-time child offset.  Loads run 16 / RB - 1
// taps ahead of the MFMAs (a register ring), which covers the latency of
// the gathers (mostly L2 hits).
// A workgroup takes GT = 16 RB WM groups (a tile) and 16 WN output channels
// (a column block): wave w owns channels 16 (w % WN) and RB row blocks of 16
// groups.  Results go straight to the parents' rows (rows_of_label at depth
// l-1), ReLU applied if relu; the workgroups of column block 0 also zero the
// rows of empty depth-(l-1) octants, an equal share each.
// bf16 stays on the column buffer and GEMM: with one 16x16x32 MFMA per
// 16-byte gather, this kernel was bound by the vector-memory path (0.57 vs
// 0.41 ms for the 16-shape depth-7 64 -> 128 layer).
typedef float s2v4f __attribute__((ext_vector_type(4)));
typedef uint32_t s2v4u __attribute__((ext_vector_type(4)));

// wt[k][n][c] = w[k][c][n] (27 taps), so that a lane of k_s2_fwd reads its
// channels of one output column with one 16-byte load.
template <typename T>
__global__ __launch_bounds__(TB) void k_s2_wt(const T* __restrict__ w, int cin, int cout,
                                              T* __restrict__ wt) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= (int64_t)27 * cin * cout) return;
  const int c = (int)(t % cin);
  const int n = (int)((t / cin) % cout);
  const int64_t k = t / ((int64_t)cin * cout);
  wt[t] = w[(k * cin + c) * cout + n];
}

// Four 16x16x4 MFMAs, the s-th taking element s of a and b.
__device__ __forceinline__ s2v4f s2_mfma4(s2v4u a, s2v4u b, s2v4f c) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[s]), __uint_as_float(b[s]), c, 0, 0,
                                             0);
  return c;
}

template <int WN, int RB>
__global__ __launch_bounds__(TB) void k_s2_fwd(const int32_t* __restrict__ nbr, int64_t G,
                                               const void* __restrict__ xv, int cin,
                                               const void* __restrict__ wv, int cout,
                                               const int32_t* __restrict__ prow,
                                               const int32_t* __restrict__ labels, int64_t n_out,
                                               float* __restrict__ y, int relu, int xbytes,
                                               int wbytes, int ntiles, int gy) {
  constexpr int WAVES = TB / 64, WM = WAVES / WN;
  constexpr int CH = 16;                 // reduction channels per chunk
  constexpr int EPL = 4;                 // channels per lane per load
  constexpr int ES = 4;                  // element bytes
  constexpr int GT = 16 * RB * WM;       // groups per workgroup
  constexpr int PD = 16 / RB;            // taps of gathered loads in the ring
  static_assert(WN * WM == WAVES, "waves");
  // x through a buffer resource of xbytes bytes: offsets at or past the end
  // read zeros, which is how absent neighbours are read
  const __amdgpu_buffer_rsrc_t xr =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(xv), (short)0, xbytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t wr_ =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(wv), (short)0, wbytes, 0x00020000);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, q = lane >> 4;
  const int wn = wave % WN, wm = wave / WN;
  // workgroup -> (tile, column block): the workgroups of one XCD (dispatch
  // order modulo 8) take a contiguous run of tiles, all column blocks of a
  // tile in a row, so neighbouring groups' rows are gathered from one L2
  const int per = (int)(gridDim.x / 8), bid = (int)blockIdx.x;
  const int lin = gridDim.x % 8 == 0 ? (bid % 8) * per + bid / 8 : bid;
  if (lin >= ntiles * gy) return;  // uniform over the workgroup
  const int tile = lin / gy, cbk = lin % gy;
  const int n0 = cbk * 16 * WN + 16 * wn;
  const int64_t gb = (int64_t)tile * GT + (int64_t)wm * 16 * RB;

  // zero this workgroup's share of the rows of empty depth-(l-1) octants
  if (cbk == 0) {
    const int64_t r0 = n_out * tile / ntiles, r1 = n_out * (tile + 1) / ntiles;
    const int c4 = cout / 4, ne = (int)(r1 - r0) * c4;
    for (int e = tid; e < ne; e += TB) {
      const int64_t i = r0 + e / c4;
      if (labels[i] == 0)
        *reinterpret_cast<s2v4f*>(y + i * cout + 4 * (e % c4)) = s2v4f{0.f, 0.f, 0.f, 0.f};
    }
  }

  // byte offsets of this lane's channels in the first-child rows of the 8
  // parent neighbours at offsets {-1,0}^3 (index 4 ox + 2 oy + oz, o = 1 for
  // offset 0); 2^31 (past the end of x, read as zeros) if absent.  The tap's
  // child row and the chunk go into the scalar offset of each load.
  const int lane_cb = q * EPL * ES;  // this lane's byte offset within a chunk's channels
  uint32_t pbo[RB][8];
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    const int64_t g = gb + 16 * r + li;
#pragma unroll
    for (int o = 0; o < 8; ++o) {
      const int slot = ((o >> 2) & 1) * 9 + ((o >> 1) & 1) * 3 + (o & 1);
      const int32_t f = g < G ? nbr[27 * g + slot] : -1;
      pbo[r][o] = f < 0 ? 0x80000000u : (uint32_t)(f * cin * ES + lane_cb);
    }
  }
  // tap k = 9 (dx+1) + 3 (dy+1) + (dz+1): parent offset index and child row
  auto tap_o = [](int k) {
    const int dx = k / 9 - 1, dy = (k / 3) % 3 - 1, dz = k % 3 - 1;
    return 4 * (dx >= 0) + 2 * (dy >= 0) + (dz >= 0);
  };
  auto tap_c = [](int k) {
    const int dx = k / 9 - 1, dy = (k / 3) % 3 - 1, dz = k % 3 - 1;
    return 4 * (dx & 1) + 2 * (dy & 1) + (dz & 1);
  };

  s2v4f acc[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) acc[r] = s2v4f{0.f, 0.f, 0.f, 0.f};
  s2v4u wr[27];
  const uint32_t wlane = (uint32_t)((n0 + li) * cin * ES + lane_cb);

  for (int c0 = 0; c0 < cin; c0 += CH) {
    // the chunk's weights: wr[k] = W[k][c0 + EPL q + j][n0 + li], j < EPL,
    // one 16-byte load from the transposed copy wt[k][n][c]
#pragma unroll
    for (int k = 0; k < 27; ++k)
      wr[k] = __builtin_bit_cast(
          s2v4u, __builtin_amdgcn_raw_buffer_load_b128(wr_, wlane, (k * cout * cin + c0) * ES, 0));
    auto gload = [&](int r, int k) {
      return __builtin_bit_cast(
          s2v4u, __builtin_amdgcn_raw_buffer_load_b128(xr, pbo[r][tap_o(k)],
                                                       (tap_c(k) * cin + c0) * ES, 0));
    };
    // a ring of PD taps' loads: tap k + PD - 1 is issued before tap k's MFMAs
    s2v4u bv[PD][RB];
#pragma unroll
    for (int k = 0; k + 1 < PD; ++k)
#pragma unroll
      for (int r = 0; r < RB; ++r) bv[k][r] = gload(r, k);
#pragma unroll
    for (int k = 0; k < 27; ++k) {
      if (k + PD - 1 < 27) {
#pragma unroll
        for (int r = 0; r < RB; ++r) bv[(k + PD - 1) % PD][r] = gload(r, k + PD - 1);
      }
      __builtin_amdgcn_sched_barrier(0);  // PD - 1 taps of loads ahead, no more
#pragma unroll
      for (int r = 0; r < RB; ++r) acc[r] = s2_mfma4(wr[k], bv[k % PD][r], acc[r]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  // D[4q + j][i] = output channel n0 + 4q + j of group gb + 16 r + i
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    const int64_t g = gb + 16 * r + li;
    if (g < G) {
      s2v4f v = acc[r];
      if (relu) {
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = fmaxf(v[j], 0.f);
      }
      *reinterpret_cast<s2v4f*>(y + (int64_t)prow[g] * cout + n0 + 4 * q) = v;
    }
  }
}

// Stride-4 input gradient.  Depth-l row n = 8h + c is child c of the
// depth-(l-1) octant q with label h + 1, itself child a of its parent P.  Per
// axis, n's position 4P + 2a + c is read by exactly one output when
// 2a + c != 2: output P (tap offset c) when a = 0, output P + 1 (offset -1)
// when a = 1 and c = 1.  So the eight rows of group h all read the same
// output, P's neighbour at offset a (through P's depth-(l-1) group table),
// and dx[n][ci] = sum_co W[d][ci][co] dyg[p][co]; rows that no output reads
// get 0.  One thread per (row, input channel), four output channels per step.
template <typename T>
__global__ __launch_bounds__(TB) void k_s4_dx(const int32_t* __restrict__ rows1,
                                              const int32_t* __restrict__ nbr1, int64_t n_in,
                                              const T* __restrict__ dyg, const T* __restrict__ w,
                                              int cin, int cout, float* __restrict__ dx) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_in * cin) return;
  const int64_t n = t / cin;
  const int ci = (int)(t - n * cin);
  const int c = (int)(n & 7);
  const int32_t rq = rows1[n >> 3];
  const int a = rq & 7;
  const int axx = a >> 2, ayy = (a >> 1) & 1, azz = a & 1;
  const int cx = c >> 2, cy = (c >> 1) & 1, cz = c & 1;
  float acc = 0.f;
  if (!((axx && !cx) || (ayy && !cy) || (azz && !cz))) {
    const int32_t f = nbr1[27 * (int64_t)(rq >> 3) + (axx + 1) * 9 + (ayy + 1) * 3 + (azz + 1)];
    if (f >= 0) {
      const int64_t p = f >> 3;
      const int dxo = axx ? -1 : cx, dyo = ayy ? -1 : cy, dzo = azz ? -1 : cz;
      const int k = (dxo + 1) * 9 + (dyo + 1) * 3 + (dzo + 1);
      const T* wr = w + ((int64_t)k * cin + ci) * cout;
      const T* gr = dyg + p * cout;
      for (int co = 0; co < cout; ++co) acc += to_f(wr[co]) * to_f(gr[co]);
    }
  }
  dx[t] = acc;
}

// The same for fp32 with cin and cout multiples of 4: one thread per (row,
// 4 input channels), 4 x 4 weight blocks and 4 upstream channels per step.
__global__ __launch_bounds__(TB) void k_s4_dx4(const int32_t* __restrict__ rows1,
                                               const int32_t* __restrict__ nbr1, int64_t n_in,
                                               const float* __restrict__ dyg,
                                               const float* __restrict__ w, int cin, int cout,
                                               float* __restrict__ dx) {
  const int cq = cin / 4;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_in * cq) return;
  const int64_t n = t / cq;
  const int ci = 4 * (int)(t - n * cq);
  const int c = (int)(n & 7);
  const int32_t rq = rows1[n >> 3];
  const int a = rq & 7;
  const int axx = a >> 2, ayy = (a >> 1) & 1, azz = a & 1;
  const int cx = c >> 2, cy = (c >> 1) & 1, cz = c & 1;
  float4 acc = {0.f, 0.f, 0.f, 0.f};
  if (!((axx && !cx) || (ayy && !cy) || (azz && !cz))) {
    const int32_t f = nbr1[27 * (int64_t)(rq >> 3) + (axx + 1) * 9 + (ayy + 1) * 3 + (azz + 1)];
    if (f >= 0) {
      const int64_t p = f >> 3;
      const int dxo = axx ? -1 : cx, dyo = ayy ? -1 : cy, dzo = azz ? -1 : cz;
      const int k = (dxo + 1) * 9 + (dyo + 1) * 3 + (dzo + 1);
      const float* wr = w + ((int64_t)k * cin + ci) * cout;
      const float4* gr = reinterpret_cast<const float4*>(dyg + p * cout);
      for (int co = 0; co < cout; co += 4) {
        const float4 g = gr[co / 4];
        const float4 w0 = *reinterpret_cast<const float4*>(wr + co);
        const float4 w1 = *reinterpret_cast<const float4*>(wr + cout + co);
        const float4 w2 = *reinterpret_cast<const float4*>(wr + 2 * cout + co);
        const float4 w3 = *reinterpret_cast<const float4*>(wr + 3 * cout + co);
        acc.x += w0.x * g.x + w0.y * g.y + w0.z * g.z + w0.w * g.w;
        acc.y += w1.x * g.x + w1.y * g.y + w1.z * g.z + w1.w * g.w;
        acc.z += w2.x * g.x + w2.y * g.y + w2.z * g.z + w2.w * g.w;
        acc.w += w3.x * g.x + w3.y * g.y + w3.z * g.z + w3.w * g.w;
      }
    }
  }
  *reinterpret_cast<float4*>(dx + n * cin + ci) = acc;
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

// The same for `batch` GEMMs whose operands lie sa, sb and sd elements apart.
oc_status gemm_batched(hipStream_t s, bool ta, bool tb, int64_t m, int64_t n, int64_t k,
                       const void* A, rocblas_datatype at, int64_t lda, int64_t sa, const void* B,
                       rocblas_datatype bt, int64_t ldb, int64_t sb, float beta, float* D,
                       int64_t ldd, int64_t sd, int64_t batch) {
  if (m == 0 || n == 0 || batch == 0) return OC_OK;
  if (m > INT32_MAX || n > INT32_MAX || k > INT32_MAX || lda > INT32_MAX || ldb > INT32_MAX ||
      batch > INT32_MAX)
    return oc::fail(OC_ERR_UNSUPPORTED, "stride-2 convolution: GEMM size beyond 32 bits");
  std::lock_guard<std::mutex> lk(g_blas_mu);
  rocblas_handle h;
  oc_status st = blas_for(s, &h);
  if (st != OC_OK) return st;
  const float alpha = 1.f;
  const rocblas_status r = rocblas_gemm_strided_batched_ex(
      h, ta ? rocblas_operation_transpose : rocblas_operation_none,
      tb ? rocblas_operation_transpose : rocblas_operation_none, (rocblas_int)m, (rocblas_int)n,
      (rocblas_int)k, &alpha, A, at, (rocblas_int)lda, sa, B, bt, (rocblas_int)ldb, sb, &beta, D,
      rocblas_datatype_f32_r, (rocblas_int)ldd, sd, D, rocblas_datatype_f32_r, (rocblas_int)ldd, sd,
      (rocblas_int)batch, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0);
  if (r != rocblas_status_success)
    return oc::fail(OC_ERR_DEVICE, "stride-2 convolution: batched GEMM failed (%d)", (int)r);
  return OC_OK;
}

// out[e] = sum_{b < nb} part[b][e] in the order b = 0, 1, ...
__global__ __launch_bounds__(TB) void k_s2_sum(const float* __restrict__ part, int nb, int64_t n,
                                               float* __restrict__ out) {
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e >= n) return;
  float v = 0.f;
  for (int b = 0; b < nb; ++b) v += part[b * n + e];
  out[e] = v;
}

// Batches of the weight gradient's GEMM: the groups of a column-buffer chunk
// are split into DW_BATCH runs whose products go to separate partial sums (a
// single GEMM over the groups has too few output tiles to fill the GPU).
constexpr int DW_BATCH = 8;

struct S2Shape {
  int64_t G, n_in, n_out;
  int64_t kc;  // 27 cin
  int64_t gc;  // groups per column-buffer chunk
};

S2Shape s2_shape(const oc_octree* t, int l, int r, int cin, size_t elsize) {
  S2Shape h;
  h.G = t->M[l - r];
  h.n_in = t->N[l];
  h.n_out = t->N[l - r];
  h.kc = 27 * (int64_t)cin;
  h.gc = std::max<int64_t>(1, std::min<int64_t>(h.G, (int64_t)(COL_CAP / (h.kc * elsize))));
  return h;
}

// Shapes the implicit-GEMM forward takes (the rest use the column buffer).
bool s2_fwd_direct(const oc_octree* t, int l, int cin, int cout, bool bf16) {
  return !bf16 && t->M[l - 1] > 0 && cin % 16 == 0 && cout % 16 == 0 &&
         (int64_t)t->N[l] * cin * 4 < ((int64_t)1 << 31);
}

template <int WN, int RB>
void launch_s2_fwd(const oc_octree* t, int l, const void* x, int cin, const void* w, int cout,
                   float* y, int relu, void* ws, hipStream_t s) {
  const int64_t nw = (int64_t)27 * cin * cout;
  oc::launch(k_s2_wt<float>, dim3((unsigned)oc::cdiv(nw, TB)), dim3(TB), 0, s,
                     (const float*)w, cin, cout, (float*)ws);
  w = ws;
  const int64_t G = t->M[l - 1];
  constexpr int GT = 16 * RB * (TB / 64 / WN);
  const int ntiles = (int)oc::cdiv(G, GT), gy = cout / (16 * WN);
  const int64_t nwg = (int64_t)ntiles * gy;
  const dim3 grid((unsigned)(nwg >= 8 ? oc::cdiv(nwg, 8) * 8 : nwg));
  oc::launch((k_s2_fwd<WN, RB>), grid, dim3(TB), 0, s, (const int32_t*)t->nbr[l], G,
                     x, cin, w, cout, (const int32_t*)t->rows[l - 1],
                     (const int32_t*)t->labels[l - 1], t->N[l - 1], y, relu,
                     (int)(t->N[l] * cin * 4), (int)(nw * 4), ntiles, gy);
}

}  // namespace

namespace oc {

size_t conv_s2_fwd_ws(const oc_octree* t, int l, int r, int cin, int cout, bool bf16) {
  const S2Shape h = s2_shape(t, l, r, cin, bf16 ? 2 : 4);
  if (h.G == 0) return 0;
  if (r == 1 && s2_fwd_direct(t, l, cin, cout, bf16))  // the transposed weights
    return align256((size_t)27 * cin * cout * 4);
  return align256((size_t)h.gc * h.kc * (bf16 ? 2 : 4)) + align256((size_t)h.G * cout * 4);
}

size_t conv_s2_bwd_ws(const oc_octree* t, int l, int r, int cin, int cout, bool bf16, bool dx,
                      bool dw) {
  const size_t es = bf16 ? 2 : 4;
  const S2Shape h = s2_shape(t, l, r, cin, es);
  if (h.G == 0 || (!dx && !dw)) return 0;
  const size_t b = align256((size_t)h.G * cout * es);                         // dY_g
  const size_t a = !dx ? 0
                   : r == 2 ? 0                                               // (stride 4: none)
                            : align256((size_t)64 * cin * cout * es) +        // Wx
                                  align256((size_t)h.G * 8 * cout * es);      // D
  const size_t c = dw ? align256((size_t)h.gc * h.kc * es) +                 // Col chunk
                            align256((size_t)DW_BATCH * h.kc * cout * 4)      // partial dW
                      : 0;
  return b + std::max(a, c);
}

namespace {

// Column buffer of ng groups from g0, 16-byte pieces when the rows allow;
// r = 1: nbr is the depth-l table; r = 2: the depth-(l-1) table with the
// depth-(l-1) labels lab.
template <int RR>
void launch_col_r(hipStream_t s, const int32_t* nbr, const int32_t* lab, int64_t g0, int64_t ng,
                  const void* x, int cin, bool bf16, void* col) {
  const int rb = cin * (bf16 ? 2 : 4);
  if (rb % 16 == 0) {
    const int64_t nt = ng * 27 * (rb / 16);
    if (bf16)
      oc::launch((k_s2_col<uint16_t, RR>), dim3(grid_for(nt)), dim3(TB), 0, s, nbr, lab,
                         g0, ng, (const uint16_t*)x, rb, (uint16_t*)col);
    else
      oc::launch((k_s2_col<float, RR>), dim3(grid_for(nt)), dim3(TB), 0, s, nbr, lab, g0,
                         ng, (const float*)x, rb, (float*)col);
  } else {
    const int64_t nt = ng * 27 * cin;
    if (bf16)
      oc::launch((k_s2_col1<uint16_t, RR>), dim3(grid_for(nt)), dim3(TB), 0, s, nbr, lab,
                         g0, ng, (const uint16_t*)x, cin, (uint16_t*)col);
    else
      oc::launch((k_s2_col1<float, RR>), dim3(grid_for(nt)), dim3(TB), 0, s, nbr, lab,
                         g0, ng, (const float*)x, cin, (float*)col);
  }
}

void launch_col(hipStream_t s, const oc_octree* t, int l, int r, int64_t g0, int64_t ng,
                const void* x, int cin, bool bf16, void* col) {
  if (r == 1)
    launch_col_r<1>(s, (const int32_t*)t->nbr[l], nullptr, g0, ng, x, cin, bf16, col);
  else
    launch_col_r<2>(s, (const int32_t*)t->nbr[l - 1], (const int32_t*)t->labels[l - 1], g0, ng, x,
                    cin, bf16, col);
}

}  // namespace

oc_status conv_s2_fwd(const oc_octree* t, int l, int r, const void* x, int cin, const void* w,
                      int cout, bool bf16, float* y, int relu, void* ws, hipStream_t s) {
  PassEvents ev(s);
  if (r == 1 && s2_fwd_direct(t, l, cin, cout, bf16)) {
    if ((uintptr_t)x % 16 != 0 || (uintptr_t)y % 16 != 0)
      return fail(OC_ERR_ARG, "oc_conv_fwd: stride 2 needs 16-byte aligned x and y");
    // output channels per workgroup: 16 WN; row blocks per wave: the most
    // that still gives two workgroups per compute unit
    const int wn = cout % 64 == 0 ? 4 : cout % 32 == 0 ? 2 : 1;
    const int64_t G = t->M[l - 1], gy = cout / (16 * wn), wm = 4 / wn;
    int rb = 4;
    while (rb > 1 && oc::cdiv(G, 16 * rb * wm) * gy < 2 * (int64_t)cu_count()) rb /= 2;
#define OC_S2F(WN_, RB_)                                                  \
  if (wn == WN_ && rb == RB_) {                                           \
    launch_s2_fwd<WN_, RB_>(t, l, x, cin, w, cout, y, relu, ws, s);       \
    return OC_OK;                                                         \
  }
    OC_S2F(4, 4) OC_S2F(4, 2) OC_S2F(4, 1) OC_S2F(2, 4) OC_S2F(2, 2) OC_S2F(2, 1)
    OC_S2F(1, 4) OC_S2F(1, 2) OC_S2F(1, 1)
#undef OC_S2F
    return fail(OC_ERR_UNSUPPORTED, "stride-2 forward: no kernel for %d -> %d", cin, cout);
  }
  const S2Shape h = s2_shape(t, l, r, cin, bf16 ? 2 : 4);
  const int32_t* nbr = t->nbr[l];
  char* p = (char*)ws;
  void* col = p;
  float* yg = (float*)(p + (h.G ? align256((size_t)h.gc * h.kc * (bf16 ? 2 : 4)) : 0));
  const rocblas_datatype dt = bf16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
  for (int64_t g0 = 0; g0 < h.G; g0 += h.gc) {
    const int64_t ng = std::min<int64_t>(h.gc, h.G - g0);
    launch_col(s, t, l, r, g0, ng, x, cin, bf16, col);
    // yg^T [cout][ng] = W^T-view [cout][27 cin] x Col^T-view [27 cin][ng] (column-major)
    oc_status st = gemm(s, false, false, cout, ng, h.kc, w, dt, cout, col, dt, h.kc, 0.f,
                        yg + g0 * cout, cout);
    if (st != OC_OK) return st;
  }
  if (cout % 4 == 0 && (uintptr_t)y % 16 == 0)
    oc::launch(k_s2_rows_out, dim3(grid_for(h.n_out * (cout / 4))), dim3(TB), 0, s,
                       (const int32_t*)t->labels[l - r], h.n_out, (const float*)yg, cout, relu, y);
  else
    oc::launch(k_s2_rows_out1, dim3(grid_for(h.n_out * cout)), dim3(TB), 0, s,
                       (const int32_t*)t->labels[l - r], h.n_out, (const float*)yg, cout, relu, y);
  return OC_OK;
}

oc_status conv_s2_bwd(const oc_octree* t, int l, int r, const void* x, int cin, const void* w,
                      int cout, bool bf16, const float* ym, const float* dy, float* dx, float* dw,
                      void* ws, hipStream_t s) {
  PassEvents ev(s);
  const size_t es = bf16 ? 2 : 4;
  const S2Shape h = s2_shape(t, l, r, cin, es);
  const int64_t entries = h.kc * cout;
  if (h.G == 0) {
    if (dx && h.n_in > 0) fill_u32(dx, 0u, h.n_in * cin, s);
    if (dw) fill_u32(dw, 0u, entries, s);
    return OC_OK;
  }
  const int32_t* nbr = t->nbr[l];
  const rocblas_datatype dt = bf16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
  char* p = (char*)ws;
  void* dyg = p;
  p += align256((size_t)h.G * cout * es);
  const bool vec = cout % 4 == 0 && (uintptr_t)dy % 16 == 0 && (uintptr_t)ym % 16 == 0;
  const int32_t* prow = (const int32_t*)t->rows[l - r];
  if (vec && bf16)
    oc::launch(k_s2_dy_rows<uint16_t>, dim3(grid_for(h.G * (cout / 4))), dim3(TB), 0, s,
                       prow, h.G, dy, ym, cout, (uint16_t*)dyg);
  else if (vec)
    oc::launch(k_s2_dy_rows<float>, dim3(grid_for(h.G * (cout / 4))), dim3(TB), 0, s,
                       prow, h.G, dy, ym, cout, (float*)dyg);
  else if (bf16)
    oc::launch(k_s2_dy_rows1<uint16_t>, dim3(grid_for(h.G * cout)), dim3(TB), 0, s, prow,
                       h.G, dy, ym, cout, (uint16_t*)dyg);
  else
    oc::launch(k_s2_dy_rows1<float>, dim3(grid_for(h.G * cout)), dim3(TB), 0, s, prow,
                       h.G, dy, ym, cout, (float*)dyg);
  if (dx && r == 2) {
    const int64_t nt = h.n_in * (int64_t)cin;
    if (bf16)
      oc::launch(k_s4_dx<uint16_t>, dim3(grid_for(nt)), dim3(TB), 0, s,
                         (const int32_t*)t->rows[l - 1], (const int32_t*)t->nbr[l - 1], h.n_in,
                         (const uint16_t*)dyg, (const uint16_t*)w, cin, cout, dx);
    else if (cin % 4 == 0 && cout % 4 == 0 && (uintptr_t)w % 16 == 0 && (uintptr_t)dx % 16 == 0 &&
             (uintptr_t)dyg % 16 == 0)
      oc::launch(k_s4_dx4, dim3(grid_for(nt / 4)), dim3(TB), 0, s,
                         (const int32_t*)t->rows[l - 1], (const int32_t*)t->nbr[l - 1], h.n_in,
                         (const float*)dyg, (const float*)w, cin, cout, dx);
    else
      oc::launch(k_s4_dx<float>, dim3(grid_for(nt)), dim3(TB), 0, s,
                         (const int32_t*)t->rows[l - 1], (const int32_t*)t->nbr[l - 1], h.n_in,
                         (const float*)dyg, (const float*)w, cin, cout, dx);
  } else if (dx) {
    void* wx = p;
    void* D = p + align256((size_t)64 * cin * cout * es);
    const int64_t nw = (int64_t)64 * cin * cout;
    const int rb = (int)(cout * es);  // bytes of a dY_g row (16-byte aligned rows when rb % 16 == 0)
    const unsigned gd = rb % 16 == 0 ? grid_for(h.G * 8 * (int64_t)(rb / 16)) : grid_for(h.G * 8 * (int64_t)cout);
    if (bf16) {
      oc::launch(k_s2_wx<uint16_t>, dim3(grid_for(nw)), dim3(TB), 0, s,
                         (const uint16_t*)w, cin, cout, (uint16_t*)wx);
      if (rb % 16 == 0)
        oc::launch(k_s2_dgather<uint16_t>, dim3(gd), dim3(TB), 0, s, nbr, h.G,
                           (const uint16_t*)dyg, rb, (uint16_t*)D);
      else
        oc::launch(k_s2_dgather1<uint16_t>, dim3(gd), dim3(TB), 0, s, nbr, h.G,
                           (const uint16_t*)dyg, cout, (uint16_t*)D);
    } else {
      oc::launch(k_s2_wx<float>, dim3(grid_for(nw)), dim3(TB), 0, s, (const float*)w, cin,
                         cout, (float*)wx);
      if (rb % 16 == 0)
        oc::launch(k_s2_dgather<float>, dim3(gd), dim3(TB), 0, s, nbr, h.G,
                           (const float*)dyg, rb, (float*)D);
      else
        oc::launch(k_s2_dgather1<float>, dim3(gd), dim3(TB), 0, s, nbr, h.G,
                           (const float*)dyg, cout, (float*)D);
    }
    // dX-view^T [8 cin][G] = Wx-view^T [8 cin][8 cout] x D-view^T [8 cout][G] (column-major)
    oc_status st = gemm(s, false, false, 8 * (int64_t)cin, h.G, 8 * (int64_t)cout, wx, dt,
                        8 * (int64_t)cin, D, dt, 8 * (int64_t)cout, 0.f, dx, 8 * (int64_t)cin);
    if (st != OC_OK) return st;
  }
  if (dw) {
    void* col = p;
    float* pw = (float*)(p + align256((size_t)h.gc * h.kc * es));  // [DW_BATCH][27 cin][cout]
    const int64_t E = h.kc * cout;
    fill_u32(pw, 0u, DW_BATCH * E, s);
    for (int64_t g0 = 0; g0 < h.G; g0 += h.gc) {
      const int64_t ng = std::min<int64_t>(h.gc, h.G - g0);
      launch_col(s, t, l, r, g0, ng, x, cin, bf16, col);
      // partial b: dW^T [cout][27 cin] += dyg^T-view [cout][sz] x Col-view^T [sz][27 cin]
      // over groups g0 + b sz .. g0 + (b+1) sz; the rest of the chunk adds to partial 0
      const int64_t sz = ng / DW_BATCH, done = sz * DW_BATCH;
      const char* dy0 = (const char*)dyg + g0 * cout * es;
      oc_status st = gemm_batched(s, false, true, cout, h.kc, sz, dy0, dt, cout, sz * cout,
                                  col, dt, h.kc, sz * h.kc, 1.f, pw, cout, E,
                                  sz > 0 ? DW_BATCH : 0);
      if (st != OC_OK) return st;
      if (ng > done) {
        st = gemm(s, false, true, cout, h.kc, ng - done, dy0 + done * cout * es, dt, cout,
                  (const char*)col + done * h.kc * es, dt, h.kc, 1.f, pw, cout);
        if (st != OC_OK) return st;
      }
    }
    oc::launch(k_s2_sum, dim3(grid_for(E)), dim3(TB), 0, s, (const float*)pw, DW_BATCH, E,
                       dw);
  }
  return OC_OK;
}

}  // namespace oc
