// Strided octree convolution, K = 3, stride 2^r for any r >= 1 (Sec. 3.2,
// the stride-2 paragraphs and the stride-2^r remark), forward and both
// gradients, as implicit GEMMs on the matrix cores: the operand rows are
// gathered straight from the feature maps into LDS tiles, with no column
// buffer and no library GEMM.
//
// Geometry.  Output p is the p-th non-empty octant of depth l-r (coordinates
// P); the convolution is evaluated at depth-l position 2^r P and written to
// p's row of depth l-r; rows of empty depth-(l-r) octants are 0.  Per axis,
// tap offset d in {-1, 0, 1} reaches depth-l position 2^r P + d = 2 Q + c:
//   d = -1:  Q = 2^(r-1) P - 1, child c = 1
//   d =  0:  Q = 2^(r-1) P,     child c = 0
//   d = +1:  Q = 2^(r-1) P,     child c = 1
// so the 27 taps read children of the eight depth-(l-1) octants
// Q_o = 2^(r-1) P + a, a in {-1, 0}^3, indexed o = 4 [ax = 0] + 2 [ay = 0] +
// [az = 0]; the child is a compile-time function of the tap.  The table
// tab[p][o] holds the first-child row (depth l) of Q_o, or -1 when Q_o is
// outside the cube or empty.  For r = 1, Q_o is p's neighbour at parent
// offset a, read from the depth-l group table.  For r >= 2, Q_o descends from
// p's neighbour N_a at offset a (whose first child at depth l-r+1 the
// depth-(l-r+1) group table gives) through child (a = -1 ? 1 : 0) per axis at
// every depth l-r+1 .. l-1, following the labels.
//
// Passes (G = M_{l-r} outputs; dyg[p] = dy at p's row of depth l-r, masked by
// the ReLU when the forward fused one, rounded to bf16 for bf16 layers):
//   forward         y[row(p)] = sum_k x[src(p,k)] W[k]              (k_sr_mm, FWD)
//   input gradient  r = 1: each depth-l row 8h + c (child c of group h) is
//                   read by the outputs at parent offsets o in {0,1}^3 from
//                   h's parent with o_a <= c_a per axis, through tap
//                   c - 2o; so dx[8h + c] = sum over those o of
//                   dyg[n_o(h)] W[c - 2o]^T, a gathered GEMM per child class
//                   c (k_sr_mm, DX1), every row written once, no atomics.
//                   r >= 2: each depth-l row is read by at most one (p, k)
//                   (per axis only d = 0 at 2^r P, d = 1 at 2^r P + 1 and
//                   d = -1 at 2^r P - 1 reach it), so dx[src(p,k)] =
//                   dyg[p] W[k]^T is scattered without conflicts over a
//                   zeroed dx (k_sr_mm, DXS).
//   weight gradient dW[k] = sum_p x[src(p,k)]^T dyg[p]: reduction over the
//                   outputs, ranges of them in parallel, partial sums added
//                   in a fixed order (k_sr_dw).
// Every result is reproducible bit for bit (no floating-point atomics).
//
// Matrix cores.  fp32: v_mfma_f32_16x16x4_f32, four in a row over the four
// channels of one 16-byte operand piece.  bf16: v_mfma_f32_16x16x32_bf16, one
// per 16-byte piece.  Either way a piece of 64 bytes of a row is the
// reduction chunk (16 fp32 or 32 bf16 channels).  Operands are staged in LDS
// tiles of 64-byte rows (80-byte pitch) in double buffers: the next chunk's
// global loads are in flight while the current one is multiplied.  Absent
// rows, and channels or columns past the end, load zeros through
// buffer-resource range checks (offsets past the buffer's size read 0).
#include <algorithm>

#include "common.h"
#include "conv_sr.h"
#include "conv_cin.h"

namespace {

constexpr int TB = 256;
constexpr int LROW = 80;  // LDS bytes per tile row: 64 bytes of data + 16 of padding
constexpr uint32_t OOB = 0x80000000u;  // a buffer offset past every buffer: reads 0

typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* p, int64_t bytes) {
  const int32_t n = bytes >= INT32_MAX ? INT32_MAX : (int32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, n, 0x00020000);
}
__device__ __forceinline__ v4u bload16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(v4u, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ uint32_t bload4(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0);
}
__device__ __forceinline__ uint16_t bload2(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0);
}

// One 64-byte reduction chunk: a and b are this lane's 16-byte pieces.
__device__ __forceinline__ v4f mma(v4u a, v4u b, v4f c, float) {
#pragma unroll
  for (int s = 0; s < 4; ++s)
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[s]), __uint_as_float(b[s]), c, 0,
                                             0, 0);
  return c;
}
__device__ __forceinline__ v4f mma(v4u a, v4u b, v4f c, uint16_t) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(v8bf, a),
                                                  __builtin_bit_cast(v8bf, b), c, 0, 0, 0);
}

// Tap k = 9 (dx+1) + 3 (dy+1) + (dz+1): the depth-(l-1) octant index o and
// the child it reads (see the file comment).
__host__ __device__ constexpr int tap_o(int k) { return oc::sr_tap_o(k); }
__host__ __device__ constexpr int tap_c(int k) { return oc::sr_tap_c(k); }

// r = 1 input gradient: the j-th subset o of child class c (bits of j
// deposited on the set bits of c), the tap c - 2o and the group-table column
// of parent offset +o.
__device__ __forceinline__ int subset(int c, int j) {
  int o = 0, b = 0;
#pragma unroll
  for (int a = 0; a < 3; ++a)
    if ((c >> a) & 1) {
      if ((j >> b) & 1) o |= 1 << a;
      ++b;
    }
  return o;
}
__device__ __forceinline__ int dx1_tap(int c, int o) {
  int k = 0;
#pragma unroll
  for (int a = 2; a >= 0; --a) k = 3 * k + (((c >> a) & 1) - 2 * ((o >> a) & 1) + 1);
  return k;
}
__host__ __device__ constexpr int up_col(int o) {  // nbr column of parent offset +o, o in {0,1}^3
  return ((o >> 2) + 1) * 9 + (((o >> 1) & 1) + 1) * 3 + ((o & 1) + 1);
}

// ---------------------------------------------------------------------------
// The table tab[p][o] (see the file comment).
__global__ __launch_bounds__(TB) void k_sr_table(const int32_t* __restrict__ nbr, int64_t G, int r,
                                                 oc::SrLabels L, int32_t* __restrict__ tab) {
  const int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (e >= G * 8) return;
  tab[e] = oc::sr_first_child(nbr, L, e >> 3, (int)(e & 7), r);
}

// ---------------------------------------------------------------------------
// Implicit GEMM over gathered rows:
//   out[row(m, ...)][n] = sum_slots sum_c A[arow(m, slot)][c] B[slot][n][c]
// MODE_FWD: m = output p, slots = the 27 taps, arow = src(p, k) (tab), B =
//   the weights transposed to [27][cout][cin], row(m) = orow[m] (p's row of
//   depth l-r), ReLU optional.
// MODE_DX1: m = group h of depth l, class c = blockIdx.z, slots = the subsets
//   o of c, arow = the output group at parent offset +o (nbr), B = W[c - 2o]
//   as [cin][cout] (the weights' own layout), row = 8h + c.
// MODE_DXS: m = output p, slots = the 27 taps, arow = p, B = W[k] as
//   [cin][cout], row = src(p, k) for each tap separately (stored after the
//   tap's last chunk), skipped when absent.
// A workgroup is WGM x WGN waves; a wave owns WR x WC blocks of 16 rows x 16
// columns, so one LDS read of A feeds WC MFMA groups and one of B feeds WR.
// A stage is KS consecutive (slot, chunk) steps: its global loads are issued
// a stage ahead, and one barrier per stage separates the LDS buffers.
enum { MODE_FWD = 0, MODE_DX1 = 1, MODE_DXS = 2 };

struct MmArgs {
  const void* a;
  int64_t a_bytes;  // A rows [..][C] of T
  const void* b;
  int64_t b_bytes;  // [27][N][C] of T
  float* out;
  const int32_t* tab;   // FWD, DXS: [M][8]; DX1: the depth-l group table [M][27]
  const int32_t* orow;  // FWD: output rows
  int64_t M;
  int C, N, relu, vec;  // vec: C * sizeof(T) % 16 == 0 and aligned buffers (16-byte pieces)
};

template <typename T, int MODE, int WGM, int WGN, int WR, int WC, int KS>
__global__ __launch_bounds__(TB) void k_sr_mm(MmArgs g) {
  static_assert(WGM * WGN * 64 == TB, "waves");
  constexpr int BM = 16 * WR * WGM, BN = 16 * WC * WGN;
  constexpr int ES = sizeof(T), EPP = 16 / ES, KC = 64 / ES;  // elements per piece, per chunk
  constexpr int APT = BM * 4 / TB, BPT = (BN * 4 + TB - 1) / TB;  // pieces per thread
  static_assert(BM * 4 % TB == 0, "A pieces");
  __shared__ __attribute__((aligned(16))) char lA[2][KS][BM * LROW];
  __shared__ __attribute__((aligned(16))) char lB[2][KS][BN * LROW];
  __shared__ int32_t ltab[BM][8];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, q = lane >> 4;
  const int wm = wave / WGN, wn = wave % WGN;
  const int64_t m0 = (int64_t)blockIdx.x * BM;
  const int n0 = blockIdx.y * BN;
  const int cls = blockIdx.z;
  const int64_t M = g.M;
  const int C = g.C, N = g.N;
  const __amdgpu_buffer_rsrc_t ra = rsrc(g.a, g.a_bytes), rb = rsrc(g.b, g.b_bytes);

  for (int e = tid; e < BM * 8; e += TB) {
    const int mm = e >> 3, o = e & 7;
    const int64_t m = m0 + mm;
    int32_t v = -1;
    if (m < M) {
      if constexpr (MODE == MODE_DX1) {
        const int32_t f = g.tab[27 * m + up_col(o)];
        v = f < 0 ? -1 : f >> 3;
      } else {
        v = g.tab[8 * m + o];
      }
    }
    ltab[mm][o] = v;
  }
  __syncthreads();

  const int nslot = MODE == MODE_DX1 ? 1 << __builtin_popcount(cls) : 27;
  const int nch = (C + KC - 1) / KC;
  const int nsteps = nslot * nch;

  // A row (index into the A source) of tile row mm at slot j, or -1
  auto arow = [&](int mm, int j) -> int64_t {
    if constexpr (MODE == MODE_FWD) {
      const int32_t f = ltab[mm][tap_o(j)];
      return f < 0 ? -1 : (int64_t)f + tap_c(j);
    } else if constexpr (MODE == MODE_DX1) {
      return ltab[mm][subset(cls, j)];
    } else {
      return m0 + mm < M ? m0 + mm : -1;
    }
  };
  auto btap = [&](int j) -> int { return MODE == MODE_DX1 ? dx1_tap(cls, subset(cls, j)) : j; };

  v4u pa[KS][APT], pb[KS][BPT];
  // global loads of step t into pa, pb (zeros past the last step)
  auto load = [&](int t, v4u (&pa)[APT], v4u (&pb)[BPT]) {
    const bool live = t < nsteps;
    const int j = live ? t / nch : 0, c0 = (t - j * nch) * KC;
#pragma unroll
    for (int u = 0; u < APT; ++u) {
      const int e = tid + TB * u, mm = e >> 2, part = e & 3;
      const int c = c0 + part * EPP;
      const int64_t row = live ? arow(mm, j) : -1;
      if (g.vec) {
        const uint32_t off = row >= 0 && c < C ? (uint32_t)((row * C + c) * ES) : OOB;
        pa[u] = bload16(ra, off);
      } else {
        v4u v = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int i = 0; i < EPP; ++i) {
          const uint32_t off = row >= 0 && c + i < C ? (uint32_t)((row * C + c + i) * ES) : OOB;
          if constexpr (ES == 4) {
            v[i] = bload4(ra, off);
          } else {
            v[i / 2] |= (uint32_t)bload2(ra, off) << (16 * (i & 1));
          }
        }
        pa[u] = v;
      }
    }
    const int64_t bbase = (int64_t)btap(j) * N;
#pragma unroll
    for (int u = 0; u < BPT; ++u) {
      const int e = tid + TB * u, nn = e >> 2, part = e & 3;
      const int c = c0 + part * EPP, n = n0 + nn;
      const bool ok = live && e < BN * 4 && n < N;
      if (g.vec) {
        const uint32_t off = ok && c < C ? (uint32_t)(((bbase + n) * C + c) * ES) : OOB;
        pb[u] = bload16(rb, off);
      } else {
        v4u v = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int i = 0; i < EPP; ++i) {
          const uint32_t off =
              ok && c + i < C ? (uint32_t)(((bbase + n) * C + c + i) * ES) : OOB;
          if constexpr (ES == 4) {
            v[i] = bload4(rb, off);
          } else {
            v[i / 2] |= (uint32_t)bload2(rb, off) << (16 * (i & 1));
          }
        }
        pb[u] = v;
      }
    }
  };
  auto load_stage = [&](int st) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) load(st * KS + ks, pa[ks], pb[ks]);
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int u = 0; u < APT; ++u) {
        const int e = tid + TB * u;
        *reinterpret_cast<v4u*>(&lA[buf][ks][(e >> 2) * LROW + (e & 3) * 16]) = pa[ks][u];
      }
#pragma unroll
      for (int u = 0; u < BPT; ++u) {
        const int e = tid + TB * u;
        if (e < BN * 4)
          *reinterpret_cast<v4u*>(&lB[buf][ks][(e >> 2) * LROW + (e & 3) * 16]) = pb[ks][u];
      }
    }
  };

  v4f acc[WR][WC];
#pragma unroll
  for (int i = 0; i < WR; ++i)
#pragma unroll
    for (int k = 0; k < WC; ++k) acc[i][k] = v4f{0.f, 0.f, 0.f, 0.f};

  // D[n][m]: lane (li, q) holds columns n .. n+3 (n = .. + 4q) of row m (.. + li)
  auto store = [&](int j) {
#pragma unroll
    for (int i = 0; i < WR; ++i) {
      const int mm = (wm * WR + i) * 16 + li;
      const int64_t m = m0 + mm;
      int64_t row = -1;
      if (m < M) {
        if constexpr (MODE == MODE_FWD) {
          row = g.orow[m];
        } else if constexpr (MODE == MODE_DX1) {
          row = 8 * m + cls;
        } else {
          const int32_t f = ltab[mm][tap_o(j)];
          row = f < 0 ? -1 : (int64_t)f + tap_c(j);
        }
      }
      if (row < 0) continue;
#pragma unroll
      for (int k = 0; k < WC; ++k) {
        const int n = n0 + (wn * WC + k) * 16 + 4 * q;
        v4f v = acc[i][k];
        if (MODE == MODE_FWD && g.relu) {
#pragma unroll
          for (int x = 0; x < 4; ++x) v[x] = fmaxf(v[x], 0.f);
        }
        float* dst = g.out + row * N + n;
        if (g.vec && n + 3 < N && N % 4 == 0) {
          *reinterpret_cast<v4f*>(dst) = v;
        } else {
#pragma unroll
          for (int x = 0; x < 4; ++x)
            if (n + x < N) dst[x] = v[x];
        }
      }
    }
  };

  const int nstages = (nsteps + KS - 1) / KS;
  load_stage(0);
  stash(0);
  __syncthreads();
  for (int st = 0; st < nstages; ++st) {
    const int buf = st & 1;
    if (st + 1 < nstages) load_stage(st + 1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int t = st * KS + ks;
      if (t < nsteps) {  // uniform
        v4u av[WC], bv[WR];
#pragma unroll
        for (int k = 0; k < WC; ++k)
          av[k] = *reinterpret_cast<const v4u*>(
              &lB[buf][ks][((wn * WC + k) * 16 + li) * LROW + q * 16]);
#pragma unroll
        for (int i = 0; i < WR; ++i)
          bv[i] = *reinterpret_cast<const v4u*>(
              &lA[buf][ks][((wm * WR + i) * 16 + li) * LROW + q * 16]);
#pragma unroll
        for (int i = 0; i < WR; ++i)
#pragma unroll
          for (int k = 0; k < WC; ++k) acc[i][k] = mma(av[k], bv[i], acc[i][k], T{});
        if (MODE == MODE_DXS && (t + 1) % nch == 0) {
          store(t / nch);
#pragma unroll
          for (int i = 0; i < WR; ++i)
#pragma unroll
            for (int k = 0; k < WC; ++k) acc[i][k] = v4f{0.f, 0.f, 0.f, 0.f};
        }
      }
    }
    if (st + 1 < nstages) stash(buf ^ 1);
    __syncthreads();
  }
  if (MODE != MODE_DXS) store(0);
}

// ---------------------------------------------------------------------------
// Weight gradient: part[range][k][ci][co] = sum over the outputs p of the
// range of x[src(p, k)][ci] dyg[p][co].  Grid: x = range, y = tap k, z = the
// (input-channel block, output-channel block) pair.  The reduction runs over
// the outputs, so the MFMA operands hold consecutive outputs of one channel
// per lane.  Tiles stay row-major in LDS ([output][channel], as in HBM, one
// 16-byte piece per thread and load) and the operands are read across rows:
//   fp32: one 4-byte read per lane and MFMA (output 4s + q of the chunk for
//         sub-step s, channel li);
//   bf16: the transposing read ds_read_b64_tr_b16, which gives lane i of a
//         16-lane group element i mod 4 of the 8-byte rows read by lanes
//         4r + i/4 (r = 0..3): lane li reads row 4h + (li >> 2) of its
//         group's eight outputs, channels 4 (li & 3) .. of the 16-channel
//         block, so lane li receives channel li of the eight outputs.
// Row pitches spread the rows a read touches over distinct LDS banks.
struct DwArgs {
  const void* x;
  int64_t x_bytes;
  const void* dy;  // dyg [G][cout] of T
  int64_t dy_bytes;
  const int32_t* tab;  // [G][8]
  float* part;
  int64_t G, per;  // outputs, outputs per range
  int cin, cout, ncb, vec;  // ncb: output-channel blocks
};

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s;

__device__ __forceinline__ v4u tr_pair(const char* lo, const char* hi) {
  const v4s a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(lo));
  const v4s b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(hi));
  const uint64_t ua = __builtin_bit_cast(uint64_t, a), ub = __builtin_bit_cast(uint64_t, b);
  return v4u{(uint32_t)ua, (uint32_t)(ua >> 32), (uint32_t)ub, (uint32_t)(ub >> 32)};
}

// LDS row pitch in bytes for rows of `row` bytes: bf16 rows are read 8 bytes
// at a time from four rows (pitch = 8 dwords mod 16), fp32 rows 4 bytes at a
// time from four rows (pitch = 16 dwords mod 64).
__host__ __device__ constexpr int dw_pitch(int row, int es) {
  return es == 2 ? row + 32 : row + 4 * ((16 - (row / 4) % 64 + 64) % 64);
}

template <typename T, int WGM, int WGN, int WR, int WC>
__global__ __launch_bounds__(TB) void k_sr_dw(DwArgs g) {
  static_assert(WGM * WGN * 64 == TB, "waves");
  constexpr int BI = 16 * WR * WGM, BO = 16 * WC * WGN;  // input x output channels
  constexpr int ES = sizeof(T), EPP = 16 / ES;
  constexpr int KSUB = ES == 2 ? 2 : 1;       // MFMA k-steps per chunk
  constexpr int KP = (ES == 2 ? 32 : 16) * KSUB;  // outputs per chunk
  constexpr int XPITCH = dw_pitch(BI * ES, ES), DPITCH = dw_pitch(BO * ES, ES);
  constexpr int XR = BI / EPP, DR = BO / EPP;  // pieces per row
  constexpr int XP = KP * XR, DP = KP * DR;    // pieces per chunk
  constexpr int XPT = (XP + TB - 1) / TB, DPT = (DP + TB - 1) / TB;
  __shared__ __attribute__((aligned(16))) char lX[2][KP * XPITCH];
  __shared__ __attribute__((aligned(16))) char lD[2][KP * DPITCH];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, q = lane >> 4;
  const int wm = wave / WGN, wn = wave % WGN;
  const int k = blockIdx.y;
  const int ci0 = (blockIdx.z / g.ncb) * BI, co0 = (blockIdx.z % g.ncb) * BO;
  const int64_t p0 = (int64_t)blockIdx.x * g.per;
  const int64_t p1 = std::min<int64_t>(g.G, p0 + g.per);
  const int cin = g.cin, cout = g.cout;
  const int o = tap_o(k), cc = tap_c(k);
  const __amdgpu_buffer_rsrc_t rx = rsrc(g.x, g.x_bytes), rd = rsrc(g.dy, g.dy_bytes);
  const int nsteps = p1 > p0 ? (int)((p1 - p0 + KP - 1) / KP) : 0;

  int32_t srcn[XPT];  // source rows of this thread's x pieces for the next chunk
  auto src_rows = [&](int t) {
#pragma unroll
    for (int u = 0; u < XPT; ++u) {
      const int e = tid + TB * u;
      const int64_t p = p0 + (int64_t)t * KP + e / XR;
      int32_t f = -1;
      if (e < XP && p < p1) f = g.tab[8 * p + o];
      srcn[u] = f < 0 ? -1 : f + cc;
    }
  };
  auto piece = [&](__amdgpu_buffer_rsrc_t rs, int64_t row, int c, int C) -> v4u {
    if (g.vec) return bload16(rs, row >= 0 && c < C ? (uint32_t)((row * C + c) * ES) : OOB);
    v4u v = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int i = 0; i < EPP; ++i) {
      const uint32_t off = row >= 0 && c + i < C ? (uint32_t)((row * C + c + i) * ES) : OOB;
      if constexpr (ES == 4)
        v[i] = bload4(rs, off);
      else
        v[i / 2] |= (uint32_t)bload2(rs, off) << (16 * (i & 1));
    }
    return v;
  };
  v4u px[XPT], pd[DPT];
  auto load = [&](int t) {
#pragma unroll
    for (int u = 0; u < XPT; ++u) {
      const int e = tid + TB * u;
      px[u] = piece(rx, e < XP ? srcn[u] : -1, ci0 + (e % XR) * EPP, cin);
    }
#pragma unroll
    for (int u = 0; u < DPT; ++u) {
      const int e = tid + TB * u;
      const int64_t p = p0 + (int64_t)t * KP + e / DR;
      pd[u] = piece(rd, e < DP && p < p1 ? p : -1, co0 + (e % DR) * EPP, cout);
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int u = 0; u < XPT; ++u) {
      const int e = tid + TB * u;
      if (e < XP) *reinterpret_cast<v4u*>(&lX[buf][(e / XR) * XPITCH + (e % XR) * 16]) = px[u];
    }
#pragma unroll
    for (int u = 0; u < DPT; ++u) {
      const int e = tid + TB * u;
      if (e < DP) *reinterpret_cast<v4u*>(&lD[buf][(e / DR) * DPITCH + (e % DR) * 16]) = pd[u];
    }
  };

  v4f acc[WR][WC];
#pragma unroll
  for (int i = 0; i < WR; ++i)
#pragma unroll
    for (int j = 0; j < WC; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) {
    const char* X = lX[buf];
    const char* D = lD[buf];
#pragma unroll
    for (int ks = 0; ks < KSUB; ++ks) {
      if constexpr (ES == 2) {
        // rows 32 ks + 8 q + 4 h + (li >> 2), channels 4 (li & 3) of each block
        const int r0 = 32 * ks + 8 * q + (li >> 2), cb = 4 * (li & 3) * ES;
        v4u av[WR], bv[WC];
#pragma unroll
        for (int i = 0; i < WR; ++i) {
          const int c = ((wm * WR + i) * 16) * ES + cb;
          av[i] = tr_pair(X + r0 * XPITCH + c, X + (r0 + 4) * XPITCH + c);
        }
#pragma unroll
        for (int j = 0; j < WC; ++j) {
          const int c = ((wn * WC + j) * 16) * ES + cb;
          bv[j] = tr_pair(D + r0 * DPITCH + c, D + (r0 + 4) * DPITCH + c);
        }
#pragma unroll
        for (int i = 0; i < WR; ++i)
#pragma unroll
          for (int j = 0; j < WC; ++j) acc[i][j] = mma(av[i], bv[j], acc[i][j], T{});
      } else {
        // sub-step s: output 4 s + q, channel li of each block
        v4u av[WR], bv[WC];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          const int r = 4 * s + q;
#pragma unroll
          for (int i = 0; i < WR; ++i)
            av[i][s] = *reinterpret_cast<const uint32_t*>(
                X + r * XPITCH + ((wm * WR + i) * 16 + li) * ES);
#pragma unroll
          for (int j = 0; j < WC; ++j)
            bv[j][s] = *reinterpret_cast<const uint32_t*>(
                D + r * DPITCH + ((wn * WC + j) * 16 + li) * ES);
        }
#pragma unroll
        for (int i = 0; i < WR; ++i)
#pragma unroll
          for (int j = 0; j < WC; ++j) acc[i][j] = mma(av[i], bv[j], acc[i][j], T{});
      }
    }
  };

  if (nsteps > 0) {
    src_rows(0);
    load(0);
    stash(0);
    if (nsteps > 1) src_rows(1);
    __syncthreads();
  }
  for (int t = 0; t < nsteps; ++t) {
    const int buf = t & 1;
    if (t + 1 < nsteps) {
      load(t + 1);
      if (t + 2 < nsteps) src_rows(t + 2);
    }
    compute(buf);
    if (t + 1 < nsteps) stash(buf ^ 1);
    __syncthreads();
  }
  // D[ci][co]: lane (li, q) holds input channels ci .. ci+3 (4q) of output channel co (li)
  float* dst = g.part + ((int64_t)blockIdx.x * 27 + k) * cin * cout;
#pragma unroll
  for (int i = 0; i < WR; ++i)
#pragma unroll
    for (int j = 0; j < WC; ++j) {
      const int ci = ci0 + (wm * WR + i) * 16 + 4 * q, co = co0 + (wn * WC + j) * 16 + li;
      if (co < cout) {
#pragma unroll
        for (int x = 0; x < 4; ++x)
          if (ci + x < cin) dst[(int64_t)(ci + x) * cout + co] = acc[i][j][x];
      }
    }
}

// ---------------------------------------------------------------------------
// Helpers.

__device__ __forceinline__ uint16_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

// dyg[g] = dy[rows[g]], zero where ym[rows[g]] <= 0 (ym null: no mask); T =
// bf16 rounds to nearest even.  V elements per thread (V = 4: cout % 4 == 0
// and 16-byte aligned dy, ym, dyg).
template <typename T, int V>
__global__ __launch_bounds__(TB) void k_sr_dyg(const int32_t* __restrict__ rows, int64_t ng,
                                               const float* __restrict__ dy,
                                               const float* __restrict__ ym, int cout,
                                               T* __restrict__ dyg) {
  const int cv = cout / V;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ng * cv) return;
  const int64_t g = t / cv;
  const int c = (int)(t - g * cv) * V;
  const int64_t src = (int64_t)rows[g] * cout + c;
  float v[V];
  if constexpr (V == 4) {
    const v4f a = *reinterpret_cast<const v4f*>(dy + src);
    v4f m = {1.f, 1.f, 1.f, 1.f};
    if (ym) m = *reinterpret_cast<const v4f*>(ym + src);
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = m[e] > 0.f ? a[e] : 0.f;
  } else {
    v[0] = (ym && !(ym[src] > 0.f)) ? 0.f : dy[src];
  }
  T* o = dyg + g * cout + c;
  if constexpr (sizeof(T) == 2 && V == 4) {
    *reinterpret_cast<uint2*>(o) =
        uint2{bf16_rne(v[0]) | ((uint32_t)bf16_rne(v[1]) << 16),
              bf16_rne(v[2]) | ((uint32_t)bf16_rne(v[3]) << 16)};
  } else if constexpr (sizeof(T) == 2) {
    o[0] = bf16_rne(v[0]);
  } else if constexpr (V == 4) {
    *reinterpret_cast<v4f*>(o) = v4f{v[0], v[1], v[2], v[3]};
  } else {
    o[0] = v[0];
  }
}

// wt[k][n][c] = w[k][c][n] (27 taps).
template <typename T>
__global__ __launch_bounds__(TB) void k_sr_wt(const T* __restrict__ w, int cin, int cout,
                                              T* __restrict__ wt) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= (int64_t)27 * cin * cout) return;
  const int c = (int)(t % cin);
  const int n = (int)((t / cin) % cout);
  const int64_t k = t / ((int64_t)cin * cout);
  wt[t] = w[(k * cin + c) * cout + n];
}

// Rows i of y [n][c] with label 0 set to zero.
__global__ __launch_bounds__(TB) void k_sr_zero_empty(const int32_t* __restrict__ labels, int64_t n,
                                                      int c, float* __restrict__ y) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n * c) return;
  if (labels[t / c] == 0) y[t] = 0.f;
}
// The same four channels per thread (c % 4 == 0, y 16-byte aligned).
__global__ __launch_bounds__(TB) void k_sr_zero_empty4(const int32_t* __restrict__ labels,
                                                       int64_t n, int cv, float* __restrict__ y) {
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n * cv) return;
  if (labels[t / cv] == 0) reinterpret_cast<v4f*>(y)[t] = v4f{0.f, 0.f, 0.f, 0.f};
}

inline unsigned grid_for(int64_t n) { return (unsigned)oc::cdiv(n, TB); }

struct Shape {
  int64_t G, n_in, n_out;
};

Shape shape_of(const oc_octree* t, int l, int r) { return {t->M[l - r], t->N[l], t->N[l - r]}; }

// Workspace layout (each part 256-byte aligned): tab [G][8] i32 | then per pass.
size_t tab_bytes(const Shape& h) { return oc::align256((size_t)h.G * 8 * 4); }

void build_table(const oc_octree* t, int l, int r, int32_t* tab, hipStream_t s) {
  const int64_t G = t->M[l - r];
  oc::launch(k_sr_table, dim3(grid_for(G * 8)), dim3(TB), 0, s, (const int32_t*)t->nbr[l - r + 1],
             G, r, oc::sr_labels(t, l, r), tab);
}

// Ranges of the weight gradient's outputs: enough work items to fill the GPU
// (about four per compute unit), at least 64 outputs each.
int dw_ranges(int64_t G, int cin, int cout) {
  const int64_t blocks = 27 * oc::cdiv(cin, 64) * (cout <= 64 ? 1 : oc::cdiv(cout, 128));
  int64_t r = oc::cdiv(4 * (int64_t)oc::cu_count(), blocks);
  r = std::min<int64_t>(r, std::max<int64_t>(1, G / 64));
  return (int)std::max<int64_t>(1, std::min<int64_t>(r, 256));
}

bool vec_ok(int C, size_t es, const void* a, const void* b) {
  return (C * es) % 16 == 0 && (uintptr_t)a % 16 == 0 && (uintptr_t)b % 16 == 0;
}

// Launch k_sr_mm with the tile shape picked for N output columns.
template <typename T, int MODE>
void launch_mm(const MmArgs& a, int classes, bool main_kernel, hipStream_t s) {
  const dim3 blk(TB);
  auto go = [&](auto kern, int bm, int bn) {
    const dim3 grid((unsigned)oc::cdiv(a.M, bm), (unsigned)oc::cdiv(a.N, bn), (unsigned)classes);
    if (main_kernel)
      oc::launch_main(kern, grid, blk, s, a);
    else
      oc::launch(kern, grid, blk, 0, s, a);
  };
  if (a.N <= 16)
    go(k_sr_mm<T, MODE, 4, 1, 1, 1, 4>, 64, 16);
  else if (a.N <= 32)
    go(k_sr_mm<T, MODE, 4, 1, 1, 2, 4>, 64, 32);
  else if (a.N <= 64)
    go(k_sr_mm<T, MODE, 2, 2, 2, 2, 1>, 64, 64);
  else
    go(k_sr_mm<T, MODE, 2, 2, 4, 4, 1>, 128, 128);
}

template <typename T>
void launch_dw(const DwArgs& a, int nranges, hipStream_t s) {
  const int nib = (int)oc::cdiv(a.cin, 64);
  DwArgs g = a;
  if (a.cout <= 16) {
    g.ncb = 1;
    oc::launch_main(k_sr_dw<T, 4, 1, 1, 1>, dim3(nranges, 27, nib), dim3(TB), s, g);
  } else if (a.cout <= 32) {
    g.ncb = 1;
    oc::launch_main(k_sr_dw<T, 2, 2, 2, 1>, dim3(nranges, 27, nib), dim3(TB), s, g);
  } else if (a.cout <= 64) {
    g.ncb = 1;
    oc::launch_main(k_sr_dw<T, 2, 2, 2, 2>, dim3(nranges, 27, nib), dim3(TB), s, g);
  } else {
    g.ncb = (int)oc::cdiv(a.cout, 128);
    oc::launch_main(k_sr_dw<T, 2, 2, 2, 4>, dim3(nranges, 27, nib * g.ncb), dim3(TB), s, g);
  }
}

}  // namespace

namespace oc {

const char* conv_sr_kernel_name(int pass, int r, bool bf16, int cin, int cout) {
  // must follow launch_mm / launch_dw
  const char* T = bf16 ? "unsigned short" : "float";
  static thread_local char buf[96];
  if (pass == 2) {
    const char* cfg = cout <= 16   ? "4, 1, 1, 1"
                      : cout <= 32 ? "2, 2, 2, 1"
                      : cout <= 64 ? "2, 2, 2, 2"
                                   : "2, 2, 2, 4";
    snprintf(buf, sizeof(buf), "k_sr_dw<%s, %s>", T, cfg);
  } else {
    const int n = pass == 0 ? cout : cin;
    const int mode = pass == 0 ? MODE_FWD : r == 1 ? MODE_DX1 : MODE_DXS;
    const char* cfg = n <= 16   ? "4, 1, 1, 1, 4"
                      : n <= 32 ? "4, 1, 1, 2, 4"
                      : n <= 64 ? "2, 2, 2, 2, 1"
                                : "2, 2, 4, 4, 1";
    snprintf(buf, sizeof(buf), "k_sr_mm<%s, %d, %s>", T, mode, cfg);
  }
  return buf;
}

size_t conv_s2_fwd_ws(const oc_octree* t, int l, int r, int cin, int cout, bool bf16) {
  const Shape h = shape_of(t, l, r);
  if (h.G == 0) return 0;
  return tab_bytes(h) + align256((size_t)27 * cin * cout * (bf16 ? 2 : 4));
}

size_t conv_s2_bwd_ws(const oc_octree* t, int l, int r, int cin, int cout, bool bf16, bool dx,
                      bool dw) {
  const Shape h = shape_of(t, l, r);
  if (h.G == 0 || (!dx && !dw)) return 0;
  const size_t es = bf16 ? 2 : 4;
  size_t b = tab_bytes(h) + align256((size_t)h.G * cout * es);  // tab, dyg
  if (dw) b += align256((size_t)dw_ranges(h.G, cin, cout) * 27 * cin * cout * 4);
  return b;
}

oc_status conv_s2_fwd(const oc_octree* t, int l, int r, const void* x, int cin, const void* w,
                      int cout, bool bf16, float* y, int relu, void* ws, hipStream_t s) {
  const Shape h = shape_of(t, l, r);
  const size_t es = bf16 ? 2 : 4;
  if ((int64_t)h.n_in * cin * es >= INT32_MAX || (int64_t)27 * cin * cout * es >= INT32_MAX)
    return fail(OC_ERR_UNSUPPORTED, "strided convolution: input beyond 2 GB");
  if (h.G == 0) {
    if (h.n_out > 0) fill_u32(y, 0u, h.n_out * cout, s);
    return OC_OK;
  }
  char* p = (char*)ws;
  int32_t* tab = (int32_t*)p;
  p += tab_bytes(h);
  void* wt = p;
  build_table(t, l, r, tab, s);
  const int64_t nw = (int64_t)27 * cin * cout;
  if (bf16)
    launch(k_sr_wt<uint16_t>, dim3(grid_for(nw)), dim3(TB), 0, s, (const uint16_t*)w, cin, cout,
           (uint16_t*)wt);
  else
    launch(k_sr_wt<float>, dim3(grid_for(nw)), dim3(TB), 0, s, (const float*)w, cin, cout,
           (float*)wt);
  if (cout % 4 == 0 && (uintptr_t)y % 16 == 0)
    launch(k_sr_zero_empty4, dim3(grid_for(h.n_out * (cout / 4))), dim3(TB), 0, s,
           (const int32_t*)t->labels[l - r], h.n_out, cout / 4, y);
  else
    launch(k_sr_zero_empty, dim3(grid_for(h.n_out * cout)), dim3(TB), 0, s,
           (const int32_t*)t->labels[l - r], h.n_out, cout, y);
  MmArgs a{x, (int64_t)h.n_in * cin * (int64_t)es, wt, nw * (int64_t)es, y, tab,
           t->rows[l - r], h.G, cin, cout, relu,
           (int)(vec_ok(cin, es, x, wt) && (uintptr_t)y % 16 == 0)};
  if (bf16)
    launch_mm<uint16_t, MODE_FWD>(a, 1, true, s);
  else
    launch_mm<float, MODE_FWD>(a, 1, true, s);
  return OC_OK;
}

oc_status conv_s2_bwd(const oc_octree* t, int l, int r, const void* x, int cin, const void* w,
                      int cout, bool bf16, const float* ym, const float* dy, float* dx, float* dw,
                      void* ws, hipStream_t s) {
  const Shape h = shape_of(t, l, r);
  const size_t es = bf16 ? 2 : 4;
  const int64_t entries = (int64_t)27 * cin * cout;
  if ((int64_t)h.n_in * cin * es >= INT32_MAX || (int64_t)h.G * cout * es >= INT32_MAX ||
      entries * (int64_t)es >= INT32_MAX)
    return fail(OC_ERR_UNSUPPORTED, "strided convolution: operands beyond 2 GB");
  if (h.G == 0) {
    if (dx && h.n_in > 0) fill_u32(dx, 0u, h.n_in * cin, s);
    if (dw) fill_u32(dw, 0u, entries, s);
    return OC_OK;
  }
  char* p = (char*)ws;
  int32_t* tab = (int32_t*)p;
  p += tab_bytes(h);
  void* dyg = p;
  p += align256((size_t)h.G * cout * es);
  float* part = (float*)p;
  const int32_t* prow = t->rows[l - r];
  const bool v4 = cout % 4 == 0 && (uintptr_t)dy % 16 == 0 && (!ym || (uintptr_t)ym % 16 == 0);
  if (bf16 && v4)
    launch(k_sr_dyg<uint16_t, 4>, dim3(grid_for(h.G * (cout / 4))), dim3(TB), 0, s, prow, h.G, dy,
           ym, cout, (uint16_t*)dyg);
  else if (bf16)
    launch(k_sr_dyg<uint16_t, 1>, dim3(grid_for(h.G * cout)), dim3(TB), 0, s, prow, h.G, dy, ym,
           cout, (uint16_t*)dyg);
  else if (v4)
    launch(k_sr_dyg<float, 4>, dim3(grid_for(h.G * (cout / 4))), dim3(TB), 0, s, prow, h.G, dy,
           ym, cout, (float*)dyg);
  else
    launch(k_sr_dyg<float, 1>, dim3(grid_for(h.G * cout)), dim3(TB), 0, s, prow, h.G, dy, ym,
           cout, (float*)dyg);
  if (dw || (dx && r > 1)) build_table(t, l, r, tab, s);
  if (dx) {
    // dx = sum of dyg W^T: reduction over the output channels, N = cin
    MmArgs a{dyg, (int64_t)h.G * cout * (int64_t)es, w, entries * (int64_t)es, dx,
             r == 1 ? (const int32_t*)t->nbr[l] : tab, nullptr, r == 1 ? h.G : h.G, cout, cin,
             0, (int)(vec_ok(cout, es, dyg, w) && (uintptr_t)dx % 16 == 0)};
    if (r == 1) {
      // every depth-l row is one child of one group: all written by their class
      if (bf16)
        launch_mm<uint16_t, MODE_DX1>(a, 8, true, s);
      else
        launch_mm<float, MODE_DX1>(a, 8, true, s);
    } else {
      fill_u32(dx, 0u, h.n_in * cin, s);
      if (bf16)
        launch_mm<uint16_t, MODE_DXS>(a, 1, true, s);
      else
        launch_mm<float, MODE_DXS>(a, 1, true, s);
    }
  }
  if (dw) {
    const int nr = dw_ranges(h.G, cin, cout);
    DwArgs a{x, (int64_t)h.n_in * cin * (int64_t)es, dyg, (int64_t)h.G * cout * (int64_t)es, tab,
             part, h.G, cdiv(h.G, nr), cin, cout, 1, (int)vec_ok(cin, es, x, x) &&
                                                        (int)vec_ok(cout, es, dyg, dyg)};
    if (bf16)
      launch_dw<uint16_t>(a, nr, s);
    else
      launch_dw<float>(a, nr, s);
    sum_partials(part, nr, entries, dw, s);
  }
  return OC_OK;
}

}  // namespace oc
