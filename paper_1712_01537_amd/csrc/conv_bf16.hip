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
// positions keep the layout of HBM, and dY is rounded to bf16 into a
// sibling-group layout whose 16-byte pieces are eight children of a column.  A workgroup owns the taps
// of one x-offset and up to two (K = 5) or three (K = 3) y-offsets for every
// input channel block, the waves split those (tap, channel block) pairs and
// keep their dW blocks in registers, and the workgroup streams a range of
// sibling groups, eight per step.  Ranges write partial sums that a second kernel adds in a fixed
// order, so results do not depend on scheduling.
//
// LDS layouts place the 16-byte pieces (8 channels) of a position or row at
// piece index o ^ f(position): the eight children of a group (forward), or
// the four rows of a transposing load (weight gradient), then fall on
// distinct banks.
#include "conv_bf16.h"

#include <algorithm>
#include <utility>

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef short v4s __attribute__((ext_vector_type(4)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4s lds_v4s;
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) void* lptr_t;

constexpr int TB = 256;

// Zero rows: the source of masked-off loads (absent neighbours, channels or
// columns past the end), so that every lane of every load instruction loads
// and each wave's count of outstanding loads is known in advance.  64 KB, so
// that absent lanes spread over many cache lines.
constexpr int ZROWS = 4096;
__device__ __attribute__((aligned(16))) uint32_t g_zero_rows[ZROWS][4];
// -1: the neighbour entry loaded for groups past a range (absent neighbour).
__device__ const int32_t g_minus1 = -1;

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
// Buffer resource over `bytes` bytes at p (raw: offsets in bytes, no stride);
// loads at offsets past `bytes` return zeros.
typedef int32_t sv4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ sv4 buf_rsrc(const void* p, uint32_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)p;
  sv4 r;
  r[0] = (int32_t)(uint32_t)a;
  r[1] = (int32_t)((a >> 32) & 0xffffu);
  r[2] = (int32_t)bytes;
  r[3] = 0x00020000;
  return r;
}
// The same direct load through a buffer resource: lane i's 16 bytes at byte
// offset off of the resource land at lds + 16 i; an offset past the end
// stores zeros.
__device__ __forceinline__ void lds_bload16(sv4 rsrc, uint32_t off, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(lds), "v"(off),
               "s"(rsrc)
               : "memory", "m0");
}
// The same for 4 bytes per lane (lane i's dword lands at lds + 4 i).
__device__ __forceinline__ void lds_load4(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off" ::"s"(lds), "v"(src)
               : "memory", "m0");
}
// s_waitcnt vmcnt(0): all of this wave's vector memory operations are done.
__device__ __forceinline__ void vm_wait0() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// 16-byte global load into registers, issued from inline assembly: the
// compiler neither waits for it nor counts it, so the caller waits with
// vm_wait_for() before the registers are read.
__device__ __forceinline__ void gload16(v4u& r, const void* src) {
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(r) : "v"(src) : "memory");
}
// The same with a wave-uniform 64-bit base in scalar registers and a 32-bit
// per-lane byte offset (one vector register per address instead of two).
__device__ __forceinline__ void gload16s(v4u& r, uint32_t voff, const void* sbase) {
  asm volatile("global_load_dwordx4 %0, %1, %2" : "=v"(r) : "v"(voff), "s"(sbase) : "memory");
}
// Wait until at most N vector memory operations of this wave are outstanding
// (they complete in issue order), then hand the registers w over as written.
template <int N>
__device__ __forceinline__ void vm_wait_for(v4u (&w)[4]) {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%4)" : "+v"(w[0]), "+v"(w[1]), "+v"(w[2]), "+v"(w[3]) : "n"(N));
}
template <int N>
__device__ __forceinline__ void vm_wait_n() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// f(std::integral_constant<int, 0>), ..., f(std::integral_constant<int, N-1>).
template <typename F, int... I>
__device__ __forceinline__ void static_for_(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_(f, std::make_integer_sequence<int, N>{});
}
// Workgroup barrier without the memory fence of __syncthreads (which would
// wait for every outstanding global load); LDS operations are complete first.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

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

// Neighbour row of tile position (px, py, pz) of a group whose 27-entry
// parent-neighbour row is nb (positions are offsets +R from the group's first
// child, per axis in [0, K]), or -1.
template <int R>
__device__ __forceinline__ int32_t tile_row(const int32_t* nb, int px, int py, int pz) {
  const int ux = px - R, uy = py - R, uz = pz - R;
  const int32_t b = nb[((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1)];
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

// y[e] = bf16(x[e]), eight entries per thread: two 16-byte loads and one
// 16-byte store when x and y are 16-byte aligned (vec), else element
// accesses.
__global__ __launch_bounds__(TB) void k_bf_round(const float* __restrict__ x, int64_t n, int vec,
                                                 uint16_t* __restrict__ y) {
  const int64_t e = 8 * ((int64_t)blockIdx.x * TB + threadIdx.x);
  if (e >= n) return;
  if (vec && e + 8 <= n) {
    const float4 a = *reinterpret_cast<const float4*>(x + e);
    const float4 b = *reinterpret_cast<const float4*>(x + e + 4);
    *reinterpret_cast<uint4*>(y + e) =
        uint4{f2bf(a.x) | (f2bf(a.y) << 16), f2bf(a.z) | (f2bf(a.w) << 16),
              f2bf(b.x) | (f2bf(b.y) << 16), f2bf(b.z) | (f2bf(b.w) << 16)};
  } else {
    for (int64_t i = e; i < n && i < e + 8; ++i) y[i] = (uint16_t)f2bf(x[i]);
  }
}

// The same conversion into the sibling-group layout of the weight gradient:
// outg[g][c][j] = bf16(masked in[8g + j][c]) (the eight children of a group
// contiguous per column, so that eight consecutive octants of one column are
// one 16-byte piece), and the row-major copy outr[8g + j][c] when outr is
// not NULL.  A workgroup converts 8 groups (64 rows) x 64 columns: 16-byte
// loads of the rows, the bf16 values written transposed into LDS, then
// 16-byte pieces read back and stored contiguously.  C % 4 == 0 and
// 16-byte aligned rows (vec), else element loads.
__global__ __launch_bounds__(TB) void k_bf_cvt_g(const float* __restrict__ in,
                                                 const float* __restrict__ ym, int64_t ngroups,
                                                 int C, int vec, uint16_t* __restrict__ outg,
                                                 uint16_t* __restrict__ outr) {
  constexpr int TP = 64 + 8;  // LDS row (one column of the tile) in bf16, padded
  __shared__ __attribute__((aligned(16))) uint16_t tt[64 * TP];
  const int64_t g0 = (int64_t)blockIdx.x * 8, nrows = 8 * ngroups;
  const int c0 = blockIdx.y * 64;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int idx = threadIdx.x + TB * k, r = idx >> 4, cq = (idx & 15) * 4;
    const int64_t row = 8 * g0 + r;
    const int c = c0 + cq;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (row < nrows && c < C) {
      const int64_t e = row * C + c;
      if (vec) {
        const float4 a = *reinterpret_cast<const float4*>(in + e);
        v[0] = a.x, v[1] = a.y, v[2] = a.z, v[3] = a.w;
        if (ym) {
          const float4 y = *reinterpret_cast<const float4*>(ym + e);
          v[0] = y.x > 0.f ? v[0] : 0.f, v[1] = y.y > 0.f ? v[1] : 0.f;
          v[2] = y.z > 0.f ? v[2] : 0.f, v[3] = y.w > 0.f ? v[3] : 0.f;
        }
      } else {
        for (int i = 0; i < 4 && c + i < C; ++i) v[i] = ym && !(ym[e + i] > 0.f) ? 0.f : in[e + i];
      }
      uint32_t h[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) h[i] = f2bf(v[i]);
      if (outr) {
        if (vec)
          *reinterpret_cast<uint2*>(outr + e) = uint2{h[0] | (h[1] << 16), h[2] | (h[3] << 16)};
        else
          for (int i = 0; i < 4 && c + i < C; ++i) outr[e + i] = (uint16_t)h[i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) tt[(cq + i) * TP + r] = (uint16_t)h[i];
    }
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int idx = threadIdx.x + TB * k, gl = idx >> 6, cl = idx & 63;
    const int64_t g = g0 + gl;
    if (g < ngroups && c0 + cl < C)
      reinterpret_cast<v4u*>(outg)[g * C + c0 + cl] =
          *reinterpret_cast<const v4u*>(&tt[cl * TP + 8 * gl]);
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
// Forward / input gradient, one chunk of at most 64 reduction channels.
// x [8 ngroups][kk] bf16 (kk % 8 == 0), wp as produced by k_bf_wprep, out
// [8 ngroups][nn] fp32 (nn % 16 == 0).  The chunk is the channel octets
// 8 chunk .. 8 chunk + 4 HC - 1 (HC halves of 32 channels); with acc the
// result is added to out (chunks are launched in order), relu applies
// max(0, .) to the sum.  Grid: x = tiles of 8 groups, y = blocks of 64
// output channels; 512 threads.  Slab j lives in ring buffer j % 3: 8 groups
// x S^2 positions x 8 pieces, piece o of position (j, py, pz) at
// o ^ ((j&1) << 2 | (py&1) << 1 | (pz&1)).
// A phase (x-offset) has HC K^2 steps (tap, half).  Each wave takes the same
// number MI of items: whole steps wave + NW i, then the leftover steps split
// into their four row blocks (one per wave; waves left without one take an
// empty item, whose loads are still issued).  The K phases are one unrolled
// sequence of K MI items.  Every wave issues its global loads in a fixed
// order and waits with counts (they complete in issue order): the slab DMA
// at the start of a phase, the weights of item n + RW - 1 right after item n
// is multiplied, into the register set item n - 1 used (RW sets).
// FLIP only names the pass (the weights decide what is computed).
template <int K, int HC, bool FLIP>
__global__ __launch_bounds__(512) void k_conv_bf(const int32_t* __restrict__ nbr, int64_t ngroups,
                                                  const uint16_t* __restrict__ x, int kk,
                                                  const uint16_t* __restrict__ wp, int nn,
                                                  int chunk, float* __restrict__ out, int acc_in,
                                                  int relu) {
  constexpr int R = (K - 1) / 2, S = K + 1, S2 = S * S, K2 = K * K, K3 = K2 * K;
  constexpr int GT = 8, NW = 8;
  constexpr int SLAB = GT * S2 * 8;  // 16-byte pieces of one slab buffer
  constexpr int RS = 68;             // floats per row of a reduction slot
  constexpr int RED = NW * 32 * RS;  // floats of one reduction round
  constexpr int NV = (3 * SLAB * 16 > RED * 4 ? 3 * SLAB * 16 : RED * 4) / 16;
  constexpr int NE = HC * K2;                 // steps per phase
  constexpr int NFULL = NE / NW, LEFT = NE % NW;
  constexpr int MI = NFULL + (LEFT ? 1 : 0);  // items per phase and wave
  constexpr int NI = K * MI;                  // items of the tile
  constexpr int RW = 4;                       // weight register sets
  constexpr int DC = (S2 + NW - 1) / NW;      // DMA instructions of a stage per wave
  static_assert(4 * LEFT <= NW, "leftover row blocks fit the waves");
  __shared__ __attribute__((aligned(16))) v4u lds[NV];
  __shared__ __attribute__((aligned(16))) v4u trash[64];  // destination of padding loads
  __shared__ int32_t nbs[GT * 27];  // neighbour rows of the tile's groups

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, q = lane >> 4;
  const int64_t g0 = (int64_t)blockIdx.x * GT;
  const int n0 = blockIdx.y * 64;
  const int KO = kk >> 3;  // channel octets of the reduction
  const int ob = 8 * chunk;
  if (tid < GT * 27)
    nbs[tid] = g0 + tid / 27 < ngroups ? nbr[27 * g0 + tid] : -1;
  __syncthreads();

  // a stage is S2 DMA instructions of 64 pieces (8 positions), DC per wave;
  // waves with one fewer issue a last load of zeros into a trash slot, so
  // that every wave issues DC
  auto stage = [&](int j) {
    v4u* buf = lds + (j % 3) * SLAB;
#pragma unroll
    for (int k = 0; k < DC; ++k) {
      const int i = wave + NW * k;
      const int s = i * 64 + lane;
      const int pos = s >> 3, g = pos / S2, p = pos - g * S2;
      const int py = p / S, pz = p - py * S;
      const int o = ob + ((s & 7) ^ (((j & 1) << 2) | ((py & 1) << 1) | (pz & 1)));
      const int32_t row = i < S2 && o < KO ? tile_row<R>(nbs + 27 * g, j, py, pz) : -1;
      const void* src = row >= 0 ? (const void*)(x + (int64_t)row * kk + 8 * o)
                                 : (const void*)g_zero_rows[(s + 64 * (int)blockIdx.x) & (ZROWS - 1)];
      lds_load16(src, lds_addr(i < S2 ? buf + i * 64 : trash));
    }
  };

  // lane (li, q) of row block b supplies row li: child li & 7 of group
  // 2b + (li >> 3), channels 8q..8q+7 of the step's 32
  const int cc = li & 7, cx = cc >> 2, cy = (cc >> 1) & 1, cz = cc & 1, gl = li >> 3;
  // item i of a phase: step e (tap e / HC, half e % HC) and the row blocks
  // it covers: all (-1), one (0..3) or none (-2)
  auto item_e = [&](int i) { return i < NFULL ? wave + NW * i : NFULL * NW + (wave >> 2); };
  auto item_only = [&](int i) { return i < NFULL ? -1 : (wave < 4 * LEFT ? (wave & 3) : -2); };
  auto load_w = [&](v4u (&wv)[4], int n) {  // item n of the tile
    const int ph = n / MI, i = n % MI;
    const int e = item_e(i), only = item_only(i);
    const int tap2 = e / HC, h = e - tap2 * HC;
    const int t = ph * K2 + tap2;
    const int o = ob + 4 * h + q;
#pragma unroll
    for (int nf = 0; nf < 4; ++nf) {
      const int nc = n0 + 16 * nf + li;
      const void* src = only != -2 && nc < nn && o < KO
                            ? (const void*)(wp + ((int64_t)(o * K3 + t) * nn + nc) * 8)
                            : (const void*)g_zero_rows[lane];
      gload16(wv[nf], src);
    }
  };
  v4f acc[4][4];
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int nf = 0; nf < 4; ++nf) acc[b][nf] = v4f{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const v4u (&wv)[4], int n) {
    const int ph = n / MI, i = n % MI;
    const int e = item_e(i), only = item_only(i);
    const int tap2 = e / HC, h = e - tap2 * HC;
    const int dyi = tap2 / K, dzi = tap2 - dyi * K;
    const int px = ph + cx, py = dyi + cy, pz = dzi + cz;
    const v4u* buf = lds + (px % 3) * SLAB;
    const int f = ((px & 1) << 2) | ((py & 1) << 1) | (pz & 1);
    const int base = (py * S + pz) * 8 + ((4 * h + q) ^ f);
    if (only == -1) {
      v4u a[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) a[b] = buf[(2 * b + gl) * S2 * 8 + base];
#pragma unroll
      for (int b = 0; b < 4; ++b)
#pragma unroll
        for (int nf = 0; nf < 4; ++nf) acc[b][nf] = mfma_bf(a[b], wv[nf], acc[b][nf]);
    } else {
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        if (b == only) {
          const v4u a = buf[(2 * b + gl) * S2 * 8 + base];
#pragma unroll
          for (int nf = 0; nf < 4; ++nf) acc[b][nf] = mfma_bf(a, wv[nf], acc[b][nf]);
        }
      }
    }
  };
  // Load order of a wave: stage 0, stage 1, W(0 .. RW-2); at the start of
  // phase p <= K-2, stage p+2; after item n, W(n + RW - 1).
  // Loads younger than W(n) when item n starts: W(n+1 .. n+RW-2), and the
  // stages of the phases p whose first item pMI lies in [n-RW+2, n].
  struct Counts {
    static constexpr int younger_w(int n) {
      int c = 0;
      for (int j = n + 1; j <= n + RW - 2; ++j) c += j < NI ? 4 : 0;
      for (int p = 0; p <= K - 2; ++p) c += (p * MI >= n - RW + 2 && p * MI <= n) ? DC : 0;
      return c;
    }
    // Loads younger than stage p+1 (the newer of the two slabs phase p reads)
    // when phase p starts: W(0 .. RW-2) for p = 0, otherwise the weights
    // issued after the items of phase p-1, W((p-1)MI + RW-1 .. pMI + RW-2).
    static constexpr int younger_stage(int p) {
      const int lo = p == 0 ? 0 : (p - 1) * MI + RW - 1;
      int hi = p == 0 ? RW - 2 : p * MI + RW - 2;
      hi = hi < NI - 1 ? hi : NI - 1;
      return hi >= lo ? 4 * (hi - lo + 1) : 0;
    }
  };

  v4u W[RW][4];
  stage(0);
  stage(1);
#pragma unroll
  for (int j = 0; j <= RW - 2; ++j)
    if (j < NI) load_w(W[j], j);
  static_for<NI>([&](auto nc) {
    constexpr int n = decltype(nc)::value;
    if constexpr (n % MI == 0) {
      constexpr int p = n / MI;
      vm_wait_n<Counts::younger_stage(p)>();  // slabs p, p+1 have landed
      lds_barrier();                          // ... everywhere; phase p-1 is done
      if constexpr (p + 2 < S) stage(p + 2);
    }
    vm_wait_for<Counts::younger_w(n)>(W[n % RW]);
    compute(W[n % RW], n);
    if constexpr (n + RW - 1 < NI) load_w(W[(n + RW - 1) % RW], n + RW - 1);
  });
  vm_wait0();

  // add the waves' tiles in wave order, 32 rows per round (and to out for
  // a later chunk)
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
    const int64_t row = 8 * g0 + 32 * rd + r;
    const int n = n0 + cq;
    v4f sum = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < NW; ++w) sum += *reinterpret_cast<const v4f*>(&red[(w * 32 + r) * RS + cq]);
    if (row < nrows && n < nn) {
      v4f* dst = reinterpret_cast<v4f*>(out + row * nn + n);
      if (acc_in) sum = *dst + sum;
      if (relu) {
#pragma unroll
        for (int j = 0; j < 4; ++j) sum[j] = fmaxf(sum[j], 0.f);
      }
      *dst = sum;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// The same forward / input gradient over tiles of 16 sibling groups (128 rows,
// k_conv_bfw): every weight read from L2 then feeds 8 row blocks instead of 4,
// which halves the weight traffic per row (the whole W is read once per
// tile).  To fit 16 groups' union blocks, a slab holds one 32-channel half
// of one x-slab (16 groups x S^2 positions x 4 pieces); the phases are
// (half h, x-offset dx), h outer, and phase (h, dx) reads slabs h S + dx and
// h S + dx + 1.  A ring of four slab buffers keeps two slabs in flight
// beside the two being read (the first phase of a half needs two new ones).
// Piece o of position (px, py, pz) sits at o ^ (2 (px & 1) + (py & 1)), and
// positions are 64 bytes apart, so the eight children of a group read eight
// distinct 16-byte bank groups.  A phase has K^2 steps (taps); each wave takes
// NFULL whole steps (all 8 row blocks: 8 LDS reads feed 32 MFMAs) and one
// row block of the leftover step.  Waits are compile-time counts of younger
// loads from a replay of the fixed issue order (BfwShape::younger).  The eight waves'
// partial tiles are added in wave order through LDS, 32 rows per round.
template <int K, int HC, int GT_, int NW_>
struct BfwShape {
  static constexpr int R = (K - 1) / 2, S = K + 1, S2 = S * S, K2 = K * K, K3 = K2 * K;
  static constexpr int GT = GT_, NW = NW_, NRB = GT / 2;
  static_assert(NW == NRB, "the reduction rounds give every row block one term per wave");
  static constexpr int SLAB = GT * S2 * 4;  // 16-byte pieces of one slab buffer
  static constexpr int NB = 4;              // slab buffers
  static constexpr int NSL = HC * S;        // slabs of a tile
  static constexpr int NPH = HC * K;        // phases
  static constexpr int NFULL = K2 / NW, LEFT = K2 % NW;
  static_assert(LEFT * NRB == NW, "the leftover step's row blocks are one per wave");
  static constexpr int MI = NFULL + 1;      // items per phase and wave
  static constexpr int NI = NPH * MI;       // items of the tile
  static constexpr int RW = 3;              // weight register sets
  static constexpr int NDMA = GT * S2 * 4 / 64;   // DMA instructions of a slab
  static constexpr int DC = (NDMA + NW - 1) / NW;  // ... per wave
  static constexpr int RS = 68;                    // floats per row of a reduction slot
  static constexpr int RED = NRB * 16 * RS;        // floats of the tile's sum
  static constexpr int NV = (NB * SLAB * 16 > RED * 4 ? NB * SLAB * 16 : RED * 4) / 16;
  static constexpr int slab_of_phase(int ph) { return (ph / K) * S + ph % K; }
  static constexpr int last_slab(int ph) {  // slabs issued by the start of phase ph
    return slab_of_phase(ph) + 3 < NSL - 1 ? slab_of_phase(ph) + 3 : NSL - 1;
  }
  static constexpr int NPRE = NSL < 3 ? NSL : 3;  // slabs issued before phase 0
  // Replay of a wave's issue order: stages (DC loads each) and weight sets
  // (4 loads each).  what = 0: loads issued after stage `idx` when phase
  // `at` starts (before its own stages); what = 1: loads issued after W(idx)
  // when item idx starts.
  static constexpr int younger(int what, int idx, int at) {
    int stage_end[2 * 6] = {};
    int w_end[96] = {};
    int ops = 0, issued = -1;
    for (int s = 0; s < NPRE; ++s) {
      ops += DC;
      stage_end[s] = ops;
      issued = s;
    }
    for (int j = 0; j <= RW - 2; ++j)
      if (j < NI) {
        ops += 4;
        w_end[j] = ops;
      }
    for (int ph = 0; ph < NPH; ++ph) {
      if (what == 0 && at == ph) return ops - stage_end[idx];
      for (int i = 0; i < MI; ++i) {
        const int n = ph * MI + i;
        if (what == 1 && idx == n) return ops - w_end[n];
        if (n + RW - 1 < NI) {
          ops += 4;
          w_end[n + RW - 1] = ops;
        }
        if (i == 0) {  // the phase's stages, after its first item
          for (int s = issued + 1; s <= last_slab(ph); ++s) {
            ops += DC;
            stage_end[s] = ops;
            issued = s;
          }
        }
      }
    }
    return 0;
  }
};

template <int K, int HC, bool FLIP, int GT_, int NW_>
__global__ __launch_bounds__(NW_ * 64, 8 / NW_) void k_conv_bfw(const int32_t* __restrict__ nbr, int64_t ngroups,
                                                   const uint16_t* __restrict__ x, int kk,
                                                   const uint16_t* __restrict__ wp, int nn,
                                                   int chunk, float* __restrict__ out, int acc_in,
                                                   int relu) {
  using B = BfwShape<K, HC, GT_, NW_>;
  constexpr int R = B::R, S = B::S, S2 = B::S2, K2 = B::K2, K3 = B::K3;
  constexpr int GT = B::GT, NW = B::NW, NRB = B::NRB, SLAB = B::SLAB, NB = B::NB;
  constexpr int NFULL = B::NFULL, MI = B::MI, NI = B::NI, RW = B::RW, DC = B::DC;
  constexpr int NDMA = B::NDMA, RS = B::RS;
  static_assert(B::NSL <= 12 && NI <= 96, "replay arrays");
  static_assert(GT * 27 + 27 <= NW * 64, "one neighbour entry per thread");
  __shared__ __attribute__((aligned(16))) v4u lds[B::NV];
  __shared__ __attribute__((aligned(16))) v4u trash[64];  // destination of padding loads
  // neighbour rows of the tile's groups, then 27 entries of -1 (the entries
  // that DMA lanes past a slab look up)
  __shared__ int32_t nbs[GT * 27 + 27];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, q = lane >> 4;
  // tile of this workgroup: workgroups are dealt to the eight XCDs
  // round-robin, so tile = x-th share of the tiles + blockIdx.x / 8 (x =
  // blockIdx.x % 8) keeps neighbouring tiles, which share union rows, in one
  // XCD's L2.  A bijection on 0..gridDim.x-1.
  const int ntiles = (int)gridDim.x, xcd = (int)blockIdx.x & 7, tper = ntiles >> 3;
  const int tile = xcd * tper + (xcd < (ntiles & 7) ? xcd : (ntiles & 7)) + ((int)blockIdx.x >> 3);
  const int64_t g0 = (int64_t)tile * GT;
  const int n0 = blockIdx.y * 64;
  const int ob = 8 * chunk;
  if (tid < GT * 27 + 27)
    nbs[tid] = tid < GT * 27 && g0 + tid / 27 < ngroups ? nbr[27 * g0 + tid] : -1;

  // DMA instruction i of a slab covers 16 positions x 4 pieces.  What a lane
  // loads depends on the slab (half h, x-position j) only through the x-cell
  // and x-bit of j, its parity and h, so the rest is worked out once per
  // tile: nbi[k] = the lane's neighbour entry without the x-cell, eb[k] =
  // the byte offset in the row block of its child's y, z bits and of its
  // 16-byte piece before the slab's swizzle.  The piece is
  // ((s & 3) ^ (py & 1)) ^ 2 (j & 1) of octet block ob + 4h (the launcher
  // guarantees every such octet exists), and an absent row reads zeros
  // through an offset past the end of x.
  const sv4 xr = buf_rsrc(x, (uint32_t)(8 * ngroups * kk * 2));
  int nbi[DC];
  uint32_t eb[DC];
#pragma unroll
  for (int k = 0; k < DC; ++k) {
    const int i = wave + NW * k;
    const int s = i * 64 + lane;
    const int pos = s >> 2, g = pos / S2, p = pos - g * S2;
    const int py = p / S, pz = p - py * S;
    const int uy = py - R, uz = pz - R;
    nbi[k] = i < NDMA ? 27 * g + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1) : GT * 27;
    eb[k] = 2u * (uint32_t)((2 * (uy & 1) + (uz & 1)) * kk + 8 * (ob + ((s & 3) ^ (py & 1))));
  }
  __syncthreads();

  // slab sl (half h = sl / S, x-position j = sl % S) into buffer sl % NB
  auto stage = [&](int sl) {
    const int h = sl / S, j = sl - h * S;
    const int ux = j - R, xcell = (ux >> 1) + 1;
    v4u* buf = lds + (sl % NB) * SLAB;
    // the slab's constant (the child's x bit and the half) and swizzle term
    const uint32_t cb = 2u * (uint32_t)(4 * (ux & 1) * kk + 32 * h), xo = 32u * (uint32_t)(j & 1);
    int32_t b[DC];
#pragma unroll
    for (int k = 0; k < DC; ++k) b[k] = nbs[nbi[k] + 9 * xcell];
#pragma unroll
    for (int k = 0; k < DC; ++k) {
      const int i = wave + NW * k;
      const uint32_t off =
          b[k] < 0 ? 0x80000000u : (uint32_t)b[k] * (uint32_t)(2 * kk) + ((eb[k] ^ xo) + cb);
      lds_bload16(xr, off, lds_addr(i < NDMA ? buf + i * 64 : trash));
    }
  };

  // lane (li, q) of row block b supplies row li: child li & 7 of group
  // 2b + (li >> 3), channels 8q..8q+7 of the phase's half
  const int cc = li & 7, cx = cc >> 2, cy = (cc >> 1) & 1, cz = cc & 1, gl = li >> 3;
  // weights of item n: wp[(o K3 + t) nn + nc][8] for octet o = ob + 4h + q,
  // column nc = n0 + 16 nf + li: a uniform base per (item, nf) and one lane
  // offset (the launcher guarantees every lane's octet and column exist)
  const uint32_t wlane = (uint32_t)(((int64_t)q * K3 * nn + li) * 16);
  auto load_w = [&](v4u (&wv)[4], int n) {  // item n of the tile
    const int ph = n / MI, i = n % MI;
    const int h = ph / K, dx = ph - h * K;
    const int e = i < NFULL ? wave + NW * i : NFULL * NW;
    const int t = dx * K2 + e;
    const uint16_t* wb = wp + ((int64_t)((ob + 4 * h) * K3 + t) * nn + n0) * 8;
#pragma unroll
    for (int nf = 0; nf < 4; ++nf) gload16s(wv[nf], wlane, wb + 16 * nf * 8);
  };
  v4f acc[NRB][4];
#pragma unroll
  for (int b = 0; b < NRB; ++b)
#pragma unroll
    for (int nf = 0; nf < 4; ++nf) acc[b][nf] = v4f{0.f, 0.f, 0.f, 0.f};
  // LDS byte offsets of this lane's operand piece in a phase, for taps of
  // even and odd y-offset (the piece swizzle depends on the y parity); set at
  // the start of every phase, so that each item only adds constants
  uint32_t pb[2];
  auto phase_bases = [&](int ph) {
    const int h = ph / K, dx = ph - h * K;
    const int px = dx + cx;
    const uint32_t lb = (uint32_t)(((h * S + px) % NB) * SLAB + (gl * S2 + cy * S + cz) * 4) * 16;
#pragma unroll
    for (int d = 0; d < 2; ++d) pb[d] = lb + (uint32_t)(q ^ (2 * (px & 1) + ((d + cy) & 1))) * 16;
  };
  const char* lbase = reinterpret_cast<const char*>(lds);
  // accumulator set b of wave w holds row block (b + w) % 8, so that the
  // leftover step's row block (w) is set 0 in every wave
  auto opnd = [&](int dyi, int dzi, int b) {
    const uint32_t rb = (uint32_t)(((b + wave) & (NRB - 1)) * 2 * S2 * 4 * 16);
    return *reinterpret_cast<const v4u*>(lbase + pb[dyi & 1] + rb + ((dyi * S + dzi) * 4) * 16);
  };
  auto compute = [&](const v4u (&wv)[4], int n) {
    const int i = n % MI;
    const int e = i < NFULL ? wave + NW * i : NFULL * NW;
    const int dyi = e / K, dzi = e - dyi * K;
    if (i < NFULL) {
      // row blocks in pairs; the next pair's operands are read before the
      // current pair's MFMAs are issued, so the LDS latency hides behind them
      constexpr int AB = 2, NP = NRB / AB;
      v4u a[2][AB];
#pragma unroll
      for (int b = 0; b < AB; ++b) a[0][b] = opnd(dyi, dzi, b);
#pragma unroll
      for (int bh = 0; bh < NP; ++bh) {
        if (bh + 1 < NP) {
#pragma unroll
          for (int b = 0; b < AB; ++b) a[(bh + 1) & 1][b] = opnd(dyi, dzi, (bh + 1) * AB + b);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int b = 0; b < AB; ++b)
#pragma unroll
          for (int nf = 0; nf < 4; ++nf)
            acc[bh * AB + b][nf] = mfma_bf(a[bh & 1][b], wv[nf], acc[bh * AB + b][nf]);
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      // the leftover step: this wave's own row block (set 0)
      const v4u a = opnd(dyi, dzi, 0);
#pragma unroll
      for (int nf = 0; nf < 4; ++nf) acc[0][nf] = mfma_bf(a, wv[nf], acc[0][nf]);
    }
  };

  v4u W[RW][4];
#pragma unroll
  for (int sl = 0; sl < B::NPRE; ++sl) stage(sl);
#pragma unroll
  for (int j = 0; j <= RW - 2; ++j)
    if (j < NI) load_w(W[j], j);
  static_for<NI>([&](auto nc) {
    constexpr int n = decltype(nc)::value;
    constexpr int ph = n / MI;
    if constexpr (n % MI == 0) {
      constexpr int need = B::slab_of_phase(ph) + 1;
      vm_wait_n<B::younger(0, need, ph)>();  // this phase's two slabs have landed
      lds_barrier();                          // ... everywhere; the previous phase is done
      phase_bases(ph);
    }
    vm_wait_for<B::younger(1, n, 0)>(W[n % RW]);
    compute(W[n % RW], n);
    if constexpr (n + RW - 1 < NI) load_w(W[(n + RW - 1) % RW], n + RW - 1);
    if constexpr (n % MI == 0) {
      // the slabs whose buffers the previous phase freed, issued once this
      // phase's first MFMAs are under way (their address lookups then
      // overlap the matrix work)
      constexpr int from = ph == 0 ? B::NPRE : B::last_slab(ph - 1) + 1;
      static_for<B::last_slab(ph) + 1 - from>([&](auto k) { stage(from + decltype(k)::value); });
    }
  });
  vm_wait0();

  // add the waves' tiles through one 128 x 64 sum in LDS: in round r wave w
  // adds its set r, row block (w + r) % 8, so the eight waves work on eight
  // distinct blocks; block c gets its terms from waves c, c-1, .., c-7
  // (mod 8), a fixed order.  Then the sum goes to out (added to it for a
  // later chunk).
  __syncthreads();
  float* red = reinterpret_cast<float*>(lds);
#pragma unroll
  for (int r = 0; r < NRB; ++r) {
    const int blk = (wave + r) & (NRB - 1);
#pragma unroll
    for (int nf = 0; nf < 4; ++nf)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        float* d = &red[(16 * blk + 4 * q + j) * RS + 16 * nf + li];
        *d = r == 0 ? acc[r][nf][j] : *d + acc[r][nf][j];
      }
    __syncthreads();
  }
  const int64_t nrows = 8 * ngroups;
  constexpr int RPR = NW * 64 / 16;  // rows per round, 16 threads a row
#pragma unroll
  for (int rd = 0; rd < 16 * NRB / RPR; ++rd) {
    const int r = RPR * rd + (tid >> 4), cq = (tid & 15) * 4;
    const int64_t row = 8 * g0 + r;
    const int n = n0 + cq;
    v4f sum = *reinterpret_cast<const v4f*>(&red[r * RS + cq]);
    if (row < nrows && n < nn) {
      v4f* dst = reinterpret_cast<v4f*>(out + row * nn + n);
      if (acc_in) sum = *dst + sum;
      if (relu) {
#pragma unroll
        for (int j = 0; j < 4; ++j) sum[j] = fmaxf(sum[j], 0.f);
      }
      *dst = sum;
    }
  }
}

// ---------------------------------------------------------------------------
// Weight gradient.  x [8 ngroups][cin] bf16, dy [8 ngroups][cout] bf16
// (cin, cout % 16 == 0).  A unit is a box of tap offsets, x-offsets
// [x0, x1] by y-offsets [y0, y1] by every z-offset, whose taps read a box of
// positions (x1-x0+2) by (y1-y0+2) by K+1 around a group.  K = 5: ten units
// of one x-offset and two y-offsets, two of two x-offsets and y-offset 4,
// and one of x- and y-offset 4 (half the taps); K = 3: three units of one
// x-offset and every y-offset.  Every unit but the last K = 5 one has
// 10 (K = 5) or 9 (K = 3) taps and at most 36 positions.
// Grid: x = units x ranges (a range is a contiguous run of groups), y =
// blocks of 64 output channels, z = blocks of 64 input channels; NW waves
// of MAXC (tap, 16-channel block) pairs each, two waves per SIMD (one
// wave's LDS waits overlap the other's MFMAs): K = 5 runs two workgroups of
// four waves per compute unit on steps of GS = 4 groups (one workgroup's
// step barrier then leaves the other's waves running), K = 3 one of eight
// waves on steps of 8 groups.  Per step the workgroup stages the unit's
// positions of its GS groups and their 8 GS dY rows; x piece o of box
// position (ix, iy, iz) of the step's group g sits at
// o ^ 2(((iz + 2 iy) & 3) ^ (g & 1)).  dY comes in the sibling-group layout
// dyg[g][c][8] (the eight children of a group contiguous per column), staged
// as [group][64 columns][8]: the B operand of an MFMA (eight consecutive
// octants of one column per lane) is then one 16-byte LDS read.  A transposing load of a
// 16-lane group reads four children of one group in four distinct 32-byte
// slots; the group-parity term moves the next 16-lane group (the next
// group, at the same positions) onto the other four slots of each 256-byte
// bank row, so 32 lanes read 256 distinct bytes.
// dyg [ngroups][cout][8] bf16; part [nranges][K^3][cin][cout].
template <int K, int MAXC, int NW, int GS>
__global__ __launch_bounds__(NW * 64, 8 / NW) void k_conv_bf_dw(const int32_t* __restrict__ nbr,
                                                      int64_t ngroups,
                                                      const uint16_t* __restrict__ x, int cin,
                                                      const uint16_t* __restrict__ dyg, int cout,
                                                      int nranges, float* __restrict__ part) {
  constexpr int R = (K - 1) / 2, S = K + 1, K3 = K * K * K;
  constexpr int NU = K == 5 ? 13 : 3;        // units
  static_assert(GS % 4 == 0 && NW * MAXC >= (K == 5 ? 40 : 36), "tile");
  constexpr int MAXPOS = 36;                 // staged positions per group, at most
  constexpr int XP = GS * MAXPOS * 8;        // pieces of the staged x
  constexpr int YP = GS * 8 * 8;             // pieces of the staged dY rows
  constexpr int BUF = XP + YP + 64;          // ... and a padding slot (loads past the stage)
  constexpr int NXI = GS * MAXPOS / 8, NYI = GS;  // DMA instructions of the x positions, dY rows
  constexpr int NB = 3;                      // stage buffers (two steps in flight)
  constexpr int NBP = NW * 64;               // dwords of a neighbour-row slot (27 GS used)
  static_assert(NBP >= GS * 27, "neighbour slot");
  constexpr int DC = (NXI + NYI + NW - 1) / NW;  // DMA instructions of a stage per wave
  __shared__ __attribute__((aligned(16))) v4u lds[NB * BUF];
  constexpr int NSLOT = 4;                   // neighbour-row slots
  __shared__ __attribute__((aligned(16))) int32_t nbs[NSLOT][NBP];  // neighbour rows of a step's groups

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int li = lane & 15, q = lane >> 4;
  // Work item of this workgroup: workgroups are dealt to the eight XCDs
  // round-robin (x = blockIdx.x % 8), so item = x-th share of the items +
  // blockIdx.x / 8 puts the units of a range, which stage the same rows, on
  // one XCD, where its L2 serves the re-reads.  A bijection on 0..gridDim.x-1.
  const int nitems = (int)gridDim.x, xcd = (int)blockIdx.x & 7, per = nitems >> 3;
  const int item = xcd * per + (xcd < (nitems & 7) ? xcd : (nitems & 7)) + ((int)blockIdx.x >> 3);
  const int unit = item % NU, range = item / NU, nr = nranges;
  int x0, x1, y0, y1;  // the unit's box of tap offsets (indices 0..K-1)
  if (K == 3) {
    x0 = x1 = unit, y0 = 0, y1 = 2;
  } else if (unit < 10) {
    x0 = x1 = unit >> 1, y0 = 2 * (unit & 1), y1 = y0 + 1;
  } else {
    x0 = 2 * (unit - 10), x1 = x0 + 1 < K ? x0 + 1 : x0, y0 = y1 = 4;
  }
  const int NXT = x1 - x0 + 1, NYT = y1 - y0 + 1;  // tap offsets per axis
  const int NY = NYT + 1;                          // positions along y
  const int npos = (NXT + 1) * NY * S;
  const int ntap = NXT * NYT * K;
  const int c0 = blockIdx.z * 64, n0 = blockIdx.y * 64;
  const int CB = (cin - c0 < 64 ? cin - c0 : 64) / 16;
  const int ncombo = ntap * CB;
  const int64_t gbeg = ngroups * range / nr, gend = ngroups * (range + 1) / nr;
  const int nsteps = (int)((gend - gbeg + GS - 1) / GS);

  // Stage st: the unit's x positions, MAXPOS per group (NXI DMA
  // instructions of 64 pieces; positions past npos read zeros), then the
  // 8 GS dY rows (NYI instructions), then the buffer's padding slot: every wave
  // issues DC instructions, and instruction k of wave w is number i = w +
  // NW k.  What a lane loads depends on the step only through the neighbour
  // rows and the step's first group, so the rest is worked out once: for an x
  // instruction, ta = the lane's neighbour entry (27 g + parent cell) and tb
  // = its byte offset in the row block (child offset * cin + channel; 2^31,
  // past any row, for channels past cin and positions past npos); for a dY
  // instruction (one group of the step, its 64 columns of the workgroup's
  // block, 16 bytes each), ta = that group (GS past cout and for padding
  // instructions) and tb = the byte offset of (group, column) in the step's
  // groups.  Loads go through buffer resources over x and dY, absent rows to
  // an offset past the end (zeros).
  const sv4 xr = buf_rsrc(x, (uint32_t)(8 * ngroups * cin * 2));
  const sv4 dr = buf_rsrc(dyg, (uint32_t)(8 * ngroups * cout * 2));
  int ta[DC];
  uint32_t tb[DC], dk[DC];  // dk: the instruction's byte offset in a stage buffer
#pragma unroll
  for (int k = 0; k < DC; ++k) {
    const int i = wave + NW * k;
    ta[k] = GS;
    tb[k] = 0;
    dk[k] = i < NXI ? i * 1024 : i < NXI + NYI ? (XP + (i - NXI) * 64) * 16 : (XP + YP) * 16;
    if (i < NXI) {
      const int s = i * 64 + lane;
      const int pos = s >> 3, g = pos / MAXPOS, p = pos - g * MAXPOS;
      const int ix = p / (NY * S), rem = p - ix * (NY * S), iy = rem / S, iz = rem - iy * S;
      const int ux = x0 + ix - R, uy = y0 + iy - R, uz = iz - R;
      const int o = (s & 7) ^ (2 * (((iz + 2 * iy) & 3) ^ (g & 1)));
      const int ch = c0 + 8 * o;
      ta[k] = p < npos ? 27 * g + ((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1) : 0;
      tb[k] = p < npos && ch < cin
                  ? 2u * (uint32_t)((4 * (ux & 1) + 2 * (uy & 1) + (uz & 1)) * cin + ch)
                  : 0x80000000u;
    } else if (i < NXI + NYI) {
      const int gq = i - NXI, co = n0 + lane;
      ta[k] = co < cout ? gq : GS;
      tb[k] = 16u * (uint32_t)(gq * cout + (co < cout ? co : 0));
    }
  }
  // Instruction k of every wave stages x (XK), or of none (DK); otherwise
  // the kind depends on the wave.
  auto XK = [](auto kc) { return NW * decltype(kc)::value + NW - 1 < NXI; };
  auto DK = [](auto kc) { return NW * decltype(kc)::value >= NXI; };
  // Source offsets of stage st's instructions, from the neighbour rows in
  // slot st % NSLOT (read in one batch, one LDS round trip); formed while the
  // matrix work of an earlier step runs and kept in registers until
  // stage_issue.
  auto stage_src = [&](int st, uint32_t (&src)[DC]) {
    const int64_t gs = gbeg + GS * (int64_t)st;
    const int64_t lf = gend - gs;  // groups of the step inside the range
    const int left = lf < 0 ? 0 : lf > GS ? GS : (int)lf;
    const uint32_t db = (uint32_t)(8 * gs * cout * 2);
    const int32_t* nb = nbs[st % NSLOT];
    int32_t e[DC];
    static_for<DC>([&](auto kc) {
      constexpr int k = decltype(kc)::value;
      if constexpr (!DK(kc)) e[k] = nb[ta[k]];
    });
    static_for<DC>([&](auto kc) {
      constexpr int k = decltype(kc)::value;
      auto ox = [&] { return e[k] >= 0 ? (uint32_t)e[k] * (uint32_t)(2 * cin) + tb[k] : 0x80000000u; };
      auto od = [&] { return ta[k] < left ? db + tb[k] : 0x80000000u; };
      if constexpr (XK(kc))
        src[k] = ox();
      else if constexpr (DK(kc))
        src[k] = od();
      else
        src[k] = wave + NW * k < NXI ? ox() : od();
    });
  };
  // LDS byte address of the stage buffers (buffer b at L0 + b BUF 16)
  const uint32_t L0 = lds_addr(lds);
  auto stage_issue = [&](uint32_t bo, const uint32_t (&src)[DC]) {  // bo: the buffer's offset
    static_for<DC>([&](auto kc) {
      constexpr int k = decltype(kc)::value;
      const sv4 r = XK(kc) ? xr : DK(kc) ? dr : wave + NW * k < NXI ? xr : dr;
      lds_bload16(r, src[k], L0 + bo + dk[k]);
    });
  };
  // neighbour rows of step st's groups into slot st % NSLOT: one dword DMA
  // instruction per wave; entries of groups past the range and past the
  // step's GS x 27 read -1
  const uint32_t NB0 = lds_addr(&nbs[0][0]);
  const int ne = wave * 64 + lane, neg = ne / 27;  // entry of the slot, its group
  auto nb_dma = [&](int st) {
    const int64_t gs = gbeg + GS * (int64_t)st;
    const bool ok = ne < GS * 27 && gs + neg < gend;
    const void* src = ok ? (const void*)(nbr + 27 * gs + ne) : (const void*)&g_minus1;
    lds_load4(src, NB0 + (uint32_t)(((st % NSLOT) * NBP + wave * 64) * 4));
  };

  v4f acc[MAXC][4];
#pragma unroll
  for (int m = 0; m < MAXC; ++m)
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) acc[m][nb] = v4f{0.f, 0.f, 0.f, 0.f};

  // transposing loads: source lane li reads row 4h + (li >> 2) of its
  // 16-lane group's eight, channels 4 (li & 3).. of the 16-channel block;
  // the 16-lane group q takes group 4 sub + q of the step
  const int r4 = li >> 2, tq = li & 3;
  // Each wave multiplies MAXC (tap, 16-channel block) pairs: combo m = wave +
  // NW mi of the unit's ncombo; pairs past ncombo read pair 0's operands and
  // their sums are dropped, so that the loop has no branches.
  auto a_off = [&](int m, int gq, int hh) {  // byte offset of pair m's A load hh
    const int mm = m < ncombo ? m : 0;
    const int it = mm / CB, cb = mm - it * CB;
    const int dxl = it / (NYT * K), dyl = (it / K) % NYT, dzi = it % K;
    const int iy = dyl + (r4 >> 1), iz = dzi + (r4 & 1);  // child 4 hh + r4 of group gq
    const int p = ((dxl + hh) * NY + iy) * S + iz;
    const int o = 2 * cb + (tq >> 1);
    return ((gq * MAXPOS + p) * 8 + (o ^ (2 * (((iz + 2 * iy) & 3) ^ (gq & 1))))) * 16 + (tq & 1) * 8;
  };
  // Byte offsets of this lane's loads in a stage buffer for sub-step 0: pair
  // mi's transposing A loads, and dY fragment nb (group q's eight children
  // of column n0 + 16 nb + li, one 16-byte piece).  A later sub-step sb adds
  // 512 MAXPOS sb (A) or 4096 sb (dY), constants that the loads take as
  // immediate offsets.
  uint32_t pa[MAXC][2], pbq[4];
#pragma unroll
  for (int mi = 0; mi < MAXC; ++mi)
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) pa[mi][hh] = (uint32_t)a_off(wave + NW * mi, q, hh);
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) pbq[nb] = (uint32_t)((XP + q * 64 + 16 * nb + li) * 16);

  // The step's MFMAs in the fixed order (sub-step, pair): the A operand of
  // the pair two ahead and the dY fragments of the next sub-step are read
  // before the current pair's MFMAs are issued (scheduling barriers keep the
  // order), so the LDS latency hides behind matrix work.  mid() runs after
  // the first sub-step's MFMAs.
  auto compute = [&](uint32_t bo, auto&& mid) {
    constexpr int SUBS = GS / 4, NIT = SUBS * MAXC, AD = 2;
    const lds_char* lb = (const lds_char*)(lptr_t)lds + bo;
    auto ld_b = [&](v4u (&b)[4], int sb) {
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
        b[nb] = *reinterpret_cast<const __attribute__((address_space(3))) v4u*>(lb + pbq[nb] + 4096 * sb);
    };
    auto ld_a = [&](int it) {
      const int sb = it / MAXC, mi = it % MAXC;
      const lds_char* p = lb + 512 * MAXPOS * sb;
      return join(__builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p + pa[mi][0])),
                  __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(p + pa[mi][1])));
    };
    v4u bq[2][4], a[AD + 1];
    ld_b(bq[0], 0);
#pragma unroll
    for (int it = 0; it < AD; ++it) a[it] = ld_a(it);
    static_for<NIT>([&](auto itc) {
      constexpr int it = decltype(itc)::value, sb = it / MAXC, mi = it % MAXC;
      if constexpr (it + AD < NIT) a[(it + AD) % (AD + 1)] = ld_a(it + AD);
      if constexpr (mi == 1 && sb + 1 < SUBS) ld_b(bq[(sb + 1) & 1], sb + 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) acc[mi][nb] = mfma_bf(a[it % (AD + 1)], bq[sb & 1][nb], acc[mi][nb]);
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (it == (SUBS > 1 ? MAXC - 1 : MAXC / 2)) mid();
    });
  };

  // Load order of a wave: nb(0..3) (waited for); stage(0), stage(1).  At
  // step st, after the barrier: nb(st+4), stage(st+2).  When step st starts,
  // the loads younger than stage(st) and nb(st+3) are stage(st+1)'s: DC.
  // The addresses of stage(st+3) are formed during step st from slot
  // (st+3) % NSLOT; slot st % NSLOT is refilled at step st, after every wave
  // has formed stage(st)'s addresses (at step st-3, or before the loop).
  uint32_t src[DC];
#pragma unroll
  for (int k = 0; k < 4; ++k) nb_dma(k);
  vm_wait0();
  lds_barrier();
  constexpr uint32_t BB = BUF * 16;  // bytes of a stage buffer
  static_assert(NB == 3, "the buffer offsets below cycle through three buffers");
  stage_src(0, src);
  stage_issue(0, src);
  stage_src(1, src);
  stage_issue(BB, src);
  stage_src(2, src);
  // offsets of the buffers of steps st and st + 2, advanced by a select (not
  // a multiple of st % 3, which the compiler would turn into per-address
  // corrections)
  uint32_t bo = 0, bo2 = 2 * BB;
  for (int st = 0; st < nsteps; ++st) {
    vm_wait_n<DC>();  // stage st and the neighbour rows of step st+3 have landed
    lds_barrier();    // ... everywhere; step st-1 is no longer read
    nb_dma(st + 4);
    stage_issue(bo2, src);
    compute(bo, [&] { stage_src(st + 3, src); });
    bo = __builtin_amdgcn_readfirstlane(bo == 2 * BB ? 0u : bo + BB);
    bo2 = __builtin_amdgcn_readfirstlane(bo2 == 2 * BB ? 0u : bo2 + BB);
  }
  vm_wait0();

  // partial dW of this range: lane (li, q), accumulator j holds input channel
  // c0 + 16 cb + 4q + j, output channel n0 + 16 nb + li
#pragma unroll
  for (int mi = 0; mi < MAXC; ++mi) {
    const int m = wave + NW * mi;
    if (m < ncombo) {
      const int it = m / CB, cb = m - it * CB;
      const int dxl = it / (NYT * K), dyl = (it / K) % NYT, dzi = it % K;
      const int t = ((x0 + dxl) * K + y0 + dyl) * K + dzi;
      float* dst = part + ((int64_t)range * K3 + t) * cin * cout;
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int n = n0 + 16 * nb + li;
        if (n < cout) {
#pragma unroll
          for (int j = 0; j < 4; ++j)
            dst[(int64_t)(c0 + 16 * cb + 4 * q + j) * cout + n] = acc[mi][nb][j];
        }
      }
    }
  }
}

inline unsigned blocks(int64_t n, int per) { return (unsigned)oc::cdiv(n, per); }

size_t wp_bytes(int K, int kk, int nn) { return oc::align256((size_t)kk * K * K * K * nn * 2); }

// Work items of the weight gradient for nranges ranges: units x ranges.
int dw_items(int K, int nranges) { return (K == 5 ? 13 : 3) * nranges; }

int dw_ranges(const oc_octree* t, int l, int K, int cin, int cout) {
  const int64_t G = t->M[l - 1];
  const int64_t per = oc::cdiv(cout, 64) * oc::cdiv(cin, 64) * (K == 5 ? 13 : 3);
  // about two items per compute unit (one resident at a time), at least 16
  // groups per range
  int64_t r = std::max<int64_t>(1, (2 * (int64_t)oc::cu_count()) / per);
  r = std::min<int64_t>(r, std::max<int64_t>(1, G / 16));
  return (int)std::max<int64_t>(1, r);
}

void wprep(const uint16_t* w, int K, int kk, int nn, int flip, uint16_t* wp, hipStream_t s) {
  const int K3 = K * K * K;
  oc::launch(k_bf_wprep, dim3(blocks((int64_t)kk * K3 * nn, TB)), dim3(TB), 0, s, w, K3,
                     kk, nn, flip, wp);
}

// Tiles of 16 groups (k_conv_bfw) for K = 5: half the weight reads per row
// of the 8-group kernel.  Its weight loads have no per-lane masks, so every
// chunk must hold whole 32-channel halves and the columns whole blocks of 64;
// K = 3 keeps the 8-group kernel.
// Tile groups and waves of the K = 5 forward (k_conv_bfw): 8-group tiles of
// four waves, two workgroups per compute unit, so that one workgroup's
// epilogue (its waves' partial tiles added through LDS) runs beside the
// other's MFMAs.
constexpr int BFW_GT = 8, BFW_NW = 4;

bool wide_tiles(int K, int kk, int nn, int64_t rows) {
  return K == 5 && kk % 32 == 0 && nn % 64 == 0 && rows * kk * 2 < ((int64_t)1 << 31);
}

template <int K, int HC, bool FLIP>
void launch_chunk(const oc_octree* t, int l, const uint16_t* x, int kk, const uint16_t* wp, int nn,
                  int chunk, float* out, int acc_in, int relu, bool main, hipStream_t s) {
  const int64_t G = t->M[l - 1];
  const bool wide = wide_tiles(K, kk, nn, 8 * G);
  const dim3 grid(blocks(G, wide ? BFW_GT : 8), blocks(nn, 64));
  const dim3 block(wide ? BFW_NW * 64 : 512);
  auto kern = k_conv_bf<K, HC, FLIP>;
  if constexpr (K == 5) {
    if (wide) kern = k_conv_bfw<K, HC, FLIP, BFW_GT, BFW_NW>;
  }
  if (main)
    oc::launch_main(kern, grid, block, s, (const int32_t*)t->nbr[l], G, x, kk, wp, nn, chunk, out,
                    acc_in, relu);
  else
    oc::launch(kern, grid, block, 0, s, (const int32_t*)t->nbr[l], G, x, kk, wp, nn, chunk, out,
               acc_in, relu);
}

// out = conv over kk reduction channels, in chunks of 64 added in order; the
// first chunk's launch carries the profiling events.
template <bool FLIP>
void launch_conv(const oc_octree* t, int l, int K, const uint16_t* x, int kk, const uint16_t* wp,
                 int nn, float* out, int relu, hipStream_t s) {
  const int nch = (int)oc::cdiv(kk, 64);
  for (int c = 0; c < nch; ++c) {
    const bool two = kk - 64 * c > 32;  // the chunk has a second half of 32 channels
    const int acc_in = c > 0, r = c + 1 == nch ? relu : 0;
    if (K == 5) {
      if (two)
        launch_chunk<5, 2, FLIP>(t, l, x, kk, wp, nn, c, out, acc_in, r, c == 0, s);
      else
        launch_chunk<5, 1, FLIP>(t, l, x, kk, wp, nn, c, out, acc_in, r, c == 0, s);
    } else {
      if (two)
        launch_chunk<3, 2, FLIP>(t, l, x, kk, wp, nn, c, out, acc_in, r, c == 0, s);
      else
        launch_chunk<3, 1, FLIP>(t, l, x, kk, wp, nn, c, out, acc_in, r, c == 0, s);
    }
  }
}

}  // namespace

namespace oc {

bool conv_bf16_supported(int K, int cin, int cout) {
  return (K == 3 || K == 5) && cin % 16 == 0 && cout % 16 == 0;
}

void conv_bf16_kernel_name(int K, int cin, int cout, int pass, int64_t rows, char* buf,
                           size_t n) {
  const int kk = pass == 1 ? cout : cin;  // reduction channels of the first chunk
  if (pass == 2)
    snprintf(buf, n, K == 5 ? "k_conv_bf_dw<5, 10, 4, 4>" : "k_conv_bf_dw<3, 5, 8, 8>");
  else if (wide_tiles(K, kk, pass == 1 ? cin : cout, rows))
    snprintf(buf, n, "k_conv_bfw<%d, %d, %s, %d, %d>", K, kk > 32 ? 2 : 1,
             pass == 1 ? "true" : "false", BFW_GT, BFW_NW);
  else
    snprintf(buf, n, "k_conv_bf<%d, %d, %s>", K, kk > 32 ? 2 : 1, pass == 1 ? "true" : "false");
}

size_t conv_bf16_fwd_ws(int K, int cin, int cout) { return wp_bytes(K, cin, cout); }

size_t conv_bf16_bwd_ws(const oc_octree* t, int l, int K, int cin, int cout) {
  const size_t dy16 = align256((size_t)t->N[l] * cout * 2);
  const size_t part =
      align256((size_t)dw_ranges(t, l, K, cin, cout) * K * K * K * cin * cout * sizeof(float));
  return 2 * dy16 + wp_bytes(K, cout, cin) + part;  // dy rounded to bf16: row-major, by group
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
  uint16_t* dy16 = (uint16_t*)p;  // dy rounded to bf16, row-major (input gradient)
  p += align256((size_t)N * cout * 2);
  uint16_t* dyg = (uint16_t*)p;   // ... in the sibling-group layout (weight gradient)
  p += align256((size_t)N * cout * 2);
  uint16_t* wpf = (uint16_t*)p;
  p += wp_bytes(K, cout, cin);
  float* part = (float*)p;
  const int64_t n = N * cout;
  const int vec = (uintptr_t)dy % 16 == 0 && (!ym || (uintptr_t)ym % 16 == 0);
  if (dw)
    oc::launch(k_bf_cvt_g, dim3(blocks(G, 8), blocks(cout, 64)), dim3(TB), 0, s, dy, ym, G, cout,
               vec && cout % 4 == 0, dyg, dx ? dy16 : nullptr);
  else
    oc::launch(k_bf_cvt, dim3(blocks(n, 4 * TB)), dim3(TB), 0, s, dy, ym, n, vec, dy16);
  if (dx) {
    wprep(w, K, cout, cin, 1, wpf, s);
    launch_conv<true>(t, l, K, dy16, cout, wpf, cin, dx, 0, s);
  }
  if (dw) {
    const int K3 = K * K * K;
    const int nr = dw_ranges(t, l, K, cin, cout);
    const dim3 grid((unsigned)dw_items(K, nr), blocks(cout, 64), blocks(cin, 64));
    if (K == 5)
      launch_main(k_conv_bf_dw<5, 10, 4, 4>, grid, dim3(256), s, (const int32_t*)t->nbr[l], G, x,
                  cin, dyg, cout, nr, part);
    else
      launch_main(k_conv_bf_dw<3, 5, 8, 8>, grid, dim3(512), s, (const int32_t*)t->nbr[l], G, x,
                  cin, dyg, cout, nr, part);
    const int64_t E = (int64_t)K3 * cin * cout;
    oc::launch(k_bf_sum, dim3(blocks(E, 4 * TB)), dim3(TB), 0, s, part, nr, E, dw);
  }
}

void round_bf16(const float* x, int64_t n, uint16_t* y, hipStream_t s) {
  const bool vec = ((uintptr_t)x % 16 == 0) && ((uintptr_t)y % 16 == 0);
  oc::launch_main(k_bf_round, dim3(blocks(n, 8 * TB)), dim3(TB), s, x, n, (int)vec, y);
}

}  // namespace oc
