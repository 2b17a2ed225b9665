// Octree construction on the GPU (Sec. 3.1 of O-CNN, arXiv 1712.01537).
//
// The paper builds octrees offline on the CPU by breadth-first subdivision and
// searches neighbours through a hash table from shuffle keys to indices.  Here
// every depth l of the batch is an occupancy bitmap over its B 8^l cells, cell
// index = shape << 3l | shuffle key, so that bit order is key order:
//   1. each point sets the bit of its leaf cell (quantised at the leaf depth),
//      through LDS bitmaps of consecutive cell ranges;
//   2. the bit of a cell at depth l is the OR of its eight children at l+1,
//      which are one byte of the depth-(l+1) bitmap; depths shallower than
//      full_depth are all ones (Sec. 4: every octant down to depth 2 exists);
//   3. one exclusive popcount scan over the words of all depths gives every
//      set bit its rank, which is its label minus one (Sec. 3.1 "Label");
//   4. after the one host read of the per-depth counts, each non-empty octant
//      of depth l-1 with rank r emits its children, rows 8r..8r+7 of depth l
//      (keys, labels, label->row map; Sec. 3.1 "Label"), and its row of the
//      sibling-group neighbour table: the first-child row 8 rank of each of the
//      27 depth-(l-1) octants around it, found by a bit test and a rank query
//      (this replaces the hash table H of Sec. 3.2; every neighbour within
//      offset +-2 of the eight siblings is reachable from these 27 entries,
//      Fig. 4);
//   5. the input signal (Sec. 3.1) is the mean normal of each leaf's points,
//      summed in LDS in 64-bit fixed point scaled to the largest normal
//      component in the batch, so that the sums do not depend on the order of
//      the atomics.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <vector>

#include "common.h"

namespace {

constexpr int TB = 256;

// Bit i of v moves to bit 3i (v < 2^10).
__device__ __forceinline__ uint32_t spread3(uint32_t v) {
  v &= 0x3ffu;
  v = (v | (v << 16)) & 0x030000FFu;
  v = (v | (v << 8)) & 0x0300F00Fu;
  v = (v | (v << 4)) & 0x030C30C3u;
  v = (v | (v << 2)) & 0x09249249u;
  return v;
}

// Inverse of spread3: bits 0, 3, 6, ... of v packed into the low bits.
__device__ __forceinline__ uint32_t squeeze3(uint32_t v) {
  v &= 0x09249249u;
  v = (v | (v >> 2)) & 0x030C30C3u;
  v = (v | (v >> 4)) & 0x0300F00Fu;
  v = (v | (v >> 8)) & 0x030000FFu;
  v = (v | (v >> 16)) & 0x3ffu;
  return v;
}

// Shuffle key x1y1z1...xlylzl (Sec. 3.1): x's bit i lands at key bit 3i+2.
__device__ __forceinline__ uint32_t shuffle_key(uint32_t x, uint32_t y, uint32_t z) {
  return (spread3(x) << 2) | (spread3(y) << 1) | spread3(z);
}

// Layout of the concatenated per-depth bitmaps (kernel argument).
struct Levels {
  int depth, full_depth, batch;
  int64_t cells[OC_MAX_DEPTH + 1];  // B 8^l
  int64_t wbase[OC_MAX_DEPTH + 2];  // first word of depth l; wbase[depth+1] = all words
};

// Shape offsets (kernel argument; batch <= 256).
struct Shapes {
  int32_t offs[257];
};

__device__ __forceinline__ int level_of_word(const Levels& L, int64_t w) {
  int l = 0;
  while (l < L.depth && w >= L.wbase[l + 1]) ++l;
  return l;
}

// Rank of cell c among the set cells of depth l: exclusive prefix of the word
// minus the count of shallower depths, plus the set bits below c in its word.
__device__ __forceinline__ int32_t rank_in(const uint32_t* __restrict__ bits,
                                           const int32_t* __restrict__ pre, const Levels& L,
                                           int l, int32_t mbase, uint64_t c, uint32_t* word) {
  const int64_t w = L.wbase[l] + (int64_t)(c >> 5);
  const uint32_t v = bits[w];
  *word = v;
  return pre[w] - mbase + __popc(v & ((1u << (c & 31)) - 1u));
}

// ---------------------------------------------------------------------------
// 1. leaf occupancy.  k_quant: leaf cell of every point (~0 for a point outside
//    [0,1]^3); bstat[block] = {flags: bit 0 such a point or NaN, bit 1 a
//    non-finite normal; the largest |normal component| (float bits)}.
//    k_mark: workgroup k owns leaf cells [k 32 nwd, (k+1) 32 nwd) as an LDS
//    bitmap of nwd words (a power of two from 1024 to 8192, so that a few
//    hundred workgroups cover the leaf depth), scans the points of the shapes
//    that overlap it, derives the words of the coarser depths whose part of
//    the chunk is whole words (up = log8(32 nwd / 32) of them; bit j of depth
//    l = byte j of depth l+1 != 0) and stores all of them; the workgroups also
//    fill the depths shallower than full_depth with ones.  No global atomics.

__global__ __launch_bounds__(TB) void k_quant(const float* __restrict__ pts,
                                              const float* __restrict__ nrm, Shapes S, int B,
                                              int P, int d, uint32_t* __restrict__ leafcell,
                                              uint2* __restrict__ bstat) {
  __shared__ int32_t so[257];
  for (int k = threadIdx.x; k <= B; k += TB) so[k] = S.offs[k];
  __syncthreads();
  const int i0 = blockIdx.x * TB + threadIdx.x;
  const bool live = i0 < P;
  const int i = live ? i0 : P - 1;  // the block reductions need every lane
  int lo = 0, hi = B - 1;  // last shape b with offs[b] <= i
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (so[mid] <= i) lo = mid;
    else hi = mid - 1;
  }
  const float scale = (float)(1u << d);  // exact power of two
  const uint32_t qmax = (1u << d) - 1u;
  uint32_t q[3];
  bool bad = false;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    const float p = pts[3 * (int64_t)i + a];
    const bool ok = p >= 0.0f && p <= 1.0f;  // false for NaN
    bad |= !ok;
    const uint32_t c = ok ? (uint32_t)floorf(p * scale) : 0u;
    q[a] = c > qmax ? qmax : c;
  }
  float m = 0.f;
  bool nbad = false;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    const float n = nrm[3 * (int64_t)i + a];
    nbad |= !isfinite(n);
    m = fmaxf(m, fabsf(n));
  }
  // flags and the largest |component| of the workgroup (float bits order
  // non-negative floats)
  __shared__ uint2 ws[TB / 64];
  uint32_t fl = (bad ? 1u : 0u) | (nbad ? 2u : 0u), mb = nbad ? 0u : __float_as_uint(m);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t o = __shfl_xor(mb, off, 64);
    fl |= __shfl_xor(fl, off, 64);
    mb = o > mb ? o : mb;
  }
  if ((threadIdx.x & 63) == 0) ws[threadIdx.x >> 6] = make_uint2(fl, mb);
  __syncthreads();
  if (threadIdx.x == 0) {
    uint2 v = make_uint2(0u, 0u);
#pragma unroll
    for (int k = 0; k < TB / 64; ++k) {
      v.x |= ws[k].x;
      v.y = ws[k].y > v.y ? ws[k].y : v.y;
    }
    bstat[blockIdx.x] = v;
  }
  if (!live) return;
  const uint64_t c = ((uint64_t)lo << (3 * d)) | shuffle_key(q[0], q[1], q[2]);
  leafcell[i] = bad ? 0xFFFFFFFFu : (uint32_t)c;
}

constexpr int MK_TB = 1024;
constexpr int MK_UNROLL = 4;  // points in flight per thread

// Leaf-depth words per k_mark workgroup and the coarser depths it derives.
struct MarkCfg {
  int words, up;
  size_t lds;  // bytes: the chunk's words at every derived depth
};
MarkCfg mark_cfg(int64_t leaf_cells) {
  MarkCfg m;
  m.words = 1024;
  while (m.words < 8192 && (int64_t)m.words * 32 * 256 < leaf_cells) m.words *= 2;
  m.up = 0;
  while (((int64_t)m.words * 32 >> (3 * (m.up + 1))) % 32 == 0 &&
         ((int64_t)m.words * 32 >> (3 * (m.up + 1))) > 0)
    ++m.up;
  int64_t n = 0;
  for (int j = 0; j <= m.up; ++j) n += (int64_t)m.words >> (3 * j);
  m.lds = 4 * (size_t)n;
  return m;
}

__global__ __launch_bounds__(MK_TB) void k_mark(const uint32_t* __restrict__ leafcell, Shapes S,
                                                Levels L, int chunk_words, int up,
                                                uint32_t* __restrict__ bits) {
  extern __shared__ uint32_t w[];
  const int d = L.depth;
  const int64_t MK_CELLS = 32ll * chunk_words;
  // depths shallower than full_depth: all ones (grid-stride over their words)
  const int64_t nforced = L.wbase[L.full_depth];
  for (int64_t k = (int64_t)blockIdx.x * MK_TB + threadIdx.x; k < nforced;
       k += (int64_t)gridDim.x * MK_TB) {
    const int l = level_of_word(L, k);
    const int64_t left = L.cells[l] - (k - L.wbase[l]) * 32;
    bits[k] = left >= 32 ? ~0u : ((1u << left) - 1u);
  }
  const int64_t c0 = (int64_t)blockIdx.x * MK_CELLS;
  const int64_t c1 = c0 + MK_CELLS < L.cells[d] ? c0 + MK_CELLS : L.cells[d];
  const int nwd = (int)((c1 - c0 + 31) >> 5);
  for (int k = threadIdx.x; k < nwd; k += MK_TB) w[k] = 0u;
  __syncthreads();
  const int64_t per = (int64_t)1 << (3 * d);  // cells per shape
  const int b0 = (int)(c0 / per), b1 = (int)((c1 - 1) / per);
  const int i1 = S.offs[b1 + 1];
  for (int i = S.offs[b0] + threadIdx.x; i < i1; i += MK_UNROLL * MK_TB) {
    uint32_t c[MK_UNROLL];
#pragma unroll
    for (int u = 0; u < MK_UNROLL; ++u)
      c[u] = i + u * MK_TB < i1 ? leafcell[i + u * MK_TB] : 0xFFFFFFFFu;
#pragma unroll
    for (int u = 0; u < MK_UNROLL; ++u)
      if (c[u] != 0xFFFFFFFFu && (int64_t)c[u] >= c0 && (int64_t)c[u] < c1)
        atomicOr(&w[(c[u] - c0) >> 5], 1u << (c[u] & 31));
  }
  __syncthreads();
  if (d >= L.full_depth) {
    uint32_t* dst = bits + L.wbase[d] + (c0 >> 5);
    for (int k = threadIdx.x; k < nwd; k += MK_TB) dst[k] = w[k];
  }
  // coarser depths d-1 .. d-up: the chunk's cells there start on a word
  // boundary (32 chunk_words / 8^up is a multiple of 32)
  uint32_t* fine = w;
  int nfine = nwd;
  int off = chunk_words;
  for (int j = 1; j <= up && d - j >= L.full_depth; ++j) {
    const int l = d - j;
    uint32_t* coarse = w + off;
    const int64_t cc0 = c0 >> (3 * j), ncell = (c1 - c0) >> (3 * j);
    const int ncw = (int)((ncell + 31) >> 5);
    for (int k = threadIdx.x; k < ncw; k += MK_TB) {
      uint32_t v = 0u;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const uint32_t cw = 8 * k + t < nfine ? fine[8 * k + t] : 0u;
#pragma unroll
        for (int b = 0; b < 4; ++b) v |= ((cw >> (8 * b)) & 0xFFu) ? (1u << (4 * t + b)) : 0u;
      }
      coarse[k] = v;
      bits[L.wbase[l] + (cc0 >> 5) + k] = v;
    }
    __syncthreads();
    fine = coarse;
    nfine = ncw;
    off += chunk_words >> (3 * j);
  }
}

// ---------------------------------------------------------------------------
// 2. depths more than `up` above the leaves (and not forced): bit j of depth
//    l = (byte j of depth l+1 != 0).

__global__ __launch_bounds__(TB) void k_reduce(Levels L, int l, uint32_t* __restrict__ bits) {
  const int64_t w = (int64_t)blockIdx.x * TB + threadIdx.x;
  const int64_t nw = L.wbase[l + 1] - L.wbase[l], nc = L.wbase[l + 2] - L.wbase[l + 1];
  if (w >= nw) return;
  const uint32_t* child = bits + L.wbase[l + 1] + 8 * w;
  uint32_t v = 0u;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const uint32_t cw = 8 * w + k < nc ? child[k] : 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j) v |= ((cw >> (8 * j)) & 0xFFu) ? (1u << (4 * k + j)) : 0u;
  }
  bits[L.wbase[l] + w] = v;
}

// ---------------------------------------------------------------------------
// 3. exclusive scan of the word popcounts of all depths: pre[w] = set bits
//    before word w; pre[nw] = total.  Blocks of SCAN_W words: k_scan_a sums
//    each block, k_scan_c adds the sums of the blocks before its own, scans
//    its words and, for every set bit, writes the cell in rank order (step 4).

constexpr int SCAN_PER = 2;
constexpr int SCAN_W = TB * SCAN_PER;

__device__ __forceinline__ int32_t block_excl_scan(int32_t v, int32_t* total) {
  __shared__ int32_t ws[TB / 64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  int32_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) ws[wv] = x;
  __syncthreads();
  int32_t before = 0, all = 0;
#pragma unroll
  for (int k = 0; k < TB / 64; ++k) {
    if (k < wv) before += ws[k];
    all += ws[k];
  }
  __syncthreads();
  *total = all;
  return before + x - v;
}

__global__ __launch_bounds__(TB) void k_scan_a(const uint32_t* __restrict__ bits, int64_t nw,
                                               int32_t* __restrict__ bsum) {
  const int64_t w0 = (int64_t)blockIdx.x * SCAN_W + threadIdx.x * SCAN_PER;
  int32_t s = 0;
#pragma unroll
  for (int k = 0; k < SCAN_PER; ++k)
    if (w0 + k < nw) s += __popc(bits[w0 + k]);
  int32_t total;
  block_excl_scan(s, &total);
  if (threadIdx.x == 0) bsum[blockIdx.x] = total;
}

// 4. (in k_scan_c) cell of every set bit, in rank order over all depths:
//    ucell[pre + k].  The thread holding the first word of depth l reports
//    pre there (info[2 + l], l <= depth + 1, the last one the total), so
//    that M_l = info[3 + l] - info[2 + l]; workgroup 0 also reports the flags
//    and largest |normal component| of the nq blocks of k_quant (info[0],
//    info[1]).
__global__ __launch_bounds__(TB) void k_scan_c(Levels L, const uint32_t* __restrict__ bits,
                                               int64_t nw, const int32_t* __restrict__ bsum,
                                               int32_t* __restrict__ pre,
                                               uint32_t* __restrict__ ucell,
                                               const uint2* __restrict__ bstat, int nq,
                                               uint32_t* __restrict__ info) {
  // set bits of the blocks before this one
  int32_t sb = 0;
  for (int k = threadIdx.x; k < (int)blockIdx.x; k += TB) sb += bsum[k];
  int32_t before;
  block_excl_scan(sb, &before);
  const int64_t w0 = (int64_t)blockIdx.x * SCAN_W + threadIdx.x * SCAN_PER;
  uint32_t wd[SCAN_PER];
  int32_t c[SCAN_PER], s = 0;
#pragma unroll
  for (int k = 0; k < SCAN_PER; ++k) {
    wd[k] = w0 + k < nw ? bits[w0 + k] : 0u;
    c[k] = __popc(wd[k]);
    s += c[k];
  }
  int32_t total;
  int32_t run = before + block_excl_scan(s, &total);
  int l = level_of_word(L, w0 < nw ? w0 : nw - 1);
#pragma unroll
  for (int k = 0; k < SCAN_PER; ++k) {
    const int64_t w = w0 + k;
    if (w < nw) {
      while (l < L.depth && w >= L.wbase[l + 1]) ++l;
      if (w == L.wbase[l]) info[2 + l] = (uint32_t)run;
      pre[w] = run;
      const uint32_t base = (uint32_t)((w - L.wbase[l]) * 32);
      int32_t r = run;
      uint32_t m = wd[k];
      while (m) {
        ucell[r++] = base + (uint32_t)(__ffs(m) - 1);
        m &= m - 1u;
      }
      run += c[k];
    }
  }
  if (w0 < nw && w0 + SCAN_PER >= nw) {  // the thread of the last word
    pre[nw] = run;
    info[3 + L.depth] = (uint32_t)run;
  }
  if (blockIdx.x != 0) return;
  __shared__ uint2 ws[TB / 64];
  const int t = threadIdx.x;
  uint32_t fl = 0u, mb = 0u;
  for (int k = t; k < nq; k += TB) {
    const uint2 v = bstat[k];
    fl |= v.x;
    mb = v.y > mb ? v.y : mb;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t o = __shfl_xor(mb, off, 64);
    fl |= __shfl_xor(fl, off, 64);
    mb = o > mb ? o : mb;
  }
  if ((t & 63) == 0) ws[t >> 6] = make_uint2(fl, mb);
  __syncthreads();
  if (t == 0) {
    uint2 v = make_uint2(0u, 0u);
#pragma unroll
    for (int k = 0; k < TB / 64; ++k) {
      v.x |= ws[k].x;
      v.y = ws[k].y > v.y ? ws[k].y : v.y;
    }
    info[0] = v.x;
    info[1] = v.y;
  }
}

// ---------------------------------------------------------------------------
// 5. mean normal of every leaf.  The leaves of shape b hold a contiguous range
//    of ranks; workgroup (b, k) owns ranks lo .. lo + LM_LEAVES - 1 of it (a
//    contiguous cell range), scans the shape's points and adds the normals of
//    those in range into LDS in 64-bit fixed point, 2^s units with
//    s = 62 - e for P * max|n| < 2^e: no sum can overflow and integer
//    additions make the result independent of their order.  The scan reads
//    four cells per 16-byte load; each wave queues its in-range points in LDS
//    and adds them with all lanes, so the few in-range points of a pass cost
//    one round of lookups and atomics rather than one per point slot.

constexpr int LM_TB = 1024;
constexpr int LM_LEAVES = 2048;  // 2048 * (3 * 8 + 4) bytes of LDS, plus the queues
constexpr int LM_UNROLL = 2;     // 16-byte loads (four points each) per thread and pass

__device__ __forceinline__ int fixed_shift(uint32_t maxbits, int P) {
  const double m = (double)__uint_as_float(maxbits) * (double)P;
  int e = 0;
  if (m > 0.0) frexp(m, &e);  // m < 2^e
  return 62 - e;
}

__global__ __launch_bounds__(LM_TB) void k_leaf_mean(const float* __restrict__ nrm,
                                                     const uint32_t* __restrict__ leafcell,
                                                     Shapes S, int P,
                                                     Levels L, const uint32_t* __restrict__ bits,
                                                     const int32_t* __restrict__ pre,
                                                     const uint32_t* __restrict__ ucell,
                                                     const uint32_t* __restrict__ info,
                                                     float* __restrict__ leafmean) {
  constexpr int NP = 4 * LM_UNROLL;  // points per lane and pass
  __shared__ unsigned long long sum[3 * LM_LEAVES];
  __shared__ int32_t cnt[LM_LEAVES];
  __shared__ uint2 queue[LM_TB / 64][NP * 64];  // per wave: (point, cell) in range
  if (info[0]) return;  // the build fails on any bad input
  const int b = blockIdx.x, d = L.depth;
  const int32_t mb = pre[L.wbase[d]], md = pre[L.wbase[d + 1]] - mb;
  const uint64_t cfirst = (uint64_t)b << (3 * d), cend = (uint64_t)(b + 1) << (3 * d);
  uint32_t word;
  const int32_t r0 = rank_in(bits, pre, L, d, mb, cfirst, &word);
  const int32_t r1 = cend >= (uint64_t)L.cells[d] ? md : rank_in(bits, pre, L, d, mb, cend, &word);
  const int32_t lo = r0 + (int32_t)blockIdx.y * LM_LEAVES;
  if (lo >= r1) return;
  const int32_t hi = lo + LM_LEAVES < r1 ? lo + LM_LEAVES : r1;
  const uint32_t clo = ucell[mb + lo];
  const uint64_t chi = hi < r1 ? (uint64_t)ucell[mb + hi] : cend;  // cells [clo, chi)
  for (int j = threadIdx.x; j < hi - lo; j += LM_TB) {
    sum[3 * j] = sum[3 * j + 1] = sum[3 * j + 2] = 0ull;
    cnt[j] = 0;
  }
  __syncthreads();
  const int s = fixed_shift(info[1], P);
  auto in_range = [&](uint32_t c) { return c >= clo && (uint64_t)c < chi; };
  // a point of the shape whose leaf is in range adds its normal and a count
  auto add = [&](int64_t i, uint32_t c) {
    const int64_t wi = L.wbase[d] + (int64_t)(c >> 5);
    const int32_t j = pre[wi] - mb + __popc(bits[wi] & ((1u << (c & 31)) - 1u)) - lo;
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      const long long v = llrint(ldexp((double)nrm[3 * i + a], s));
      atomicAdd(&sum[3 * j + a], (unsigned long long)v);
    }
    atomicAdd(&cnt[j], 1);
  };
  // the shape's points: a 16-byte-aligned body read four cells per load, and
  // the points before and after it
  const int i0 = S.offs[b], i1 = S.offs[b + 1];
  const int a0 = ((i0 + 3) & ~3) < i1 ? ((i0 + 3) & ~3) : i1;
  const int a1 = (i1 & ~3) > a0 ? (i1 & ~3) : a0;
  const int t = threadIdx.x;
  if (t < a0 - i0 && in_range(leafcell[i0 + t])) add(i0 + t, leafcell[i0 + t]);
  if (t < i1 - a1 && in_range(leafcell[a1 + t])) add(a1 + t, leafcell[a1 + t]);
  // body: LM_UNROLL 16-byte loads per thread and pass.  Most points of a
  // pass are out of range, so each wave compacts its in-range points into a
  // queue in LDS (ballot + lane count) and then adds them with every lane
  // busy, after issuing the next pass's cell loads.
  const uint4* lc4 = reinterpret_cast<const uint4*>(leafcell);
  const int v1 = a1 >> 2;
  const int lane = t & 63;
  uint2* qw = queue[t >> 6];
  auto load_cells = [&](int v, uint32_t (&c)[NP]) {
#pragma unroll
    for (int u = 0; u < LM_UNROLL; ++u) {
      uint4 q = make_uint4(0u, 0u, 0u, 0u);
      if (v + u * LM_TB < v1) q = lc4[v + u * LM_TB];
      c[4 * u] = q.x, c[4 * u + 1] = q.y, c[4 * u + 2] = q.z, c[4 * u + 3] = q.w;
    }
  };
  uint32_t cc[NP];
  const int vb = (a0 >> 2) + t - lane;  // the wave's first load index
  load_cells(vb + lane, cc);
  // every lane of a wave runs the same passes (wave-uniform loop bounds)
  for (int v = vb; v < v1; v += LM_UNROLL * LM_TB) {
    int n = 0;  // in-range points queued by the wave
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      const int vi = v + lane + (k / 4) * LM_TB;
      const bool in = vi < v1 && in_range(cc[k]);
      const uint64_t m = __ballot(in);
      if (in) {
        const int pos = n + __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                      __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        qw[pos] = make_uint2((uint32_t)(4 * vi + (k & 3)), cc[k]);
      }
      n += __popcll(m);
    }
    load_cells(v + LM_UNROLL * LM_TB + lane, cc);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (int r = lane; r < n; r += 64) {
      const uint2 e = qw[r];
      add((int64_t)e.x, e.y);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  __syncthreads();
  const double unit = ldexp(1.0, -s);
  for (int j = threadIdx.x; j < hi - lo; j += LM_TB) {
    const double inv = unit / (double)cnt[j];
    float* o = leafmean + 3 * (int64_t)(lo + j);
#pragma unroll
    for (int a = 0; a < 3; ++a) o[a] = (float)((double)(long long)sum[3 * j + a] * inv);
  }
}

// ---------------------------------------------------------------------------
// 6. emission.  Item it < B: root b of depth 0.  Otherwise the non-empty
//    octant of rank r at depth l-1 (items ibase[l] + r): its children are rows
//    8r .. 8r+7 of depth l, its neighbour row is nbr_l[r].

struct Emit {
  int32_t mbase[OC_MAX_DEPTH + 2];  // set bits before depth l (all depths)
  int64_t ibase[OC_MAX_DEPTH + 2];  // first item of depth l (l >= 1); ibase[d+1] = items
  uint32_t* keys[OC_MAX_DEPTH + 1];
  int32_t* labels[OC_MAX_DEPTH + 1];
  int32_t* rows[OC_MAX_DEPTH + 1];
  int32_t* nbr[OC_MAX_DEPTH + 1];
  float* signal;
};

__global__ __launch_bounds__(TB) void k_emit(Levels L, Emit E, const uint32_t* __restrict__ bits,
                                             const int32_t* __restrict__ pre,
                                             const uint32_t* __restrict__ ucell,
                                             const float* __restrict__ leafmean) {
  // 16 lanes per item: lane j < 8 emits child j and every lane neighbours j
  // and j + 16 (< 27), their lookups in flight together
  const int64_t it = ((int64_t)blockIdx.x * TB + threadIdx.x) >> 4;
  const int j = threadIdx.x & 15;
  const int d = L.depth;
  if (it >= E.ibase[d + 1]) return;
  uint32_t word;
  if (it < L.batch) {  // depth 0: one root per shape
    if (j != 0) return;
    const int b = (int)it;
    const int32_t r = rank_in(bits, pre, L, 0, E.mbase[0], (uint64_t)b, &word);
    const bool on = (word >> (b & 31)) & 1u;
    E.keys[0][b] = (uint32_t)b << 24;
    E.labels[0][b] = on ? r + 1 : 0;
    if (on) E.rows[0][r] = b;
    return;
  }
  int l = 1;
  while (l < d && it >= E.ibase[l + 1]) ++l;
  const int32_t r = (int32_t)(it - E.ibase[l]);
  const int pl = l - 1;
  const uint64_t p = ucell[E.mbase[pl] + r];  // parent cell at depth l-1

  // every rank lookup of the lane first (clamped to a valid word when
  // absent), then the stores
  const uint32_t pkb = 3u * (uint32_t)pl;
  const uint32_t pshape = (uint32_t)(p >> pkb);
  const uint32_t pkey = (uint32_t)p & (uint32_t)((1ull << pkb) - 1ull);
  const int side = 1 << pl;
  const int px = (int)squeeze3(pkey >> 2), py = (int)squeeze3(pkey >> 1), pz = (int)squeeze3(pkey);
  uint64_t q[2];
  bool in[2];
  uint32_t qw[2];
  int32_t qp[2];
#pragma unroll
  for (int h = 0; h < 2; ++h) {  // neighbour jj = j + 16 h of the parent at depth l-1
    const int jj = j + 16 * h;
    const int nx = px + jj / 9 - 1, ny = py + (jj / 3) % 3 - 1, nz = pz + jj % 3 - 1;
    in[h] = jj < 27 && nx >= 0 && nx < side && ny >= 0 && ny < side && nz >= 0 && nz < side;
    q[h] = in[h] ? ((uint64_t)pshape << pkb) |
                       shuffle_key((uint32_t)nx, (uint32_t)ny, (uint32_t)nz)
                 : p;
    const int64_t w = L.wbase[pl] + (int64_t)(q[h] >> 5);
    qw[h] = bits[w];
    qp[h] = pre[w];
  }
  const uint64_t cc = (p << 3) + (uint64_t)(j & 7);  // child j: cell 8p + j of depth l
  const int64_t cwi = L.wbase[l] + (int64_t)(cc >> 5);
  const uint32_t cw = bits[cwi];
  const int32_t cp = pre[cwi];
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const int jj = j + 16 * h;
    if (jj < 27) {  // first-child row of the neighbour, or -1
      const bool on = in[h] && ((qw[h] >> (q[h] & 31)) & 1u);
      const int32_t rq = qp[h] - E.mbase[pl] + __popc(qw[h] & ((1u << (q[h] & 31)) - 1u));
      E.nbr[l][27 * (int64_t)r + jj] = on ? 8 * rq : -1;
    }
  }
  if (j < 8) {  // child j, row 8r + j
    const int32_t rk = cp - E.mbase[l] + __popc(cw & ((1u << (cc & 31)) - 1u));
    const bool on = (cw >> (cc & 31)) & 1u;
    const uint32_t kb = 3u * (uint32_t)l;
    const int64_t row = 8 * (int64_t)r + j;
    E.keys[l][row] = ((uint32_t)(cc >> kb) << 24) | ((uint32_t)cc & (uint32_t)((1ull << kb) - 1ull));
    E.labels[l][row] = on ? rk + 1 : 0;
    if (on) E.rows[l][rk] = (int32_t)row;
    if (l == d) {
      float* o = E.signal + 3 * row;
#pragma unroll
      for (int a = 0; a < 3; ++a) o[a] = on ? leafmean[3 * (int64_t)rk + a] : 0.f;
    }
  }
}

__global__ __launch_bounds__(TB) void k_fill_u32(uint32_t* __restrict__ p, uint32_t v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (i < n) p[i] = v;
}

inline unsigned blocks_for(int64_t n) { return (unsigned)oc::cdiv(n, TB); }

// Bump allocator over one device allocation.
struct Arena {
  char* base = nullptr;
  size_t used = 0;
  template <class T>
  T* take(int64_t n) {
    T* p = reinterpret_cast<T*>(base + used);
    used += oc::align256(sizeof(T) * (size_t)std::max<int64_t>(n, 1));
    return p;
  }
};

struct Scratch {
  uint32_t* bits;
  int32_t* pre;
  int32_t* bsum;
  uint32_t* leafcell;
  uint2* bstat;
  uint32_t* ucell;
  float* leafmean;
  uint32_t* info;  // [0] flags, [1] max |normal|, [2 + l] M_l
};

void carve(Arena& a, int B, int64_t P, int64_t nw, int nb, int64_t ucap, Scratch& s) {
  s.bits = a.take<uint32_t>(nw);
  s.pre = a.take<int32_t>(nw + 1);
  s.bsum = a.take<int32_t>(nb + 1);
  s.leafcell = a.take<uint32_t>(P);
  s.bstat = a.take<uint2>(oc::cdiv(P, TB));
  s.ucell = a.take<uint32_t>(ucap);
  s.leafmean = a.take<float>(3 * P);
  s.info = a.take<uint32_t>(16);
}

}  // namespace

namespace oc {

void fill_u32(void* p, uint32_t v, int64_t n, hipStream_t s) {
  if (n <= 0) return;
  oc::launch(k_fill_u32, dim3(blocks_for(n)), dim3(TB), 0, s, (uint32_t*)p, v, n);
}

}  // namespace oc

namespace {

// Pinned host word block and event for the counts of one build in flight
// (reused across builds; one pool per process, each slot tied to a device).
struct CountSlot {
  uint32_t* host = nullptr;
  hipEvent_t ready = nullptr;
  int device = -1;
};

std::mutex g_slot_mu;
std::vector<CountSlot> g_slots;

bool take_slot(CountSlot* out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  {
    std::lock_guard<std::mutex> lk(g_slot_mu);
    for (size_t k = 0; k < g_slots.size(); ++k)
      if (g_slots[k].device == dev) {
        *out = g_slots[k];
        g_slots.erase(g_slots.begin() + (long)k);
        return true;
      }
  }
  CountSlot c;
  c.device = dev;
  if (hipHostMalloc((void**)&c.host, 16 * sizeof(uint32_t), hipHostMallocDefault) != hipSuccess)
    return false;
  if (hipEventCreateWithFlags(&c.ready, hipEventDisableTiming) != hipSuccess) {
    (void)hipHostFree(c.host);
    return false;
  }
  *out = c;
  return true;
}

void give_slot(const CountSlot& c) {
  std::lock_guard<std::mutex> lk(g_slot_mu);
  g_slots.push_back(c);
}

}  // namespace

// State of a build between oc_build_async and oc_build_finish.
struct oc_build_job {
  Levels L{};
  Shapes S{};
  std::vector<int32_t> offs;
  int B = 0, d = 0, fd = 0, nq = 0;
  int64_t P = 0;
  const float* normals = nullptr;
  oc_allocator A{};
  hipStream_t stream = nullptr;  // of the first half and of the scratch
  char* scratch = nullptr;
  Scratch s{};
  CountSlot slot;
};

namespace {

void drop_job(oc_build_job* j, hipStream_t s) {
  if (j->scratch) oc::dev_free(j->A, j->scratch, s);
  give_slot(j->slot);
  delete j;
}

}  // namespace

extern "C" oc_status oc_build_async(const float* points, const float* normals,
                                    const int32_t* shape_offsets, int32_t batch, int32_t depth,
                                    int32_t full_depth, const oc_allocator* alloc,
                                    hipStream_t stream, oc_build_job** job) {
  using oc::fail;
  if (!job) return fail(OC_ERR_ARG, "oc_build_async: job is NULL");
  *job = nullptr;
  if (!shape_offsets) return fail(OC_ERR_ARG, "oc_build: shape_offsets is NULL");
  if (batch < 1 || batch > 256) return fail(OC_ERR_ARG, "oc_build: batch %d not in 1..256", batch);
  if (depth < 1 || depth > OC_MAX_DEPTH)
    return fail(OC_ERR_ARG, "oc_build: depth %d not in 1..%d", depth, OC_MAX_DEPTH);
  if (full_depth < 0 || full_depth > depth)
    return fail(OC_ERR_ARG, "oc_build: full_depth %d not in 0..depth", full_depth);
  if (shape_offsets[0] != 0) return fail(OC_ERR_ARG, "oc_build: shape_offsets[0] != 0");
  for (int b = 0; b < batch; ++b)
    if (shape_offsets[b + 1] < shape_offsets[b])
      return fail(OC_ERR_ARG, "oc_build: shape_offsets decrease at %d", b);
  const int64_t P = shape_offsets[batch];
  if (P > (int64_t(1) << 28))
    return fail(OC_ERR_UNSUPPORTED, "oc_build: %lld points > 2^28", (long long)P);
  if (P > 0 && (!points || !normals)) return fail(OC_ERR_ARG, "oc_build: points/normals NULL");
  if (((int64_t)batch << (3 * full_depth)) > (int64_t(1) << 28))
    return fail(OC_ERR_UNSUPPORTED, "oc_build: batch * 8^full_depth too large");

  oc_build_job* j = new oc_build_job;
  if (!take_slot(&j->slot)) {
    delete j;
    return fail(OC_ERR_DEVICE, "oc_build: pinned count buffer or event unavailable");
  }
  j->A = alloc ? *alloc : oc_allocator{nullptr, nullptr, nullptr};
  j->B = batch, j->d = depth, j->fd = full_depth, j->P = P;
  j->normals = normals;
  j->stream = stream;
  j->offs.assign(shape_offsets, shape_offsets + batch + 1);
  const int B = batch, d = depth, fd = full_depth;

  Levels& L = j->L;
  L.depth = d, L.full_depth = fd, L.batch = B;
  int64_t ucap = 0;  // bound on the set bits of all depths
  L.wbase[0] = 0;
  for (int l = 0; l <= d; ++l) {
    L.cells[l] = (int64_t)B << (3 * l);
    L.wbase[l + 1] = L.wbase[l] + oc::cdiv(L.cells[l], 32);
    ucap += l < fd ? L.cells[l] : std::min<int64_t>(P, L.cells[l]);
  }
  const int64_t nw = L.wbase[d + 1];
  const int nb = (int)oc::cdiv(nw, SCAN_W);

  Arena meas;
  Scratch& s = j->s;
  carve(meas, B, P, nw, nb, ucap, s);
  Arena ar;
  ar.base = (char*)oc::dev_alloc(j->A, meas.used, stream);
  if (!ar.base) {
    drop_job(j, stream);
    return fail(OC_ERR_NOMEM, "oc_build: scratch allocation of %zu bytes failed", meas.used);
  }
  j->scratch = ar.base;
  carve(ar, B, P, nw, nb, ucap, s);

  Shapes& S = j->S;
  for (int b = 0; b <= B; ++b) S.offs[b] = shape_offsets[b];
  const int nq = (int)oc::cdiv(P, TB);
  j->nq = nq;
  if (P > 0)
    oc::launch(k_quant, dim3(nq), dim3(TB), 0, stream, points, normals, S, B, (int)P, d,
                       s.leafcell, s.bstat);
  const MarkCfg mc = mark_cfg(L.cells[d]);
  oc::launch(k_mark, dim3((unsigned)oc::cdiv(L.cells[d], 32ll * mc.words)), dim3(MK_TB),
                     mc.lds, stream, (const uint32_t*)s.leafcell, S, L, mc.words, mc.up, s.bits);
  for (int l = d - mc.up - 1; l >= fd; --l)
    oc::launch(k_reduce, dim3(blocks_for(L.wbase[l + 1] - L.wbase[l])), dim3(TB), 0,
                       stream, L, l, s.bits);
  oc::launch(k_scan_a, dim3(nb), dim3(TB), 0, stream, (const uint32_t*)s.bits, nw, s.bsum);
  oc::launch(k_scan_c, dim3(nb), dim3(TB), 0, stream, L, (const uint32_t*)s.bits, nw,
                     (const int32_t*)s.bsum, s.pre, s.ucell, (const uint2*)s.bstat, nq, s.info);
  hipError_t he = hipGetLastError();
  if (he == hipSuccess)
    he = hipMemcpyAsync(j->slot.host, s.info, 16 * sizeof(uint32_t), hipMemcpyDeviceToHost,
                        stream);
  if (he == hipSuccess) he = hipEventRecord(j->slot.ready, stream);
  if (he != hipSuccess) {
    (void)hipStreamSynchronize(stream);
    drop_job(j, stream);
    return fail(OC_ERR_DEVICE, "oc_build: %s", hipGetErrorString(he));
  }
  *job = j;
  return OC_OK;
}

extern "C" oc_status oc_build_finish(oc_build_job* j, hipStream_t stream, oc_octree** out) {
  using oc::fail;
  if (out) *out = nullptr;
  if (!j) return fail(OC_ERR_ARG, "oc_build_finish: job is NULL");
  if (!out) {
    oc_build_cancel(j);
    return fail(OC_ERR_ARG, "oc_build_finish: out is NULL");
  }
  const int B = j->B, d = j->d;
  const Levels& L = j->L;
  const Scratch& s = j->s;
  // the one wait: the first half's counts
  hipError_t he = hipEventSynchronize(j->slot.ready);
  if (he == hipSuccess && stream != j->stream) he = hipStreamWaitEvent(stream, j->slot.ready, 0);
  if (he != hipSuccess) {
    drop_job(j, j->stream);
    return fail(OC_ERR_DEVICE, "oc_build: %s", hipGetErrorString(he));
  }
  uint32_t info[16];
  std::memcpy(info, j->slot.host, sizeof(info));
  if (info[0] & 1u) {
    drop_job(j, stream);
    return fail(OC_ERR_RANGE, "oc_build: a point is outside [0,1]^3 or NaN");
  }
  if (info[0] & 2u) {
    drop_job(j, stream);
    return fail(OC_ERR_RANGE, "oc_build: a normal is not finite");
  }

  oc_octree* t = new oc_octree;
  t->depth = d;
  t->full_depth = j->fd;
  t->batch = B;
  t->alloc = j->A;
  t->stream = stream;
  for (int l = 0; l <= d; ++l) {
    t->M[l] = info[3 + l] - info[2 + l];
    t->N[l] = l == 0 ? B : 8 * t->M[l - 1];
    if (t->N[l] > INT32_MAX / 2) {
      drop_job(j, stream);
      delete t;
      return fail(OC_ERR_UNSUPPORTED, "oc_build: depth %d has too many octants", l);
    }
  }
  size_t bytes = 0;
  for (int l = 0; l <= d; ++l) {
    bytes += oc::align256(4 * (size_t)t->N[l]) * 2 + oc::align256(4 * (size_t)t->M[l]);
    if (l > 0) bytes += oc::align256(4 * 27 * (size_t)t->M[l - 1]);
  }
  bytes += oc::align256(12 * (size_t)t->N[d]);
  char* blk = (char*)oc::dev_alloc(j->A, bytes, stream);
  if (!blk) {
    drop_job(j, stream);
    delete t;
    return fail(OC_ERR_NOMEM, "oc_build: octree allocation of %zu bytes failed", bytes);
  }
  t->block = blk;
  size_t off = 0;
  auto take = [&](size_t b) {
    char* p = blk + off;
    off += oc::align256(b);
    return b ? (void*)p : nullptr;
  };
  for (int l = 0; l <= d; ++l) {
    t->keys[l] = (uint32_t*)take(4 * (size_t)t->N[l]);
    t->labels[l] = (int32_t*)take(4 * (size_t)t->N[l]);
    t->rows[l] = (int32_t*)take(4 * (size_t)t->M[l]);
    t->nbr[l] = l > 0 ? (int32_t*)take(4 * 27 * (size_t)t->M[l - 1]) : nullptr;
  }
  t->signal = (float*)take(12 * (size_t)t->N[d]);

  // leaf signal (needs only device data of the first half), then emission
  if (j->P > 0) {
    int64_t kmax = 1;  // leaf chunks of the largest shape
    for (int b = 0; b < B; ++b)
      kmax = std::max<int64_t>(
          kmax, oc::cdiv(std::min<int64_t>(j->offs[b + 1] - j->offs[b], L.cells[d] / B),
                         LM_LEAVES));
    oc::launch(k_leaf_mean, dim3((unsigned)B, (unsigned)kmax), dim3(LM_TB), 0, stream,
                       j->normals, (const uint32_t*)s.leafcell, j->S, (int)j->P, L,
                       (const uint32_t*)s.bits, (const int32_t*)s.pre, (const uint32_t*)s.ucell,
                       (const uint32_t*)s.info, s.leafmean);
  }
  Emit E{};
  int32_t m = 0;
  for (int l = 0; l <= d + 1; ++l) {
    E.mbase[l] = m;
    if (l <= d) m += (int32_t)t->M[l];
  }
  E.ibase[0] = 0;
  E.ibase[1] = B;
  for (int l = 1; l <= d; ++l) E.ibase[l + 1] = E.ibase[l] + t->M[l - 1];
  for (int l = 0; l <= d; ++l) {
    E.keys[l] = t->keys[l];
    E.labels[l] = t->labels[l];
    E.rows[l] = t->rows[l];
    E.nbr[l] = t->nbr[l];
  }
  E.signal = t->signal;
  oc::launch(k_emit, dim3(blocks_for(16 * E.ibase[d + 1])), dim3(TB), 0, stream, L, E,
                     (const uint32_t*)s.bits, (const int32_t*)s.pre, (const uint32_t*)s.ucell,
                     (const float*)s.leafmean);
  he = hipGetLastError();
  drop_job(j, stream);  // the scratch is released in stream order after the emission
  if (he != hipSuccess) {
    oc_octree_free(t);
    return fail(OC_ERR_DEVICE, "oc_build: launch failed: %s", hipGetErrorString(he));
  }
  *out = t;
  return OC_OK;
}

extern "C" void oc_build_cancel(oc_build_job* j) {
  if (!j) return;
  (void)hipEventSynchronize(j->slot.ready);
  drop_job(j, j->stream);
}

extern "C" oc_status oc_build(const float* points, const float* normals,
                              const int32_t* shape_offsets, int32_t batch, int32_t depth,
                              int32_t full_depth, const oc_allocator* alloc, hipStream_t stream,
                              oc_octree** out) {
  if (!out) return oc::fail(OC_ERR_ARG, "oc_build: out is NULL");
  *out = nullptr;
  oc_build_job* j = nullptr;
  const oc_status st =
      oc_build_async(points, normals, shape_offsets, batch, depth, full_depth, alloc, stream, &j);
  if (st != OC_OK) return st;
  return oc_build_finish(j, stream, out);
}
