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
//    k_mark: workgroup k owns leaf cells [k MK_CELLS, (k+1) MK_CELLS) as an LDS
//    bitmap, scans the points of the shapes that overlap it, derives the words
//    of up to MK_UP coarser depths from it (bit j of depth l = byte j of depth
//    l+1 != 0) and stores all of them; the workgroups also fill the depths
//    shallower than full_depth with ones.  No global atomics.

__global__ __launch_bounds__(TB) void k_quant(const float* __restrict__ pts,
                                              const float* __restrict__ nrm, Shapes S, int B,
                                              int P, int d, uint32_t* __restrict__ leafcell,
                                              uint2* __restrict__ bstat) {
  const int i0 = blockIdx.x * TB + threadIdx.x;
  const bool live = i0 < P;
  const int i = live ? i0 : P - 1;  // the block reductions need every lane
  int lo = 0, hi = B - 1;  // last shape b with offs[b] <= i
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (S.offs[mid] <= i) lo = mid;
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
constexpr int MK_WORDS = 16384;                // 64 KB of LDS for the leaf depth
constexpr int64_t MK_CELLS = 32ll * MK_WORDS;  // leaf cells per workgroup
constexpr int MK_UP = 4;                       // coarser depths derived in LDS

__global__ __launch_bounds__(MK_TB) void k_mark(const uint32_t* __restrict__ leafcell, Shapes S,
                                                Levels L, uint32_t* __restrict__ bits) {
  __shared__ uint32_t w[MK_WORDS + MK_WORDS / 8 + MK_WORDS / 64 + MK_WORDS / 512 + MK_WORDS / 4096];
  const int d = L.depth;
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
  for (int i = S.offs[b0] + threadIdx.x; i < S.offs[b1 + 1]; i += MK_TB) {
    const uint32_t c = leafcell[i];
    if (c == 0xFFFFFFFFu || (int64_t)c < c0 || (int64_t)c >= c1) continue;
    atomicOr(&w[(c - c0) >> 5], 1u << (c & 31));
  }
  __syncthreads();
  if (d >= L.full_depth) {
    uint32_t* dst = bits + L.wbase[d] + (c0 >> 5);
    for (int k = threadIdx.x; k < nwd; k += MK_TB) dst[k] = w[k];
  }
  // coarser depths d-1 .. d-MK_UP: the chunk's cells there start on a word
  // boundary (MK_CELLS / 8^MK_UP is a multiple of 32)
  uint32_t* fine = w;
  int nfine = nwd;
  int off = MK_WORDS;
  for (int j = 1; j <= MK_UP && d - j >= L.full_depth; ++j) {
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
    off += MK_WORDS >> (3 * j);
  }
}

// ---------------------------------------------------------------------------
// 2. depths more than MK_UP above the leaves (and not forced): bit j of depth
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
//    before word w; pre[nw] = total.  Blocks of SCAN_W words.

constexpr int SCAN_PER = 8;
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

// One block: exclusive scan of nb block sums in place; grand total at bsum[nb].
__global__ __launch_bounds__(TB) void k_scan_b(int32_t* __restrict__ bsum, int nb) {
  const int per = (nb + TB - 1) / TB;
  const int b0 = threadIdx.x * per;
  int32_t s = 0;
  for (int k = 0; k < per; ++k)
    if (b0 + k < nb) s += bsum[b0 + k];
  int32_t total;
  int32_t run = block_excl_scan(s, &total);
  for (int k = 0; k < per; ++k)
    if (b0 + k < nb) {
      const int32_t v = bsum[b0 + k];
      bsum[b0 + k] = run;
      run += v;
    }
  if (threadIdx.x == 0) bsum[nb] = total;
}

__global__ __launch_bounds__(TB) void k_scan_c(const uint32_t* __restrict__ bits, int64_t nw,
                                               const int32_t* __restrict__ bsum,
                                               int32_t* __restrict__ pre, int nb) {
  const int64_t w0 = (int64_t)blockIdx.x * SCAN_W + threadIdx.x * SCAN_PER;
  int32_t c[SCAN_PER], s = 0;
#pragma unroll
  for (int k = 0; k < SCAN_PER; ++k) {
    c[k] = w0 + k < nw ? __popc(bits[w0 + k]) : 0;
    s += c[k];
  }
  int32_t total;
  int32_t run = bsum[blockIdx.x] + block_excl_scan(s, &total);
#pragma unroll
  for (int k = 0; k < SCAN_PER; ++k)
    if (w0 + k < nw) {
      pre[w0 + k] = run;
      run += c[k];
    }
  if (blockIdx.x == 0 && threadIdx.x == 0) pre[nw] = bsum[nb];
}

// ---------------------------------------------------------------------------
// 4. cell of every set bit, in rank order over all depths: ucell[pre + k].
//    Workgroup 0 also reports the per-depth counts M_l (info[2 + l]) and the
//    flags and largest |normal component| of the nq blocks of k_quant
//    (info[0], info[1]).

__global__ __launch_bounds__(TB) void k_compact(Levels L, const uint32_t* __restrict__ bits,
                                                const int32_t* __restrict__ pre,
                                                uint32_t* __restrict__ ucell,
                                                const uint2* __restrict__ bstat, int nq,
                                                uint32_t* __restrict__ info) {
  const int64_t w = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (w < L.wbase[L.depth + 1]) {
    uint32_t v = bits[w];
    if (v) {
      const int l = level_of_word(L, w);
      const uint32_t base = (uint32_t)((w - L.wbase[l]) * 32);
      int32_t r = pre[w];
      while (v) {
        const int b = __ffs(v) - 1;
        ucell[r++] = base + (uint32_t)b;
        v &= v - 1u;
      }
    }
  }
  if (blockIdx.x != 0) return;
  __shared__ uint2 ws[TB / 64];
  const int t = threadIdx.x;
  if (t <= L.depth) info[2 + t] = (uint32_t)(pre[L.wbase[t + 1]] - pre[L.wbase[t]]);
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
//    additions make the result independent of their order.

constexpr int LM_TB = 1024;
constexpr int LM_LEAVES = 3072;  // 3072 * (3 * 8 + 4) bytes of LDS

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
  __shared__ unsigned long long sum[3 * LM_LEAVES];
  __shared__ int32_t cnt[LM_LEAVES];
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
  for (int i = S.offs[b] + threadIdx.x; i < S.offs[b + 1]; i += LM_TB) {
    const uint32_t c = leafcell[i];
    if (c < clo || (uint64_t)c >= chi) continue;
    const int32_t j = rank_in(bits, pre, L, d, mb, c, &word) - lo;
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      const long long v = llrint(ldexp((double)nrm[3 * (int64_t)i + a], s));
      atomicAdd(&sum[3 * j + a], (unsigned long long)v);
    }
    atomicAdd(&cnt[j], 1);
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
  // 32 lanes per item: lane j < 8 emits child j, lane j < 27 neighbour j
  const int64_t it = ((int64_t)blockIdx.x * TB + threadIdx.x) >> 5;
  const int j = threadIdx.x & 31;
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

  if (j < 8) {  // child j: cell 8p + j of depth l, row 8r + j
    const uint64_t cc = (p << 3) + (uint64_t)j;
    const int32_t rk = rank_in(bits, pre, L, l, E.mbase[l], cc, &word);
    const bool on = (word >> (cc & 31)) & 1u;
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
  if (j < 27) {  // neighbour j of the parent at depth l-1: first-child row or -1
    const uint32_t pkb = 3u * (uint32_t)pl;
    const uint32_t pshape = (uint32_t)(p >> pkb);
    const uint32_t pkey = (uint32_t)p & (uint32_t)((1ull << pkb) - 1ull);
    const int side = 1 << pl;
    const int nx = (int)squeeze3(pkey >> 2) + j / 9 - 1;
    const int ny = (int)squeeze3(pkey >> 1) + (j / 3) % 3 - 1;
    const int nz = (int)squeeze3(pkey) + j % 3 - 1;
    int32_t v = -1;
    if (nx >= 0 && nx < side && ny >= 0 && ny < side && nz >= 0 && nz < side) {
      const uint64_t q = ((uint64_t)pshape << pkb) |
                         shuffle_key((uint32_t)nx, (uint32_t)ny, (uint32_t)nz);
      const int32_t rq = rank_in(bits, pre, L, pl, E.mbase[pl], q, &word);
      v = ((word >> (q & 31)) & 1u) ? 8 * rq : -1;
    }
    E.nbr[l][27 * (int64_t)r + j] = v;
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
  hipLaunchKernelGGL(k_fill_u32, dim3(blocks_for(n)), dim3(TB), 0, s, (uint32_t*)p, v, n);
}

}  // namespace oc

extern "C" oc_status oc_build(const float* points, const float* normals,
                              const int32_t* shape_offsets, int32_t batch, int32_t depth,
                              int32_t full_depth, const oc_allocator* alloc, hipStream_t stream,
                              oc_octree** out) {
  using oc::fail;
  if (!out) return fail(OC_ERR_ARG, "oc_build: out is NULL");
  *out = nullptr;
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

  const oc_allocator A = alloc ? *alloc : oc_allocator{nullptr, nullptr, nullptr};
  const int B = batch, d = depth, fd = full_depth;

  Levels L{};
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
  Scratch s{};
  carve(meas, B, P, nw, nb, ucap, s);
  Arena ar;
  ar.base = (char*)oc::dev_alloc(A, meas.used, stream);
  if (!ar.base) return fail(OC_ERR_NOMEM, "oc_build: scratch allocation of %zu bytes failed", meas.used);
  carve(ar, B, P, nw, nb, ucap, s);
  auto release = [&](void* p) { oc::dev_free(A, p, stream); };

  Shapes S;
  for (int b = 0; b <= B; ++b) S.offs[b] = shape_offsets[b];
  const int nq = (int)oc::cdiv(P, TB);
  if (P > 0)
    hipLaunchKernelGGL(k_quant, dim3(nq), dim3(TB), 0, stream, points, normals, S, B, (int)P, d,
                       s.leafcell, s.bstat);
  hipLaunchKernelGGL(k_mark, dim3((unsigned)oc::cdiv(L.cells[d], MK_CELLS)), dim3(MK_TB), 0,
                     stream, (const uint32_t*)s.leafcell, S, L, s.bits);
  for (int l = d - MK_UP - 1; l >= fd; --l)
    hipLaunchKernelGGL(k_reduce, dim3(blocks_for(L.wbase[l + 1] - L.wbase[l])), dim3(TB), 0,
                       stream, L, l, s.bits);
  hipLaunchKernelGGL(k_scan_a, dim3(nb), dim3(TB), 0, stream, (const uint32_t*)s.bits, nw, s.bsum);
  hipLaunchKernelGGL(k_scan_b, dim3(1), dim3(TB), 0, stream, s.bsum, nb);
  hipLaunchKernelGGL(k_scan_c, dim3(nb), dim3(TB), 0, stream, (const uint32_t*)s.bits, nw,
                     (const int32_t*)s.bsum, s.pre, nb);
  hipLaunchKernelGGL(k_compact, dim3(blocks_for(nw)), dim3(TB), 0, stream, L,
                     (const uint32_t*)s.bits, (const int32_t*)s.pre, s.ucell,
                     (const uint2*)s.bstat, nq, s.info);
  if (P > 0) {
    int64_t kmax = 1;  // leaf chunks of the largest shape
    for (int b = 0; b < B; ++b)
      kmax = std::max<int64_t>(
          kmax, oc::cdiv(std::min<int64_t>(shape_offsets[b + 1] - shape_offsets[b], L.cells[d] / B),
                         LM_LEAVES));
    hipLaunchKernelGGL(k_leaf_mean, dim3((unsigned)B, (unsigned)kmax), dim3(LM_TB), 0, stream,
                       normals, (const uint32_t*)s.leafcell, S, (int)P, L,
                       (const uint32_t*)s.bits, (const int32_t*)s.pre, (const uint32_t*)s.ucell,
                       (const uint32_t*)s.info, s.leafmean);
  }

  uint32_t info[16] = {};
  hipError_t he = hipGetLastError();
  if (he == hipSuccess)
    he = hipMemcpyAsync(info, s.info, sizeof(info), hipMemcpyDeviceToHost, stream);
  if (he == hipSuccess) he = hipStreamSynchronize(stream);
  if (he != hipSuccess) {
    release(ar.base);
    return fail(OC_ERR_DEVICE, "oc_build: %s", hipGetErrorString(he));
  }
  if (info[0] & 1u) {
    release(ar.base);
    return fail(OC_ERR_RANGE, "oc_build: a point is outside [0,1]^3 or NaN");
  }
  if (info[0] & 2u) {
    release(ar.base);
    return fail(OC_ERR_RANGE, "oc_build: a normal is not finite");
  }

  oc_octree* t = new oc_octree;
  t->depth = d;
  t->full_depth = fd;
  t->batch = B;
  t->alloc = A;
  t->stream = stream;
  for (int l = 0; l <= d; ++l) {
    t->M[l] = info[2 + l];
    t->N[l] = l == 0 ? B : 8 * t->M[l - 1];
    if (t->N[l] > INT32_MAX / 2) {
      release(ar.base);
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
  char* blk = (char*)oc::dev_alloc(A, bytes, stream);
  if (!blk) {
    release(ar.base);
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
  hipLaunchKernelGGL(k_emit, dim3(blocks_for(32 * E.ibase[d + 1])), dim3(TB), 0, stream, L, E,
                     (const uint32_t*)s.bits, (const int32_t*)s.pre, (const uint32_t*)s.ucell,
                     (const float*)s.leafmean);
  he = hipGetLastError();
  release(ar.base);
  if (he != hipSuccess) {
    oc_octree_free(t);
    return fail(OC_ERR_DEVICE, "oc_build: launch failed: %s", hipGetErrorString(he));
  }
  *out = t;
  return OC_OK;
}
