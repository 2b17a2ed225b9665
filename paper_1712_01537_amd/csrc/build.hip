// Octree construction on the GPU (Sec. 3.1 of O-CNN, arXiv 1712.01537).
//
// The paper builds octrees offline on the CPU by breadth-first subdivision.
// Here the same structure is produced bottom-up with data-parallel passes:
//   1. quantise every point at the leaf depth and form its compact key
//      (shape index above the 3d shuffle-key bits);
//   2. LSD radix sort of the compact keys (8-bit digits, stable ranks from
//      wavefront ballots);
//   3. adjacent-unique of the sorted keys gives the non-empty leaves; the
//      points of a leaf are contiguous, so the mean normal is a segmented sum;
//   4. parent keys are key >> 3, already sorted, so each shallower depth is
//      another adjacent-unique (ballot/popcount scan), down to full_depth,
//      below which every octant is forced non-empty (Sec. 4);
//   5. after the single host read of the per-depth counts, every depth's
//      keys, labels and label->row map are emitted top-down: the children of
//      the j-th non-empty octant occupy rows 8j..8j+7 (Sec. 3.1 "Label");
//   6. a hash table per depth maps a non-empty octant's key to its rank
//      (Sec. 3.2, H: key -> index), and for every sibling group the 27
//      parent-level neighbours are looked up once: the (K+1)^3 union
//      neighbourhood of the eight siblings (Sec. 3.2, Fig. 4) is then a fixed
//      function of those 27 entries.
#include <algorithm>
#include <cstring>
#include <vector>

#include "common.h"

namespace {

constexpr int TB = 256;  // threads per block in every kernel of this file
constexpr int WAVE = 64;

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

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & (WAVE - 1);
  return lane == 0 ? 0ull : (~0ull >> (WAVE - lane));
}

// ---------------------------------------------------------------------------
// 1. quantise + compact key

__global__ __launch_bounds__(TB) void k_quant_key(const float* __restrict__ pts,
                                                  const int32_t* __restrict__ offs, int B, int P,
                                                  int depth, uint32_t* __restrict__ key,
                                                  int32_t* __restrict__ idx, int* __restrict__ err) {
  const int i = blockIdx.x * TB + threadIdx.x;
  if (i >= P) return;
  int lo = 0, hi = B - 1;  // last shape b with offs[b] <= i
  while (lo < hi) {
    int mid = (lo + hi + 1) >> 1;
    if (offs[mid] <= i) lo = mid;
    else hi = mid - 1;
  }
  const float scale = (float)(1u << depth);  // exact power of two
  const uint32_t qmax = (1u << depth) - 1u;
  uint32_t q[3];
  bool bad = false;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    float p = pts[3 * i + a];
    bool ok = p >= 0.0f && p <= 1.0f;  // false for NaN
    bad |= !ok;
    uint32_t c = ok ? (uint32_t)floorf(p * scale) : 0u;
    q[a] = c > qmax ? qmax : c;
  }
  if (bad) atomicOr(err, 1);
  key[i] = ((uint32_t)lo << (3 * depth)) | shuffle_key(q[0], q[1], q[2]);
  idx[i] = i;
}

// ---------------------------------------------------------------------------
// 2. LSD radix sort of (key, index) pairs, 8-bit digits.

constexpr int RS_ITEMS = 32;
constexpr int RS_TILE = TB * RS_ITEMS;

// Per-tile digit histogram, stored digit-major: hist[d * nblk + tile].
__global__ __launch_bounds__(TB) void k_radix_hist(const uint32_t* __restrict__ keys, int n,
                                                   int shift, uint32_t* __restrict__ hist,
                                                   int nblk) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int base = blockIdx.x * RS_TILE;
  for (int j = 0; j < RS_ITEMS; ++j) {
    int i = base + j * TB + threadIdx.x;
    if (i < n) atomicAdd(&h[(keys[i] >> shift) & 255u], 1u);
  }
  __syncthreads();
  hist[threadIdx.x * nblk + blockIdx.x] = h[threadIdx.x];
}

// Exclusive scan of the digit-major histogram (one block, thread = digit).
__global__ __launch_bounds__(TB) void k_radix_scan(uint32_t* __restrict__ hist, int nblk) {
  __shared__ uint32_t s[256];
  const int d = threadIdx.x;
  uint32_t tot = 0;
  for (int b = 0; b < nblk; ++b) tot += hist[d * nblk + b];
  s[d] = tot;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {  // Hillis-Steele inclusive scan
    uint32_t v = d >= off ? s[d - off] : 0u;
    __syncthreads();
    s[d] += v;
    __syncthreads();
  }
  uint32_t run = s[d] - tot;
  for (int b = 0; b < nblk; ++b) {
    uint32_t v = hist[d * nblk + b];
    hist[d * nblk + b] = run;
    run += v;
  }
}

// Stable scatter.  The tile is walked in slices of TB consecutive elements;
// within a slice, lanes holding the same digit are found with 8 ballots, and
// per-wave digit counts in LDS order the waves.
__global__ __launch_bounds__(TB) void k_radix_scatter(const uint32_t* __restrict__ kin,
                                                      const int32_t* __restrict__ vin,
                                                      uint32_t* __restrict__ kout,
                                                      int32_t* __restrict__ vout, int n, int shift,
                                                      const uint32_t* __restrict__ offs, int nblk) {
  __shared__ uint32_t base[256];
  __shared__ uint32_t run[256];
  __shared__ uint32_t wcnt[TB / WAVE][256];
  const int tid = threadIdx.x, wave = tid / WAVE, lane = tid % WAVE;
  base[tid] = offs[tid * nblk + blockIdx.x];
  run[tid] = 0;
  const uint64_t lt = lanemask_lt();
  for (int j = 0; j < RS_ITEMS; ++j) {
    const int i = blockIdx.x * RS_TILE + j * TB + tid;
    const bool valid = i < n;
    const uint32_t key = valid ? kin[i] : 0u;
    const int32_t val = valid ? vin[i] : 0;
    const uint32_t d = (key >> shift) & 255u;
#pragma unroll
    for (int w = 0; w < TB / WAVE; ++w) wcnt[w][tid] = 0;
    __syncthreads();
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t m = __ballot(bit);
      peers &= bit ? m : ~m;
    }
    const uint32_t rank = __popcll(peers & lt);
    if (valid && rank == 0) wcnt[wave][d] = __popcll(peers);
    __syncthreads();
    if (valid) {
      uint32_t pos = base[d] + run[d] + rank;
      for (int w = 0; w < wave; ++w) pos += wcnt[w][d];
      kout[pos] = key;
      vout[pos] = val;
    }
    __syncthreads();
    uint32_t add = 0;
#pragma unroll
    for (int w = 0; w < TB / WAVE; ++w) add += wcnt[w][tid];
    run[tid] += add;
  }
}

// ---------------------------------------------------------------------------
// 3./4. adjacent-unique of a sorted key array, keys compared after >> shift.
//   pass 1: per-tile count of run starts;  pass 2: scan of the tile counts
//   (one block), total -> *count;  pass 3: unique keys, the run index of every
//   element (optional) and the first element of every run (optional).
// The input length may live on the device (n_dev) so that these passes can
// be enqueued before any host read; grids are sized for an upper bound.

constexpr int UQ_ITEMS = 8;
constexpr int UQ_TILE = TB * UQ_ITEMS;

__device__ __forceinline__ bool run_start(const uint32_t* keys, int i, int shift) {
  return i == 0 || (keys[i] >> shift) != (keys[i - 1] >> shift);
}

__device__ __forceinline__ int load_n(const int* n_dev, int n_host) {
  return n_dev ? *n_dev : n_host;
}

__global__ __launch_bounds__(TB) void k_unique_count(const uint32_t* __restrict__ keys,
                                                     const int* n_dev, int n_host, int shift,
                                                     uint32_t* __restrict__ tile_cnt) {
  __shared__ uint32_t part[TB / WAVE];
  const int n = load_n(n_dev, n_host);
  uint32_t c = 0;
  for (int j = 0; j < UQ_ITEMS; ++j) {
    int i = blockIdx.x * UQ_TILE + j * TB + threadIdx.x;
    if (i < n && run_start(keys, i, shift)) ++c;
  }
  // wave reduction, then across waves
  for (int off = WAVE / 2; off > 0; off >>= 1) c += __shfl_down(c, off, WAVE);
  if ((threadIdx.x & (WAVE - 1)) == 0) part[threadIdx.x / WAVE] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t s = 0;
    for (int w = 0; w < TB / WAVE; ++w) s += part[w];
    tile_cnt[blockIdx.x] = s;
  }
}

// Exclusive scan of ntile counts in one block; total to *count.
__global__ __launch_bounds__(TB) void k_scan_tiles(uint32_t* __restrict__ tile_cnt, int ntile,
                                                   int* __restrict__ count) {
  __shared__ uint32_t s[TB];
  const int t = threadIdx.x;
  const int per = (ntile + TB - 1) / TB;  // contiguous chunk per thread
  uint32_t tot = 0;
  for (int k = 0; k < per; ++k) {
    int i = t * per + k;
    if (i < ntile) tot += tile_cnt[i];
  }
  s[t] = tot;
  __syncthreads();
  for (int off = 1; off < TB; off <<= 1) {
    uint32_t v = t >= off ? s[t - off] : 0u;
    __syncthreads();
    s[t] += v;
    __syncthreads();
  }
  uint32_t run = s[t] - tot;
  for (int k = 0; k < per; ++k) {
    int i = t * per + k;
    if (i < ntile) {
      uint32_t v = tile_cnt[i];
      tile_cnt[i] = run;
      run += v;
    }
  }
  if (t == TB - 1) *count = (int)s[TB - 1];
}

__global__ __launch_bounds__(TB) void k_unique_write(const uint32_t* __restrict__ keys,
                                                     const int* n_dev, int n_host, int shift,
                                                     const uint32_t* __restrict__ tile_off,
                                                     uint32_t* __restrict__ uniq,
                                                     int32_t* __restrict__ run_of,
                                                     int32_t* __restrict__ first) {
  __shared__ uint32_t wsum[TB / WAVE];
  const int n = load_n(n_dev, n_host);
  const int tid = threadIdx.x, wave = tid / WAVE;
  const uint64_t lt = lanemask_lt();
  uint32_t off = tile_off[blockIdx.x];
  if (blockIdx.x * UQ_TILE >= n) return;
  for (int j = 0; j < UQ_ITEMS; ++j) {
    const int i = blockIdx.x * UQ_TILE + j * TB + tid;
    const bool f = i < n && run_start(keys, i, shift);
    const uint64_t m = __ballot(f);
    if ((tid & (WAVE - 1)) == 0) wsum[wave] = __popcll(m);
    __syncthreads();
    uint32_t before = off, slice = 0;
    for (int w = 0; w < TB / WAVE; ++w) {
      if (w < wave) before += wsum[w];
      slice += wsum[w];
    }
    // inclusive count of run starts up to and including element i
    const uint32_t incl = before + __popcll(m & lt) + (f ? 1u : 0u);
    if (i < n) {
      const uint32_t r = incl - 1u;
      if (f) {
        uniq[r] = keys[i] >> shift;
        if (first) first[r] = i;
      }
      if (run_of) run_of[i] = (int32_t)r;
    }
    off += slice;
    __syncthreads();
  }
}

// Complete depth (shallower than full_depth): every octant non-empty; the
// compact key of the r-th octant is r.
__global__ __launch_bounds__(TB) void k_iota(uint32_t* __restrict__ u, int n) {
  int i = blockIdx.x * TB + threadIdx.x;
  if (i < n) u[i] = (uint32_t)i;
}

// ---------------------------------------------------------------------------
// 5. top-down emission of keys / labels / label->row map.

// Keys of depth l: row t is child (t & 7) of the (t >> 3)-th non-empty octant
// of depth l-1.  Labels are zeroed here and set by k_emit_labels.
__global__ __launch_bounds__(TB) void k_emit_keys(const uint32_t* __restrict__ uparent, int n, int l,
                                                  uint32_t* __restrict__ keys,
                                                  int32_t* __restrict__ labels) {
  const int t = blockIdx.x * TB + threadIdx.x;
  if (t >= n) return;
  uint32_t sk;
  if (l == 0) {
    sk = (uint32_t)t << 24;
  } else {
    const uint32_t ck = (uparent[t >> 3] << 3) | (uint32_t)(t & 7);
    const uint32_t kb = 3u * (uint32_t)l;
    sk = ((ck >> kb) << 24) | (ck & ((1u << kb) - 1u));
  }
  keys[t] = sk;
  labels[t] = 0;
}

// Non-empty octant r of depth l sits at row 8 parent(r) + (key & 7).
// parent_complete: depth l-1 is complete, so parent(r) = key >> 3.
__global__ __launch_bounds__(TB) void k_emit_labels(const uint32_t* __restrict__ u,
                                                    const int32_t* __restrict__ parent_of, int m,
                                                    int l, int parent_complete,
                                                    int32_t* __restrict__ labels,
                                                    int32_t* __restrict__ rows) {
  const int r = blockIdx.x * TB + threadIdx.x;
  if (r >= m) return;
  const uint32_t ck = u[r];
  int32_t row;
  if (l == 0) row = (int32_t)ck;  // the shape index
  else {
    const int32_t p = parent_complete ? (int32_t)(ck >> 3) : parent_of[r];
    row = 8 * p + (int32_t)(ck & 7u);
  }
  labels[row] = r + 1;
  rows[r] = row;
}

// Mean normal of leaf r (points first[r] .. first[r+1]-1 of the sorted order),
// accumulated in double, written to its row of the signal.
__global__ __launch_bounds__(TB) void k_leaf_mean(const int32_t* __restrict__ first, int m, int P,
                                                  const int32_t* __restrict__ perm,
                                                  const float* __restrict__ normals,
                                                  const int32_t* __restrict__ rows,
                                                  float* __restrict__ signal) {
  const int r = blockIdx.x * TB + threadIdx.x;
  if (r >= m) return;
  const int s = first[r], e = r + 1 < m ? first[r + 1] : P;
  double a = 0.0, b = 0.0, c = 0.0;
  for (int i = s; i < e; ++i) {
    const int p = perm[i];
    a += (double)normals[3 * p];
    b += (double)normals[3 * p + 1];
    c += (double)normals[3 * p + 2];
  }
  const double inv = (double)(e - s);
  float* o = signal + 3 * (int64_t)rows[r];
  o[0] = (float)(a / inv);
  o[1] = (float)(b / inv);
  o[2] = (float)(c / inv);
}

// ---------------------------------------------------------------------------
// 6. hash of non-empty keys -> rank, and the 27-entry sibling-group table.

constexpr uint64_t HASH_EMPTY = ~0ull;

__device__ __forceinline__ uint32_t hash_slot(uint32_t ck, uint32_t mask_bits) {
  return (ck * 0x9E3779B1u) >> (32u - mask_bits);  // Fibonacci hashing
}

__global__ __launch_bounds__(TB) void k_hash_insert(const uint32_t* __restrict__ u, int m,
                                                    unsigned long long* __restrict__ table,
                                                    int log_cap) {
  const int r = blockIdx.x * TB + threadIdx.x;
  if (r >= m) return;
  const uint32_t ck = u[r];
  const uint32_t mask = (1u << log_cap) - 1u;
  const unsigned long long entry = ((unsigned long long)(uint32_t)r << 32) | ck;
  uint32_t s = hash_slot(ck, log_cap);
  for (uint32_t probe = 0; probe <= mask; ++probe, s = (s + 1) & mask) {
    unsigned long long prev = atomicCAS(&table[s], (unsigned long long)HASH_EMPTY, entry);
    if (prev == HASH_EMPTY) return;
  }
}

__device__ __forceinline__ int32_t hash_find(const unsigned long long* table, uint32_t ck,
                                             int log_cap) {
  const uint32_t mask = (1u << log_cap) - 1u;
  uint32_t s = hash_slot(ck, log_cap);
  for (uint32_t probe = 0; probe <= mask; ++probe, s = (s + 1) & mask) {
    const unsigned long long e = table[s];
    if (e == HASH_EMPTY) return -1;
    if ((uint32_t)e == ck) return (int32_t)(e >> 32);
  }
  return -1;
}

// nbr[g][o]: first-child row 8 rank of the depth-(l-1) octant at parent
// offset o from group g's parent, -1 if outside the cube or not non-empty.
__global__ __launch_bounds__(TB) void k_nbr(const uint32_t* __restrict__ uparent, int m, int l,
                                            const unsigned long long* __restrict__ table,
                                            int log_cap, int32_t* __restrict__ nbr) {
  const int t = blockIdx.x * TB + threadIdx.x;
  if (t >= 27 * m) return;
  const int g = t / 27, o = t - 27 * g;
  const int pl = l - 1;
  const uint32_t ck = uparent[g];
  const uint32_t kb = 3u * (uint32_t)pl;
  const uint32_t b = ck >> kb, key = ck & ((1u << kb) - 1u);
  const int side = 1 << pl;
  const int x = (int)squeeze3(key >> 2) + (o / 9 - 1);
  const int y = (int)squeeze3(key >> 1) + ((o / 3) % 3 - 1);
  const int z = (int)squeeze3(key) + (o % 3 - 1);
  int32_t v = -1;
  if (x >= 0 && x < side && y >= 0 && y < side && z >= 0 && z < side) {
    const uint32_t nk = (b << kb) | shuffle_key((uint32_t)x, (uint32_t)y, (uint32_t)z);
    const int32_t r = hash_find(table, nk, log_cap);
    v = r >= 0 ? 8 * r : -1;
  }
  nbr[t] = v;
}

__global__ __launch_bounds__(TB) void k_fill_u32(uint32_t* __restrict__ p, uint32_t v, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (i < n) p[i] = v;
}

inline int blocks_for(int64_t n) { return (int)oc::cdiv(n, TB); }

// Scratch bump allocator over one device allocation.
struct Arena {
  char* base = nullptr;
  size_t used = 0, cap = 0;
  template <class T>
  T* take(int64_t n) {
    T* p = reinterpret_cast<T*>(base + used);
    used += oc::align256(sizeof(T) * (size_t)std::max<int64_t>(n, 1));
    return p;
  }
};

}  // namespace

namespace oc {

void fill_u32(void* p, uint32_t v, int64_t n, hipStream_t s) {
  if (n <= 0) return;
  hipLaunchKernelGGL(k_fill_u32, dim3(blocks_for(n)), dim3(TB), 0, s, (uint32_t*)p, v, n);
}

}  // namespace oc

// ---------------------------------------------------------------------------
// Host orchestration.

namespace {

struct Scratch {
  uint32_t *k0, *k1;
  int32_t *v0, *v1;
  uint32_t* hist;
  int32_t* offs;
  uint32_t* tiles;
  int* counts;  // [l] = M_l for l >= full_depth, [OC_MAX_DEPTH + 1] = range error flag
  uint32_t* U[OC_MAX_DEPTH + 1];  // compact keys of the non-empty octants of depth l
  int32_t* J[OC_MAX_DEPTH + 1];   // J[l][r]: index in U[l-1] of the parent of U[l][r]
  int32_t* first;                 // first sorted point of every non-empty leaf
};

constexpr int ERR_SLOT = OC_MAX_DEPTH + 1;

void carve(Arena& a, int B, int d, int fd, int64_t P, const int64_t* ub, int nblk_sort,
           int64_t ntile_max, Scratch& s) {
  s.k0 = a.take<uint32_t>(P);
  s.k1 = a.take<uint32_t>(P);
  s.v0 = a.take<int32_t>(P);
  s.v1 = a.take<int32_t>(P);
  s.hist = a.take<uint32_t>(256 * (int64_t)nblk_sort);
  s.offs = a.take<int32_t>(B + 1);
  s.tiles = a.take<uint32_t>(ntile_max);
  s.counts = a.take<int>(16);
  for (int l = 0; l <= d; ++l) {
    s.U[l] = a.take<uint32_t>(ub[l]);
    s.J[l] = l > fd ? a.take<int32_t>(ub[l]) : nullptr;
  }
  s.first = a.take<int32_t>(ub[d]);
}

// Adjacent-unique of n (device count n_dev, or host n_host) sorted keys >> shift.
void unique_pass(const uint32_t* keys, const int* n_dev, int64_t n_bound, int shift, Scratch& s,
                 uint32_t* uniq, int32_t* run_of, int32_t* first, int* count, hipStream_t st) {
  const int ntile = (int)oc::cdiv(n_bound, UQ_TILE);
  const int nh = n_dev ? 0 : (int)n_bound;
  hipLaunchKernelGGL(k_unique_count, dim3(ntile), dim3(TB), 0, st, keys, n_dev, nh, shift, s.tiles);
  hipLaunchKernelGGL(k_scan_tiles, dim3(1), dim3(TB), 0, st, s.tiles, ntile, count);
  hipLaunchKernelGGL(k_unique_write, dim3(ntile), dim3(TB), 0, st, keys, n_dev, nh, shift,
                     (const uint32_t*)s.tiles, uniq, run_of, first);
}

int ceil_log2(int64_t v) {
  int b = 0;
  while ((int64_t(1) << b) < v) ++b;
  return b;
}

}  // namespace

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
  if (P > (int64_t(1) << 28)) return fail(OC_ERR_UNSUPPORTED, "oc_build: %lld points > 2^28", (long long)P);
  if (P > 0 && (!points || !normals)) return fail(OC_ERR_ARG, "oc_build: points/normals NULL");
  if (((int64_t)batch << (3 * full_depth)) > (int64_t(1) << 28))
    return fail(OC_ERR_UNSUPPORTED, "oc_build: batch * 8^full_depth too large");

  const oc_allocator A = alloc ? *alloc : oc_allocator{nullptr, nullptr, nullptr};
  const int B = batch, d = depth, fd = full_depth;

  // Upper bounds of M_l (exact below full_depth).
  int64_t ub[OC_MAX_DEPTH + 1] = {};
  for (int l = 0; l <= d; ++l) {
    const int64_t full = (int64_t)B << (3 * l);
    ub[l] = l < fd ? full : std::min<int64_t>(P, full);
  }
  const int nblk_sort = (int)std::max<int64_t>(1, oc::cdiv(P, RS_TILE));
  const int64_t ntile_max = std::max<int64_t>(1, oc::cdiv(std::max<int64_t>(P, 1), UQ_TILE));

  Arena meas;
  Scratch s{};
  carve(meas, B, d, fd, P, ub, nblk_sort, ntile_max, s);
  Arena ar;
  ar.base = (char*)oc::dev_alloc(A, meas.used, stream);
  if (!ar.base) return fail(OC_ERR_NOMEM, "oc_build: scratch allocation of %zu bytes failed", meas.used);
  carve(ar, B, d, fd, P, ub, nblk_sort, ntile_max, s);
  auto release = [&](void* p) { oc::dev_free(A, p, stream); };

  hipError_t he = hipMemcpyAsync(s.offs, shape_offsets, sizeof(int32_t) * (B + 1),
                                 hipMemcpyHostToDevice, stream);
  if (he != hipSuccess) {
    release(ar.base);
    return fail(OC_ERR_DEVICE, "oc_build: offsets copy: %s", hipGetErrorString(he));
  }
  oc::fill_u32(s.counts, 0u, 16, stream);

  // 1.-2. keys and sort
  uint32_t* ks = s.k0;
  int32_t* vs = s.v0;
  if (P > 0) {
    hipLaunchKernelGGL(k_quant_key, dim3(blocks_for(P)), dim3(TB), 0, stream, points, s.offs, B,
                       (int)P, d, s.k0, s.v0, s.counts + ERR_SLOT);
    const int bits = 3 * d + ceil_log2(B);
    uint32_t* kt = s.k1;
    int32_t* vt = s.v1;
    for (int shift = 0; shift < bits; shift += 8) {
      hipLaunchKernelGGL(k_radix_hist, dim3(nblk_sort), dim3(TB), 0, stream, ks, (int)P, shift,
                         s.hist, nblk_sort);
      hipLaunchKernelGGL(k_radix_scan, dim3(1), dim3(TB), 0, stream, s.hist, nblk_sort);
      hipLaunchKernelGGL(k_radix_scatter, dim3(nblk_sort), dim3(TB), 0, stream, ks, vs, kt, vt,
                         (int)P, shift, (const uint32_t*)s.hist, nblk_sort);
      std::swap(ks, kt);
      std::swap(vs, vt);
    }
    // 3. non-empty leaves and their first points
    unique_pass(ks, nullptr, P, 0, s, s.U[d], nullptr, s.first, s.counts + d, stream);
    // 4. shallower depths down to full_depth
    for (int l = d - 1; l >= fd; --l)
      unique_pass(s.U[l + 1], s.counts + (l + 1), std::max<int64_t>(ub[l + 1], 1), 3, s, s.U[l],
                  s.J[l + 1], nullptr, s.counts + l, stream);
  }
  for (int l = 0; l < fd; ++l)
    hipLaunchKernelGGL(k_iota, dim3(blocks_for(ub[l])), dim3(TB), 0, stream, s.U[l], (int)ub[l]);

  int host_counts[16] = {};
  he = hipGetLastError();
  if (he == hipSuccess)
    he = hipMemcpyAsync(host_counts, s.counts, sizeof(host_counts), hipMemcpyDeviceToHost, stream);
  if (he == hipSuccess) he = hipStreamSynchronize(stream);
  if (he != hipSuccess) {
    release(ar.base);
    return fail(OC_ERR_DEVICE, "oc_build: %s", hipGetErrorString(he));
  }
  if (host_counts[ERR_SLOT]) {
    release(ar.base);
    return fail(OC_ERR_RANGE, "oc_build: a point is outside [0,1]^3 or NaN");
  }

  oc_octree* t = new oc_octree;
  t->depth = d;
  t->full_depth = fd;
  t->batch = B;
  t->alloc = A;
  t->stream = stream;
  for (int l = 0; l <= d; ++l) {
    t->M[l] = l < fd ? ub[l] : host_counts[l];
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

  // 5. top-down emission
  for (int l = 0; l <= d; ++l) {
    if (t->N[l] > 0)
      hipLaunchKernelGGL(k_emit_keys, dim3(blocks_for(t->N[l])), dim3(TB), 0, stream,
                         l > 0 ? (const uint32_t*)s.U[l - 1] : nullptr, (int)t->N[l], l, t->keys[l],
                         t->labels[l]);
    if (t->M[l] > 0)
      hipLaunchKernelGGL(k_emit_labels, dim3(blocks_for(t->M[l])), dim3(TB), 0, stream,
                         (const uint32_t*)s.U[l], (const int32_t*)s.J[l], (int)t->M[l], l,
                         (l == 0 || l - 1 < fd) ? 1 : 0, t->labels[l], t->rows[l]);
  }
  // input signal
  oc::fill_u32(t->signal, 0u, 3 * t->N[d], stream);
  if (t->M[d] > 0)
    hipLaunchKernelGGL(k_leaf_mean, dim3(blocks_for(t->M[d])), dim3(TB), 0, stream,
                       (const int32_t*)s.first, (int)t->M[d], (int)P, (const int32_t*)vs, normals,
                       (const int32_t*)t->rows[d], t->signal);

  // 6. hash tables and sibling-group neighbour tables
  int logc[OC_MAX_DEPTH + 1] = {};
  size_t hbytes = 0;
  for (int l = 1; l <= d; ++l) {
    logc[l] = std::max(6, ceil_log2(2 * t->M[l - 1]));
    if (t->M[l - 1] > 0) hbytes += oc::align256(8ull << logc[l]);
  }
  char* hb = hbytes ? (char*)oc::dev_alloc(A, hbytes, stream) : nullptr;
  if (hbytes && !hb) {
    release(ar.base);
    oc_octree_free(t);
    return fail(OC_ERR_NOMEM, "oc_build: hash allocation of %zu bytes failed", hbytes);
  }
  size_t hoff = 0;
  for (int l = 1; l <= d; ++l) {
    const int64_t m = t->M[l - 1];
    if (m == 0) continue;
    auto* table = (unsigned long long*)(hb + hoff);
    hoff += oc::align256(8ull << logc[l]);
    oc::fill_u32(table, 0xFFFFFFFFu, int64_t(2) << logc[l], stream);
    hipLaunchKernelGGL(k_hash_insert, dim3(blocks_for(m)), dim3(TB), 0, stream,
                       (const uint32_t*)s.U[l - 1], (int)m, table, logc[l]);
    hipLaunchKernelGGL(k_nbr, dim3(blocks_for(27 * m)), dim3(TB), 0, stream,
                       (const uint32_t*)s.U[l - 1], (int)m, l, (const unsigned long long*)table,
                       logc[l], t->nbr[l]);
  }
  he = hipGetLastError();
  if (hb) release(hb);
  release(ar.base);
  if (he != hipSuccess) {
    oc_octree_free(t);
    return fail(OC_ERR_DEVICE, "oc_build: launch failed: %s", hipGetErrorString(he));
  }
  *out = t;
  return OC_OK;
}
