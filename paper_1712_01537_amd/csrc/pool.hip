// 2x2x2 max-pooling and max-unpooling across depths through the label
// buffer (Sec. 3.2 "Pooling" and "Unpooling", Fig. 5 of O-CNN), and general
// pooling over the convolution's neighbourhood, stride 1 (k_gpool_*) and
// stride 2^r (k_gpool_sr_*), below.
//
// The eight children of the non-empty octant with label p occupy rows
// 8(p-1)..8(p-1)+7 of the finer depth, so pooling is a max over 8 contiguous
// rows; the paper's temporary packed array is fused away: the kernel writes
// the row of the parent directly (found through the label of that row), and
// empty parents get zeros.  One thread handles VEC consecutive channels of one
// row; a wavefront therefore streams whole rows (coalesced), and the eight
// child rows it reads are one contiguous 8*C*4-byte span.
#include "common.h"
#include "conv_sr.h"

namespace {

constexpr int TB = 256;

template <int VEC>
struct Vec;
template <>
struct Vec<1> {
  using f = float;
  using u8 = uint8_t;
};
template <>
struct Vec<4> {
  using f = float4;
  using u8 = uchar4;
};

__device__ __forceinline__ float comp(const float& v, int) { return v; }
__device__ __forceinline__ float comp(const float4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}
__device__ __forceinline__ void set(float& v, int, float a) { v = a; }
__device__ __forceinline__ void set(float4& v, int i, float a) {
  if (i == 0) v.x = a;
  else if (i == 1) v.y = a;
  else if (i == 2) v.z = a;
  else v.w = a;
}
__device__ __forceinline__ uint8_t comp(const uint8_t& v, int) { return v; }
__device__ __forceinline__ uint8_t comp(const uchar4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}
__device__ __forceinline__ void set(uint8_t& v, int, uint8_t a) { v = a; }
__device__ __forceinline__ void set(uchar4& v, int i, uint8_t a) {
  if (i == 0) v.x = a;
  else if (i == 1) v.y = a;
  else if (i == 2) v.z = a;
  else v.w = a;
}

// y[i] (depth l-1) = max over the children of row i, sw = first argmax.
template <int VEC>
__global__ __launch_bounds__(TB) void k_pool_fwd(const float* __restrict__ x,
                                                 const int32_t* __restrict__ labels, int64_t n_out,
                                                 int cv, float* __restrict__ y,
                                                 uint8_t* __restrict__ sw) {
  using F = typename Vec<VEC>::f;
  using U = typename Vec<VEC>::u8;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_out * cv) return;
  const int64_t i = t / cv;
  const int cc = (int)(t - i * cv);
  const int32_t L = labels[i];
  F out;
  if (L == 0) {
    for (int e = 0; e < VEC; ++e) set(out, e, 0.0f);
    reinterpret_cast<F*>(y)[t] = out;
    return;
  }
  const int64_t g = L - 1;
  const F* src = reinterpret_cast<const F*>(x) + (8 * g) * cv + cc;
  F best = src[0];
  U arg;
  for (int e = 0; e < VEC; ++e) set(arg, e, (uint8_t)0);
#pragma unroll
  for (int k = 1; k < 8; ++k) {
    const F v = src[(int64_t)k * cv];
#pragma unroll
    for (int e = 0; e < VEC; ++e)
      if (comp(v, e) > comp(best, e)) {  // strict: the first maximum wins ties
        set(best, e, comp(v, e));
        set(arg, e, (uint8_t)k);
      }
  }
  reinterpret_cast<F*>(y)[t] = best;
  reinterpret_cast<U*>(sw)[g * cv + cc] = arg;
}

// Routing through the switches (pool backward == unpool forward):
// out[8g + k][c] = (sw[g][c] == k) ? in[rows[g]][c] : 0 for every child row.
// With ymask, the routed value is also zeroed where ymask[rows[g]][c] <= 0.
// One thread per (non-empty parent g, VEC channels): it reads the parent's
// row, mask and switches once and writes all eight child rows (consecutive
// threads take consecutive channels, so each of the eight stores of a wave
// covers whole child rows).
template <int VEC>
__global__ __launch_bounds__(TB) void k_route_down(const float* __restrict__ in,
                                                   const float* __restrict__ ymask,
                                                   const uint8_t* __restrict__ sw,
                                                   const int32_t* __restrict__ rows, int64_t ngroups,
                                                   int cv, float* __restrict__ out) {
  using F = typename Vec<VEC>::f;
  using U = typename Vec<VEC>::u8;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ngroups * cv) return;
  const int64_t g = t / cv;
  const int cc = (int)(t - g * cv);
  const U s = reinterpret_cast<const U*>(sw)[t];
  const int64_t src = (int64_t)rows[g] * cv + cc;
  const F v = reinterpret_cast<const F*>(in)[src];
  F m;
  if (ymask) m = reinterpret_cast<const F*>(ymask)[src];
  F* dst = reinterpret_cast<F*>(out) + 8 * g * cv + cc;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    F o;
#pragma unroll
    for (int e = 0; e < VEC; ++e)
      set(o, e, comp(s, e) == k && (!ymask || comp(m, e) > 0.0f) ? comp(v, e) : 0.0f);
    dst[(int64_t)k * cv] = o;
  }
}

// Unpool backward: dx[i][c] = dy[8g + sw[g][c]][c] for label L = g+1 > 0.
template <int VEC>
__global__ __launch_bounds__(TB) void k_route_up(const float* __restrict__ dy,
                                                 const uint8_t* __restrict__ sw,
                                                 const int32_t* __restrict__ labels,
                                                 int64_t n_out, int cv, float* __restrict__ dx) {
  using F = typename Vec<VEC>::f;
  using U = typename Vec<VEC>::u8;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_out * cv) return;
  const int64_t i = t / cv;
  const int cc = (int)(t - i * cv);
  const int32_t L = labels[i];
  F o;
  if (L == 0) {
    for (int e = 0; e < VEC; ++e) set(o, e, 0.0f);
  } else {
    const int64_t g = L - 1;
    const U s = reinterpret_cast<const U*>(sw)[g * cv + cc];
    const float* base = dy + (8 * g) * (int64_t)(cv * VEC) + (int64_t)cc * VEC;
#pragma unroll
    for (int e = 0; e < VEC; ++e) set(o, e, base[(int64_t)comp(s, e) * cv * VEC + e]);
  }
  reinterpret_cast<F*>(dx)[t] = o;
}

inline unsigned grid_for(int64_t n) { return (unsigned)oc::cdiv(n, TB); }
// ---------------------------------------------------------------------------
// General pooling, stride 1 (Sec. 3.2, last paragraph of "Pooling"): the K^3
// neighbourhood of every octant is found as for the convolution, through the
// sibling group's 27 parent-neighbour entries (neighbour of child c at offset
// d: parent offset floor((c + d) / 2), child (c + d) & 1 of it), and each
// channel takes the max or the average over it.  A neighbour that is not in
// the octree reads as zero, as in the convolution.  One thread handles VEC
// consecutive channels of one row; the forward takes the taps in blocks of
// KB whose neighbour lookups, then row loads, are all issued before any is
// used, so their latencies overlap.  (Staging the groups' (K+1)^3 union blocks in LDS
// was measured slower: the blocks take so much LDS that too few waves run.)
template <int R>
__device__ __forceinline__ int64_t gp_src(const int32_t* __restrict__ nbr, int64_t i, int k) {
  constexpr int K = 2 * R + 1;
  const int c = (int)(i & 7);
  const int ux = (c >> 2) + k / (K * K) - R, uy = ((c >> 1) & 1) + (k / K) % K - R,
            uz = (c & 1) + k % K - R;
  const int32_t base = nbr[27 * (i >> 3) + ((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1)];
  return base < 0 ? -1 : (int64_t)base + 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1);
}

// taps per block: the forward's whole neighbourhood (K = 3) or a fifth of it.
// The backward takes one tap at a time: with blocks (of 9 or 5 taps, whose
// switches it holds as well) it ran fewer waves and was measured slower.
template <int R, bool BWD>
constexpr int gp_kb() { return BWD ? 1 : (R == 1 ? 27 : 25); }

// Forward: y = max (first maximum in tap order; sw = its tap, or 255 when it
// is an absent neighbour's zero) or sum / K^3 over the taps.
template <int R, bool AVG, int VEC>
__global__ __launch_bounds__(TB) void k_gpool_fwd(const int32_t* __restrict__ nbr, int64_t n,
                                                  const float* __restrict__ x, int cv,
                                                  float* __restrict__ y,
                                                  uint8_t* __restrict__ sw) {
  using F = typename Vec<VEC>::f;
  using U = typename Vec<VEC>::u8;
  constexpr int K3 = (2 * R + 1) * (2 * R + 1) * (2 * R + 1), KB = gp_kb<R, false>();
  static_assert(K3 % KB == 0, "tap blocks");
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n * cv) return;
  const int64_t i = t / cv;
  const int q = (int)(t - i * cv);
  const F* xv = reinterpret_cast<const F*>(x);
  F acc;
  U arg;
#pragma unroll
  for (int e = 0; e < VEC; ++e) set(acc, e, 0.f), set(arg, e, (uint8_t)255);
#pragma unroll 1
  for (int k0 = 0; k0 < K3; k0 += KB) {
    int64_t src[KB];
    F v[KB];
#pragma unroll
    for (int j = 0; j < KB; ++j) src[j] = gp_src<R>(nbr, i, k0 + j);
#pragma unroll
    for (int j = 0; j < KB; ++j) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) set(v[j], e, 0.f);
      if (src[j] >= 0) v[j] = xv[src[j] * cv + q];
    }
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      const int k = k0 + j;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float a = comp(v[j], e);
        if constexpr (AVG) {
          set(acc, e, comp(acc, e) + a);
        } else if (k == 0 || a > comp(acc, e)) {
          set(acc, e, a);
          set(arg, e, src[j] >= 0 ? (uint8_t)k : (uint8_t)255);
        }
      }
    }
  }
  if constexpr (AVG) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) set(acc, e, comp(acc, e) / (float)K3);
  } else {
    reinterpret_cast<U*>(sw)[t] = arg;
  }
  reinterpret_cast<F*>(y)[t] = acc;
}

// Average pooling, stride 1, as separable box sums over each sibling group's
// union block: the (2R+1)^3 neighbourhoods of the group's eight children
// tile the (2R+2)^3 block of positions around the group (Fig. 4), so their
// sums are the block's window sums along z (per (x, y) line), then along y,
// then along x, about a third of the additions and a fifth of the row reads
// of summing each child's neighbourhood.  Absent positions are zero (the
// zero-padded average, reading 16), and the sum is divided by (2R+1)^3.
// Thread (group g, channel quad q) writes rows 8g .. 8g+7.  The additions
// run in a fixed order, so results are reproducible.
template <int R>
__global__ __launch_bounds__(TB) void k_gpool_avg_sep(const int32_t* __restrict__ nbr,
                                                      int64_t ngroups,
                                                      const float* __restrict__ x, int cv,
                                                      float* __restrict__ y) {
  constexpr int K = 2 * R + 1, S = K + 1, K3 = K * K * K;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ngroups * cv) return;
  const int64_t g = t / cv;
  const int q = (int)(t - g * cv);
  const float4* xv = reinterpret_cast<const float4*>(x);
  int32_t nb[27];
#pragma unroll
  for (int c = 0; c < 27; ++c) nb[c] = nbr[27 * g + c];
  auto at = [&](int ix, int iy, int iz) -> float4 {  // block position (ix, iy, iz)
    const int ux = ix - R, uy = iy - R, uz = iz - R;
    const int32_t b = nb[((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1)];
    if (b < 0) return make_float4(0.f, 0.f, 0.f, 0.f);
    return xv[((int64_t)b + 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1)) * cv + q];
  };
  auto add = [](float4 a, float4 b) { return make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w); };
  float4 o[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) o[c] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 1
  for (int ix = 0; ix < S; ++ix) {
    float4 z[S][2];  // window sums along z of each y line, for cz = 0, 1
#pragma unroll
    for (int iy = 0; iy < S; ++iy) {
      float4 b[S];
#pragma unroll
      for (int iz = 0; iz < S; ++iz) b[iz] = at(ix, iy, iz);
      float4 m = b[1];
#pragma unroll
      for (int iz = 2; iz < K; ++iz) m = add(m, b[iz]);
      z[iy][0] = add(b[0], m);
      z[iy][1] = add(m, b[K]);
    }
#pragma unroll
    for (int cy = 0; cy < 2; ++cy)
#pragma unroll
      for (int cz = 0; cz < 2; ++cz) {
        float4 w = z[cy][cz];
#pragma unroll
        for (int dy = 1; dy < K; ++dy) w = add(w, z[cy + dy][cz]);
        // this x-slab is in the x-window of child cx = 0 when ix < K, of
        // cx = 1 when ix >= 1
        if (ix < K) o[2 * cy + cz] = add(o[2 * cy + cz], w);
        if (ix >= 1) o[4 + 2 * cy + cz] = add(o[4 + 2 * cy + cz], w);
      }
  }
  float4* yv = reinterpret_cast<float4*>(y);
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const float4 v = o[c];
    yv[(8 * g + c) * cv + q] = make_float4(v.x / (float)K3, v.y / (float)K3, v.z / (float)K3,
                                           v.w / (float)K3);
  }
}

// Max pooling, stride 1, the same way: window maxima of each group's union
// block along z, then y, then x.  Each stage keeps its first candidate and
// replaces it only by a strictly greater value, so the winner is the first
// maximum in the order (dx, dy, dz), which is the tap order k = (dx K + dy)
// K + dz of the one-tap-at-a-time scan: the switch is k, or 255 when the
// winning position is absent (absent positions take part as zeros).
// Thread (group g, channel quad q).  For finite inputs (a NaN first in a
// window would hide the rest of that window).
template <int R>
__global__ __launch_bounds__(TB) void k_gpool_max_sep(const int32_t* __restrict__ nbr,
                                                      int64_t ngroups,
                                                      const float* __restrict__ x, int cv,
                                                      float* __restrict__ y,
                                                      uint8_t* __restrict__ sw) {
  constexpr int K = 2 * R + 1, S = K + 1;
  constexpr int ABSENT = 256;  // flag on a candidate's code: the position is absent
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ngroups * cv) return;
  const int64_t g = t / cv;
  const int q = (int)(t - g * cv);
  const float4* xv = reinterpret_cast<const float4*>(x);
  int32_t nb[27];
#pragma unroll
  for (int c = 0; c < 27; ++c) nb[c] = nbr[27 * g + c];
  // candidate: four channel values and their codes (partial tap index | ABSENT)
  struct Cand {
    float v[4];
    int k[4];
  };
  auto better = [](Cand& m, const Cand& c, int add) {  // strictly greater replaces
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (c.v[e] > m.v[e]) m.v[e] = c.v[e], m.k[e] = c.k[e] + add;
  };
  auto shifted = [](const Cand& c, int add) {
    Cand r = c;
#pragma unroll
    for (int e = 0; e < 4; ++e) r.k[e] += add;
    return r;
  };
  Cand o[8];
#pragma unroll 1
  for (int ix = 0; ix < S; ++ix) {
    Cand z[S][2];  // per y line: the z-window maxima for cz = 0, 1 (code dz)
#pragma unroll
    for (int iy = 0; iy < S; ++iy) {
      Cand b[S];
#pragma unroll
      for (int iz = 0; iz < S; ++iz) {
        const int ux = ix - R, uy = iy - R, uz = iz - R;
        const int32_t base = nb[((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1)];
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        int code = ABSENT;
        if (base >= 0) {
          v = xv[((int64_t)base + 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1)) * cv + q];
          code = 0;
        }
        b[iz].v[0] = v.x, b[iz].v[1] = v.y, b[iz].v[2] = v.z, b[iz].v[3] = v.w;
#pragma unroll
        for (int e = 0; e < 4; ++e) b[iz].k[e] = code;
      }
#pragma unroll
      for (int cz = 0; cz < 2; ++cz) {
        Cand m = b[cz];
#pragma unroll
        for (int dz = 1; dz < K; ++dz) better(m, b[cz + dz], dz);
        z[iy][cz] = m;
      }
    }
#pragma unroll
    for (int cy = 0; cy < 2; ++cy)
#pragma unroll
      for (int cz = 0; cz < 2; ++cz) {
        Cand m = z[cy][cz];
#pragma unroll
        for (int dy = 1; dy < K; ++dy) better(m, z[cy + dy][cz], K * dy);
        // the x-windows of child cx take this slab at dx = ix - cx
        const int c0 = 2 * cy + cz, c1 = 4 + 2 * cy + cz;
        if (ix == 0) o[c0] = m;
        else if (ix < K) better(o[c0], m, K * K * ix);
        if (ix == 1) o[c1] = m;
        else if (ix > 1) better(o[c1], m, K * K * (ix - 1));
      }
  }
  float4* yv = reinterpret_cast<float4*>(y);
  uint32_t* sv = reinterpret_cast<uint32_t*>(sw);
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int64_t r = (8 * g + c) * cv + q;
    yv[r] = make_float4(o[c].v[0], o[c].v[1], o[c].v[2], o[c].v[3]);
    uint32_t packed = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t k = o[c].k[e] >= ABSENT ? 255u : (uint32_t)o[c].k[e];
      packed |= k << (8 * e);
    }
    sv[r] = packed;
  }
}

// Backward of the max by sibling group: the outputs whose taps can land on
// a group's eight rows are the positions of its union block (child c takes,
// for tap k = (dx, dy, dz), the output at block position c + 2R - d), so
// thread (group g, channel quad q) reads each block position's dy and
// switches once, an x-slab at a time, and adds to row 8g + c the dy of every
// position whose switch names the tap that lands on c.  The additions run
// in a fixed order (x-slab, then child, then tap).
template <int R>
__global__ __launch_bounds__(TB) void k_gpool_max_bwd_sep(const int32_t* __restrict__ nbr,
                                                          int64_t ngroups,
                                                          const float* __restrict__ dy,
                                                          const uint8_t* __restrict__ sw, int cv,
                                                          float* __restrict__ dx) {
  constexpr int K = 2 * R + 1, S = K + 1;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= ngroups * cv) return;
  const int64_t g = t / cv;
  const int q = (int)(t - g * cv);
  const float4* dv = reinterpret_cast<const float4*>(dy);
  const uint32_t* sv = reinterpret_cast<const uint32_t*>(sw);
  int32_t nb[27];
#pragma unroll
  for (int c = 0; c < 27; ++c) nb[c] = nbr[27 * g + c];
  float4 acc[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) acc[c] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 1
  for (int ix = 0; ix < S; ++ix) {
    float4 d[S][S];
    uint32_t w[S][S];  // switches; 0xffffffff for an absent position (matches no tap)
#pragma unroll
    for (int iy = 0; iy < S; ++iy)
#pragma unroll
      for (int iz = 0; iz < S; ++iz) {
        const int ux = ix - R, uy = iy - R, uz = iz - R;
        const int32_t base = nb[((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1)];
        d[iy][iz] = make_float4(0.f, 0.f, 0.f, 0.f);
        w[iy][iz] = 0xffffffffu;
        if (base >= 0) {
          const int64_t r = ((int64_t)base + 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1)) * cv + q;
          d[iy][iz] = dv[r];
          w[iy][iz] = sv[r];
        }
      }
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const int cx = c >> 2, cy = (c >> 1) & 1, cz = c & 1;
      const int ddx = cx + 2 * R - ix;  // the tap's x index that lands on c from this slab
      if (ddx < 0 || ddx >= K) continue;
#pragma unroll
      for (int ddy = 0; ddy < K; ++ddy)
#pragma unroll
        for (int ddz = 0; ddz < K; ++ddz) {
          const int py = cy + 2 * R - ddy, pz = cz + 2 * R - ddz;
          const uint32_t k = (uint32_t)((ddx * K + ddy) * K + ddz);
          const uint32_t sw4 = w[py][pz];
          const float4 v = d[py][pz];
          if ((sw4 & 0xffu) == k) acc[c].x += v.x;
          if (((sw4 >> 8) & 0xffu) == k) acc[c].y += v.y;
          if (((sw4 >> 16) & 0xffu) == k) acc[c].z += v.z;
          if ((sw4 >> 24) == k) acc[c].w += v.w;
        }
    }
  }
  float4* xv = reinterpret_cast<float4*>(dx);
#pragma unroll
  for (int c = 0; c < 8; ++c) xv[(8 * g + c) * cv + q] = acc[c];
}

// Backward of the max as a gather, in tap order: input row n receives, from
// the octant i whose tap k lands on n (i is n's neighbour at the mirrored
// offset, tap K^3 - 1 - k), dy[i] where sw[i] == k.  (The average's
// backward runs on the forward kernel; see gpool below.)
template <int R, int VEC>
__global__ __launch_bounds__(TB) void k_gpool_bwd(const int32_t* __restrict__ nbr, int64_t n,
                                                  const float* __restrict__ dy,
                                                  const uint8_t* __restrict__ sw, int cv,
                                                  float* __restrict__ dx) {
  using F = typename Vec<VEC>::f;
  using U = typename Vec<VEC>::u8;
  constexpr int K3 = (2 * R + 1) * (2 * R + 1) * (2 * R + 1), KB = gp_kb<R, true>();
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n * cv) return;
  const int64_t j0 = t / cv;
  const int q = (int)(t - j0 * cv);
  const F* gv = reinterpret_cast<const F*>(dy);
  const U* sv = reinterpret_cast<const U*>(sw);
  F acc;
#pragma unroll
  for (int e = 0; e < VEC; ++e) set(acc, e, 0.f);
#pragma unroll 1
  for (int k0 = 0; k0 < K3; k0 += KB) {
    int64_t src[KB];
    F g[KB];
    U s[KB];
#pragma unroll
    for (int j = 0; j < KB; ++j) src[j] = gp_src<R>(nbr, j0, K3 - 1 - (k0 + j));
#pragma unroll
    for (int j = 0; j < KB; ++j) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) set(g[j], e, 0.f), set(s[j], e, (uint8_t)255);
      if (src[j] >= 0) {
        g[j] = gv[src[j] * cv + q];
        s[j] = sv[src[j] * cv + q];
      }
    }
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      if (src[j] < 0) continue;
#pragma unroll
      for (int e = 0; e < VEC; ++e)
        if (comp(s[j], e) == k0 + j) set(acc, e, comp(acc, e) + comp(g[j], e));
    }
  }
  reinterpret_cast<F*>(dx)[t] = acc;
}

// Strided general pooling (stride 2^r, K = 3): the neighbourhood of the
// stride-2^r convolution (the first depth-l position below every non-empty
// depth-(l-r) octant, its 27 taps reading children of the eight depth-(l-1)
// octants of sr_first_child), absent neighbours as zeros.  Forward: one
// thread per (depth-(l-r) row, VEC channels); rows of empty octants get 0
// and switch 255.
template <bool AVG, int VEC>
__global__ __launch_bounds__(TB) void k_gpool_sr_fwd(const int32_t* __restrict__ nbr,
                                                     oc::SrLabels L, int r,
                                                     const int32_t* __restrict__ labels,
                                                     int64_t n_out, const float* __restrict__ x,
                                                     int cv, float* __restrict__ y,
                                                     uint8_t* __restrict__ sw) {
  using F = typename Vec<VEC>::f;
  using U = typename Vec<VEC>::u8;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_out * cv) return;
  const int64_t i = t / cv;
  const int q = (int)(t - i * cv);
  const F* xv = reinterpret_cast<const F*>(x);
  F acc;
  U arg;
#pragma unroll
  for (int e = 0; e < VEC; ++e) set(acc, e, 0.f), set(arg, e, (uint8_t)255);
  const int32_t lab = labels[i];
  if (lab > 0) {
    int32_t fc[8];
#pragma unroll
    for (int o = 0; o < 8; ++o) fc[o] = oc::sr_first_child(nbr, L, lab - 1, o, r);
    F v[27];
#pragma unroll
    for (int k = 0; k < 27; ++k) {
      const int32_t f = fc[oc::sr_tap_o(k)];
#pragma unroll
      for (int e = 0; e < VEC; ++e) set(v[k], e, 0.f);
      if (f >= 0) v[k] = xv[((int64_t)f + oc::sr_tap_c(k)) * cv + q];
    }
#pragma unroll
    for (int k = 0; k < 27; ++k) {
      const bool present = fc[oc::sr_tap_o(k)] >= 0;
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        const float a = comp(v[k], e);
        if constexpr (AVG) {
          set(acc, e, comp(acc, e) + a);
        } else if (k == 0 || a > comp(acc, e)) {
          set(acc, e, a);
          set(arg, e, present ? (uint8_t)k : (uint8_t)255);
        }
      }
    }
    if constexpr (AVG) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) set(acc, e, comp(acc, e) / 27.f);
    }
  }
  if constexpr (!AVG) reinterpret_cast<U*>(sw)[t] = arg;
  reinterpret_cast<F*>(y)[t] = acc;
}

// Backward, r = 1, as a gather: depth-l row 8h + c (child c of group h) is
// read by the outputs at parent offsets o in {0,1}^3 from h's parent with
// o_a <= c_a, through tap c - 2o (the strided convolution's input-gradient
// rule); their contributions are added in increasing o.
template <bool AVG, int VEC>
__global__ __launch_bounds__(TB) void k_gpool_s2_bwd(const int32_t* __restrict__ nbr, int64_t n_in,
                                                     const int32_t* __restrict__ rows,
                                                     const float* __restrict__ dy,
                                                     const uint8_t* __restrict__ sw, int cv,
                                                     float* __restrict__ dx) {
  using F = typename Vec<VEC>::f;
  using U = typename Vec<VEC>::u8;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= n_in * cv) return;
  const int64_t n = t / cv;
  const int q = (int)(t - n * cv);
  const int c = (int)(n & 7);
  const int64_t h = n >> 3;
  const F* gv = reinterpret_cast<const F*>(dy);
  const U* sv = reinterpret_cast<const U*>(sw);
  F acc;
#pragma unroll
  for (int e = 0; e < VEC; ++e) set(acc, e, 0.f);
#pragma unroll
  for (int o = 0; o < 8; ++o) {
    if ((o & ~c) != 0) continue;
    const int32_t f = nbr[27 * h + ((o >> 2) + 1) * 9 + (((o >> 1) & 1) + 1) * 3 + ((o & 1) + 1)];
    if (f < 0) continue;
    int k = 0;
#pragma unroll
    for (int a = 2; a >= 0; --a) k = 3 * k + (((c >> a) & 1) - 2 * ((o >> a) & 1) + 1);
    const int64_t row = rows[f >> 3];
    const F g = gv[row * cv + q];
    if constexpr (AVG) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) set(acc, e, comp(acc, e) + comp(g, e) / 27.f);
    } else {
      const U sgl = sv[row * cv + q];
#pragma unroll
      for (int e = 0; e < VEC; ++e)
        if (comp(sgl, e) == k) set(acc, e, comp(acc, e) + comp(g, e));
    }
  }
  reinterpret_cast<F*>(dx)[t] = acc;
}

// Backward, r >= 2: every depth-l row is read by at most one (output, tap),
// so each output scatters its taps' shares over a zeroed dx.
template <bool AVG, int VEC>
__global__ __launch_bounds__(TB) void k_gpool_sr_bwd(const int32_t* __restrict__ nbr,
                                                     oc::SrLabels L, int r, int64_t G,
                                                     const int32_t* __restrict__ rows,
                                                     const float* __restrict__ dy,
                                                     const uint8_t* __restrict__ sw, int cv,
                                                     float* __restrict__ dx) {
  using F = typename Vec<VEC>::f;
  using U = typename Vec<VEC>::u8;
  const int64_t t = (int64_t)blockIdx.x * TB + threadIdx.x;
  if (t >= G * cv) return;
  const int64_t p = t / cv;
  const int q = (int)(t - p * cv);
  const int64_t row = rows[p];
  const F g = reinterpret_cast<const F*>(dy)[row * cv + q];
  U sgl;
  if constexpr (!AVG) sgl = reinterpret_cast<const U*>(sw)[row * cv + q];
  int32_t fc[8];
#pragma unroll
  for (int o = 0; o < 8; ++o) fc[o] = oc::sr_first_child(nbr, L, p, o, r);
#pragma unroll
  for (int k = 0; k < 27; ++k) {
    const int32_t f = fc[oc::sr_tap_o(k)];
    if (f < 0) continue;
    F v;
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      if constexpr (AVG)
        set(v, e, comp(g, e) / 27.f);
      else
        set(v, e, comp(sgl, e) == k ? comp(g, e) : 0.f);
    }
    reinterpret_cast<F*>(dx)[((int64_t)f + oc::sr_tap_c(k)) * cv + q] = v;
  }
}

oc_status check_common(const oc_octree* t, int32_t l, int32_t c, const void* a, const void* b,
                       const void* s, const char* who) {
  oc_status st = oc::check_tree_level(t, l, 1);
  if (st != OC_OK) return st;
  if (c < 1 || c > 65536) return oc::fail(OC_ERR_ARG, "%s: channels %d out of range", who, c);
  if (!a || !b || !s) return oc::fail(OC_ERR_ARG, "%s: NULL buffer", who);
  return OC_OK;
}

bool vec4_ok(int c, const void* a, const void* b, const void* s) {
  return c % 4 == 0 && ((uintptr_t)a % 16 == 0) && ((uintptr_t)b % 16 == 0) &&
         ((uintptr_t)s % 4 == 0);
}

// Strided general pooling: forward over the depth-(l-r) rows; backward by
// the r = 1 gather or the r >= 2 scatter.
template <bool BWD>
oc_status gpool_sr(const oc_octree* t, int32_t l, int32_t r, bool avg, const float* in,
                   const uint8_t* swin, uint8_t* swout, int32_t c, float* out, hipStream_t s) {
  const int64_t n_in = t->N[l], n_out = t->N[l - r], G = t->M[l - r];
  const uint8_t* swp = BWD ? swin : swout;
  const bool v4 = c % 4 == 0 && (uintptr_t)in % 16 == 0 && (uintptr_t)out % 16 == 0 &&
                  (avg || (uintptr_t)swp % 4 == 0);
  const int cv = v4 ? c / 4 : c;
  const int32_t* nbr = (const int32_t*)t->nbr[l - r + 1];
  const oc::SrLabels L = oc::sr_labels(t, l, r);
#define OC_GPS(AVG_, V_)                                                                        \
  if (avg == AVG_ && (v4 ? 4 : 1) == V_) {                                                      \
    if constexpr (!BWD) {                                                                       \
      if (n_out > 0)                                                                            \
        oc::launch_main(k_gpool_sr_fwd<AVG_, V_>, dim3(grid_for(n_out * cv)), dim3(TB), s, nbr, \
                        L, r, (const int32_t*)t->labels[l - r], n_out, in, cv, out, swout);     \
    } else if (r == 1) {                                                                        \
      if (n_in > 0)                                                                             \
        oc::launch_main(k_gpool_s2_bwd<AVG_, V_>, dim3(grid_for(n_in * cv)), dim3(TB), s,       \
                        (const int32_t*)t->nbr[l], n_in, (const int32_t*)t->rows[l - 1], in,    \
                        swin, cv, out);                                                         \
    } else {                                                                                    \
      if (n_in > 0) oc::fill_u32(out, 0u, n_in * c, s);                                         \
      if (G > 0)                                                                                \
        oc::launch_main(k_gpool_sr_bwd<AVG_, V_>, dim3(grid_for(G * cv)), dim3(TB), s, nbr, L,  \
                        r, G, (const int32_t*)t->rows[l - r], in, swin, cv, out);               \
    }                                                                                           \
  }
  OC_GPS(false, 4) OC_GPS(false, 1) OC_GPS(true, 4) OC_GPS(true, 1)
#undef OC_GPS
  OC_LAUNCH_CHECK();
  return OC_OK;
}

template <bool BWD>
oc_status gpool(const oc_octree* t, int32_t l, int32_t K, int32_t stride, int32_t mode,
                const float* in, const uint8_t* swin, uint8_t* swout, int32_t c, float* out,
                hipStream_t s, const char* who) {
  oc_status st = oc::check_tree_level(t, l, 1);
  if (st != OC_OK) return st;
  if (K != 3 && K != 5) return oc::fail(OC_ERR_UNSUPPORTED, "%s: kernel size %d not 3 or 5", who, K);
  if (stride < 1 || (stride & (stride - 1)) != 0 || stride > (1 << l))
    return oc::fail(OC_ERR_ARG, "%s: stride %d not a power of two up to 2^depth", who, stride);
  if (stride > 1 && K != 3)
    return oc::fail(OC_ERR_UNSUPPORTED, "%s: stride %d supports kernel size 3 only", who, stride);
  if (mode != OC_POOL_MAX && mode != OC_POOL_AVG)
    return oc::fail(OC_ERR_ARG, "%s: mode %d not OC_POOL_MAX or OC_POOL_AVG", who, mode);
  if (c < 1 || c > 65536) return oc::fail(OC_ERR_ARG, "%s: channels %d out of range", who, c);
  const bool avg = mode == OC_POOL_AVG;
  const uint8_t* swp = BWD ? swin : swout;
  if (!in || !out || (!avg && !swp)) return oc::fail(OC_ERR_ARG, "%s: NULL buffer", who);
  if (stride > 1)
    return gpool_sr<BWD>(t, l, __builtin_ctz((unsigned)stride), avg, in, swin, swout, c, out, s);
  const int64_t n = t->N[l];
  if (n == 0) return OC_OK;
  const bool v4 = c % 4 == 0 && (uintptr_t)in % 16 == 0 && (uintptr_t)out % 16 == 0 &&
                  (avg || (uintptr_t)swp % 4 == 0);
  const int cv = v4 ? c / 4 : c;
  const dim3 grid(grid_for(n * cv));
  const int32_t* nbr = (const int32_t*)t->nbr[l];
  // The average's backward is the average itself applied to dy: the tap-k
  // neighbour relation is symmetric (n sees i at offset d iff i sees n at
  // -d), so both are dy summed over n's neighbourhood / K^3.  It runs on the
  // forward kernel, whose taps are batched (the same sum, divided once).
  if (BWD && !avg && v4 && K == 3) {  // the max's backward by sibling group
    const int64_t G = t->M[l - 1];
    oc::launch_main(k_gpool_max_bwd_sep<1>, dim3(grid_for(G * cv)), dim3(TB), s, nbr, G, in, swin,
                    cv, out);
    OC_LAUNCH_CHECK();
    return OC_OK;
  }
  if (!BWD && !avg && v4 && (K == 3 || K == 5)) {  // separable maxima over each group's union block
    const int64_t G = t->M[l - 1];
    const dim3 gg(grid_for(G * cv));
    if (K == 3)
      oc::launch_main(k_gpool_max_sep<1>, gg, dim3(TB), s, nbr, G, in, cv, out, swout);
    else
      oc::launch_main(k_gpool_max_sep<2>, gg, dim3(TB), s, nbr, G, in, cv, out, swout);
    OC_LAUNCH_CHECK();
    return OC_OK;
  }
  if (avg && v4 && (K == 3 || K == 5)) {  // separable sums over each group's union block
    const int64_t G = t->M[l - 1];
    const dim3 gg(grid_for(G * cv));
    if (K == 3)
      oc::launch_main(k_gpool_avg_sep<1>, gg, dim3(TB), s, nbr, G, in, cv, out);
    else
      oc::launch_main(k_gpool_avg_sep<2>, gg, dim3(TB), s, nbr, G, in, cv, out);
    OC_LAUNCH_CHECK();
    return OC_OK;
  }
#define OC_GP(R_, AVG_, V_)                                                                   \
  if (K == 2 * R_ + 1 && avg == AVG_ && (v4 ? 4 : 1) == V_) {                                 \
    if constexpr (BWD) {                                                                      \
      if (AVG_)                                                                               \
        oc::launch_main(k_gpool_fwd<R_, true, V_>, grid, dim3(TB), s, nbr, n, in, cv, out,    \
                        (uint8_t*)nullptr);                                                   \
      else                                                                                    \
        oc::launch_main(k_gpool_bwd<R_, V_>, grid, dim3(TB), s, nbr, n, in, swin, cv,         \
                        out);                                                                 \
    } else {                                                                                  \
      oc::launch_main(k_gpool_fwd<R_, AVG_, V_>, grid, dim3(TB), s, nbr, n, in, cv, out,      \
                      swout);                                                                 \
    }                                                                                         \
  }
  OC_GP(1, false, 4) OC_GP(1, false, 1) OC_GP(1, true, 4) OC_GP(1, true, 1)
  OC_GP(2, false, 4) OC_GP(2, false, 1) OC_GP(2, true, 4) OC_GP(2, true, 1)
#undef OC_GP
  OC_LAUNCH_CHECK();
  return OC_OK;
}

}  // namespace

extern "C" {

oc_status oc_pool_fwd(const oc_octree* t, int32_t l, const float* x, int32_t c, float* y,
                      uint8_t* sw, hipStream_t s) {
  oc_status st = check_common(t, l, c, x, y, sw, "oc_pool_fwd");
  if (st != OC_OK) return st;
  const int64_t n = t->N[l - 1];
  if (n == 0) return OC_OK;
  if (vec4_ok(c, x, y, sw)) {
    const int cv = c / 4;
    oc::launch_main(k_pool_fwd<4>, dim3(grid_for(n * cv)), dim3(TB), s, x,
                       (const int32_t*)t->labels[l - 1], n, cv, y, sw);
  } else {
    oc::launch_main(k_pool_fwd<1>, dim3(grid_for(n * c)), dim3(TB), s, x,
                       (const int32_t*)t->labels[l - 1], n, c, y, sw);
  }
  OC_LAUNCH_CHECK();
  return OC_OK;
}

static oc_status route_down(const oc_octree* t, int32_t l, const float* in, const float* ymask,
                            const uint8_t* sw, int32_t c, float* out, hipStream_t s,
                            const char* who) {
  oc_status st = check_common(t, l, c, in, out, sw, who);
  if (st != OC_OK) return st;
  const int64_t G = t->M[l - 1];  // the non-empty parents: N_l = 8 G child rows
  if (G == 0) return OC_OK;
  if (vec4_ok(c, in, out, sw) && (uintptr_t)ymask % 16 == 0) {
    const int cv = c / 4;
    oc::launch_main(k_route_down<4>, dim3(grid_for(G * cv)), dim3(TB), s, in, ymask, sw,
                       (const int32_t*)t->rows[l - 1], G, cv, out);
  } else {
    oc::launch_main(k_route_down<1>, dim3(grid_for(G * c)), dim3(TB), s, in, ymask, sw,
                       (const int32_t*)t->rows[l - 1], G, c, out);
  }
  OC_LAUNCH_CHECK();
  return OC_OK;
}

oc_status oc_pool_bwd(const oc_octree* t, int32_t l, const float* dy, const uint8_t* sw, int32_t c,
                      const float* y, float* dx, hipStream_t s) {
  return route_down(t, l, dy, y, sw, c, dx, s, "oc_pool_bwd");
}

oc_status oc_unpool_fwd(const oc_octree* t, int32_t l, const float* x, const uint8_t* sw,
                        int32_t c, float* y, hipStream_t s) {
  return route_down(t, l, x, nullptr, sw, c, y, s, "oc_unpool_fwd");
}

oc_status oc_unpool_bwd(const oc_octree* t, int32_t l, const float* dy, const uint8_t* sw,
                        int32_t c, float* dx, hipStream_t s) {
  oc_status st = check_common(t, l, c, dy, dx, sw, "oc_unpool_bwd");
  if (st != OC_OK) return st;
  const int64_t n = t->N[l - 1];
  if (n == 0) return OC_OK;
  if (vec4_ok(c, dy, dx, sw)) {
    const int cv = c / 4;
    oc::launch_main(k_route_up<4>, dim3(grid_for(n * cv)), dim3(TB), s, dy, sw,
                       (const int32_t*)t->labels[l - 1], n, cv, dx);
  } else {
    oc::launch_main(k_route_up<1>, dim3(grid_for(n * c)), dim3(TB), s, dy, sw,
                       (const int32_t*)t->labels[l - 1], n, c, dx);
  }
  OC_LAUNCH_CHECK();
  return OC_OK;
}

oc_status oc_gpool_fwd(const oc_octree* t, int32_t l, int32_t K, int32_t stride, int32_t mode,
                       const float* x,
                       int32_t c, float* y, uint8_t* sw, hipStream_t s) {
  return gpool<false>(t, l, K, stride, mode, x, nullptr, sw, c, y, s, "oc_gpool_fwd");
}

oc_status oc_gpool_bwd(const oc_octree* t, int32_t l, int32_t K, int32_t stride, int32_t mode,
                       const float* dy,
                       const uint8_t* sw, int32_t c, float* dx, hipStream_t s) {
  return gpool<true>(t, l, K, stride, mode, dy, sw, nullptr, c, dx, s, "oc_gpool_bwd");
}

}  // extern "C"
