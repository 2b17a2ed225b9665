// First-layer convolution (K = 3, 3 or 4 input channels: the octree's input
// signal, Sec. 3.1) forward and weight gradient on the fp32 matrix cores.
//
// With so few input channels a 4-deep MFMA reduction over channels leaves a
// quarter of it empty (Cin = 3), so the reduction index here is the flattened
// (tap, channel) pair k = 3 tap + c (Cin = 3: 81 pairs, 21 MFMA steps of 4,
// against 27 steps of one tap each).  The neighbourhood is the union tile of
// a sibling group (Fig. 4): 4^3 positions around the group's eight children,
// each position one 12- or 16-byte row.
//
// Each wave works alone over a contiguous range of tiles of two sibling
// groups (16 octants): it DMAs each tile's two position sets straight into
// its own LDS buffers (global_load_lds, 64 positions per instruction), one
// tile ahead of the MFMAs, and the neighbour-table rows of the tile after
// that into an LDS ring.  Absent neighbours read a zero row.  Every wave
// issues the same vector-memory instructions per tile (rows past the end
// read zeros or -1 entries, stores past the end go to a dummy row), so the
// waits are compile-time counts of younger operations (vector-memory
// operations complete in issue order).
#include "conv_cin.h"
#include "pool_fuse.h"

#include <algorithm>

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lptr_t;  // LDS
typedef __attribute__((address_space(3))) const char lds_char;
typedef __attribute__((address_space(3))) const float lds_float;

// The float at byte offset off of an LDS array (a 32-bit LDS address).
__device__ __forceinline__ float lds_at(const void* base, int off) {
  return *reinterpret_cast<lds_float*>((lds_char*)base + off);
}

constexpr int TB = 256;  // four waves
constexpr int NWAVE = TB / 64;
constexpr int D = 3;             // tiles in flight ahead of the MFMAs
constexpr int NBUF = D + 1;      // tile buffers per wave

__device__ __attribute__((aligned(16))) float g_cin_zero[4];  // the zero row (never written)
__device__ const int32_t g_cin_absent = -1;                   // neighbour entry past the last group
__device__ __attribute__((aligned(16))) float g_cin_dummy[64 * 4];  // stores past the last row

__device__ __forceinline__ uint32_t lds_addr(const void* lds) {
  return __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lptr_t)lds);
}
// Direct global->LDS loads: lane i's bytes land at LDS byte address
// lds + 16 i (16 or 12 bytes) or lds + 4 i (4 bytes); lds is wave-uniform.
__device__ __forceinline__ void lds_load16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(src)
               : "memory", "m0");
}
__device__ __forceinline__ void lds_load12(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx3 %1, off" ::"s"(lds), "v"(src)
               : "memory", "m0");
}
__device__ __forceinline__ void lds_load4(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dword %1, off" ::"s"(lds), "v"(src)
               : "memory", "m0");
}
// 16-byte store from inline assembly (counted like the loads by the waits).
// A store of more than 8 bytes may read its data registers after the next
// instruction has issued, and the compiler's hazard check does not look
// into inline assembly: without the wait states, a VALU write of those
// registers right after the store (which the compiler is free to place
// there) changes the stored data.
__device__ __forceinline__ void gstore16(void* dst, v4f v) {
  asm volatile("global_store_dwordx4 %0, %1, off\n\ts_nop 1" ::"v"(dst), "v"(v) : "memory");
}
// 4-byte and 1-byte stores, the same way.
__device__ __forceinline__ void gstore4(void* dst, uint32_t v) {
  asm volatile("global_store_dword %0, %1, off" ::"v"(dst), "v"(v) : "memory");
}
__device__ __forceinline__ void gstore1(void* dst, uint32_t v) {
  asm volatile("global_store_byte %0, %1, off" ::"v"(dst), "v"(v) : "memory");
}
// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void vm_wait_n() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void vm_wait0() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ v4f mfma4(float a, float b, v4f c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// Lane l's accumulator D[4(l/16)+j][l%16] handed over so that lane l holds
// D[4(l%4)+j][l/4] (four consecutive output channels of one row).
__device__ __forceinline__ v4f store_order(v4f d, int lane) {
  const int src = (((lane & 3) << 4) + (lane >> 2)) << 2;
  v4f r;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    r[j] = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(d[j])));
  return r;
}

// Slot of position (px, py, pz) in {0..3}^3 (relative to the first child of
// group gg minus one) in the group's 64-slot tile: 16 px + 4 py + pz, or with
// SWZ the z bits XOR-ed with (2 gg + (px & 1)).  The forward's reads take one
// channel of one tap for the 16 octants of two groups at a time; unswizzled,
// the two x-values of the eight children and the two groups fall on the same
// banks (4-way conflicts), swizzled on different ones (2-way).
template <bool SWZ>
__device__ __forceinline__ int tile_slot(int gg, int px, int py, int pz) {
  return 16 * px + 4 * py + (SWZ ? pz ^ (2 * gg + (px & 1)) : pz);
}

// Byte offset, in a tile buffer of two groups x 64 positions x 16 bytes, of
// channel c of the tap (dx, dy, dz) in {0,1,2}^3 (offsets -1..1) of child
// ch (4x + 2y + z) of group gg.
template <bool SWZ>
__device__ __forceinline__ int tap_offset(int gg, int ch, int tap, int c) {
  const int px = ((ch >> 2) & 1) + tap / 9, py = ((ch >> 1) & 1) + (tap / 3) % 3,
            pz = (ch & 1) + tap % 3;
  return ((gg * 64 + tile_slot<SWZ>(gg, px, py, pz)) * 16) + 4 * c;
}

// One tile: the two groups' 64 positions each (DMA, one instruction per
// group) from the neighbour entries in nbs (54 entries, LDS).  Lane i fills
// slot i of each group: the position tile_slot<SWZ> puts there.
template <int CIN, bool SWZ>
__device__ __forceinline__ void tile_dma(const float* __restrict__ x, const int32_t* nbs,
                                         float* buf, int lane) {
  const int px = lane >> 4, py = (lane >> 2) & 3;
#pragma unroll
  for (int gg = 0; gg < 2; ++gg) {
    const int pz = SWZ ? (lane & 3) ^ (2 * gg + (px & 1)) : lane & 3;  // tile_slot inverted
    const int ux = px - 1, uy = py - 1, uz = pz - 1;
    const int slot = ((ux >> 1) + 1) * 9 + ((uy >> 1) + 1) * 3 + ((uz >> 1) + 1);
    const int coff = 4 * (ux & 1) + 2 * (uy & 1) + (uz & 1);
    const int32_t b = nbs[27 * gg + slot];
    const float* src = b >= 0 ? x + (int64_t)(b + coff) * CIN : g_cin_zero;
    const uint32_t a = lds_addr(buf + gg * 64 * 4);
    if constexpr (CIN == 4)
      lds_load16(src, a);
    else
      lds_load12(src, a);
  }
}

// The neighbour entries of tile tl (groups 2 tl, 2 tl + 1): 54 entries into
// nbs, one instruction; entries of groups past the last read -1.  With prow
// (the pooled forward), lanes 54 and 55 bring the two groups' output rows of
// depth l-1 in the same instruction.
__device__ __forceinline__ void nb_dma(const int32_t* __restrict__ nbr, int64_t ngroups,
                                       int64_t tl, int32_t* nbs, int lane,
                                       const int32_t* __restrict__ prow = nullptr) {
  const int64_t g = 2 * tl + (lane < 54 ? lane / 27 : lane - 54);
  const int32_t* src = lane < 54 && g < ngroups            ? nbr + 27 * (2 * tl) + lane
                       : prow && lane < 56 && g < ngroups ? prow + g
                                                          : &g_cin_absent;
  lds_load4(src, lds_addr(nbs));
}

// Tiles [t0, t1) of this wave, ntiles in all.  Workgroups are dealt to the
// eight XCDs round-robin (workgroup b runs on XCD b % 8) and each XCD has its
// own L2, so the workgroups of one XCD take one contiguous run of tiles
// (neighbouring tiles share rows of their union tiles).  The grid is a
// multiple of eight workgroups.
__device__ __forceinline__ void wave_range(int64_t ntiles, int wave, int64_t& t0, int64_t& t1) {
  const int64_t per = gridDim.x / 8;
  const int64_t lw = ((int64_t)(blockIdx.x % 8) * per + blockIdx.x / 8) * NWAVE + wave;
  const int64_t nw = (int64_t)gridDim.x * NWAVE;
  t0 = ntiles * lw / nw;
  t1 = ntiles * (lw + 1) / nw;
}

// Forward: y [8 ngroups][cout] = conv(x [8 ngroups][CIN], w [27][CIN][cout]),
// relu != 0 applies max(0, .).  Grid: x = workgroups (each wave a range of
// tiles), y = blocks of 16 output channels.  The MFMA computes y^T: A = W^T
// (16 output channels x 4 pairs k), B = the gathered rows (4 pairs x 16
// octants).
// POOL: the 2x2x2 max-pool follows in the epilogue; y is then the pooled
// map [npar][cout] of depth l-1 (row prow[g] for group g, brought with the
// neighbour entries), psw the switches [ngroups][cout]; a tile then issues
// two stores (values, switches), which the counted waits include; the waves
// of column block 0 zero an equal share of the rows of empty depth-(l-1)
// octants after their last wait.
template <int CIN, bool POOL>
__global__ __launch_bounds__(TB) void k_cin_fwd(const int32_t* __restrict__ nbr, int64_t ngroups,
                                                const float* __restrict__ x,
                                                const float* __restrict__ w, int cout,
                                                float* __restrict__ y, int relu,
                                                const int32_t* __restrict__ prow,
                                                const int32_t* __restrict__ plab, int64_t npar,
                                                uint8_t* __restrict__ psw) {
  constexpr int KF = 27 * CIN, NS = (KF + 3) / 4;
  constexpr int TF = 2 * 64 * 4;  // floats of a tile buffer
  constexpr int S = POOL ? 2 : 1;  // stores per tile
  constexpr int WE = 3 + S;        // operations younger than a tile's entries at their wait
  __shared__ __attribute__((aligned(16))) float tiles[NWAVE][NBUF][TF];
  __shared__ __attribute__((aligned(16))) int32_t nbs[NWAVE][2][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int li = lane & 15, q = lane >> 4;
  const int n0 = blockIdx.y * 16;
  int64_t t0, t1;
  wave_range((ngroups + 1) / 2, wave, t0, t1);
  // rows of empty depth-(l-1) octants (pooled forward): a share per wave
  auto zero_share = [&]() {
    if constexpr (POOL) {
      if (blockIdx.y != 0) return;
      const int64_t per = gridDim.x / 8;
      const int64_t lw = ((int64_t)(blockIdx.x % 8) * per + blockIdx.x / 8) * NWAVE + wave;
      const int64_t nwv = (int64_t)gridDim.x * NWAVE;
      const int64_t r0 = npar * lw / nwv, r1 = npar * (lw + 1) / nwv;
      const int c4 = cout / 4, cnt = (int)(r1 - r0) * c4;
      for (int e = lane; e < cnt; e += 64) {
        const int64_t i = r0 + e / c4;
        if (plab[i] == 0)
          *reinterpret_cast<v4f*>(y + i * cout + 4 * (e % c4)) = v4f{0.f, 0.f, 0.f, 0.f};
      }
    }
  };
  if (t0 >= t1) {  // wave-uniform; nothing issued yet
    zero_share();
    return;
  }
  float* tw = &tiles[wave][0][0];
  int32_t* nw = &nbs[wave][0][0];
  const int32_t* pr = POOL ? prow : nullptr;
  nb_dma(nbr, ngroups, t0, nw, lane, pr);  // its latency overlaps the weight loads

  // lane (li, q): weight W[k][n0 + li] and row li's tile offset of pair
  // k = 4 s + q (pairs past KF: weight 0, any finite position)
  float wr[NS];
  int xo[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    const int k = 4 * s + q;
    const bool on = k < KF;
    wr[s] = on ? w[(int64_t)k * cout + n0 + li] : 0.f;
    xo[s] = tap_offset<true>(li >> 3, li & 7, on ? k / CIN : 0, on ? k % CIN : 0);
  }
  // the weights are in registers here (the compiler waits for their loads,
  // and for the entries above), so the counted waits below see only the
  // DMAs and stores; xo: one register each
#pragma unroll
  for (int s = 0; s < NS; ++s) asm volatile("" : "+v"(wr[s]), "+v"(xo[s]));

  // Per tile t: entries of tile t+D+1, then tile t+D (once its entries are
  // in), then the MFMAs of tile t (once it is in) and its store.  The
  // prologue runs the first D of those steps with dummy stores, so that
  // every wait counts the same younger operations: 4 for entries (tile,
  // store, entries), 4 D for a tile.
  // pooled forward: the output row of this lane's group for tiles t .. t+D
  // (read from the entries while they are valid, then shifted along)
  int32_t pq[D + 1];
#pragma unroll
  for (int j = 0; j <= D; ++j) pq[j] = -1;
#pragma unroll
  for (int j = 0; j < D; ++j) {
    nb_dma(nbr, ngroups, t0 + j + 1, nw + 64 * ((j + 1) & 1), lane, pr);
    if (j == 0)
      vm_wait_n<1>();
    else
      vm_wait_n<WE>();
    if constexpr (POOL) pq[j] = nw[64 * (j & 1) + 54 + ((lane >> 4) & 1)];
    tile_dma<CIN, true>(x, nw + 64 * (j & 1), tw + j * TF, lane);
    if constexpr (POOL) {
      gstore4(g_cin_dummy + lane, 0u);
      gstore1(reinterpret_cast<uint8_t*>(g_cin_dummy) + lane, 0u);
    } else {
      gstore16(g_cin_dummy + 4 * lane, v4f{0.f, 0.f, 0.f, 0.f});
    }
  }
  int cur = 0;  // buffer of tile t
  for (int64_t t = t0; t < t1; ++t) {
    const int ahead = (cur + D) % NBUF;  // buffer of tile t+D
    const int e = (int)((t - t0) & 1);   // entry slot of tile t (tile u: slot (u - t0) & 1)
    nb_dma(nbr, ngroups, t + D + 1, nw + 64 * ((e + D + 1) & 1), lane, pr);
    vm_wait_n<WE>();  // entries of tile t+D
    if constexpr (POOL) pq[D] = nw[64 * ((e + D) & 1) + 54 + ((lane >> 4) & 1)];
    tile_dma<CIN, true>(x, nw + 64 * ((e + D) & 1), tw + ahead * TF, lane);
    vm_wait_n<WE * D>();  // tile t
    v4f acc = {0.f, 0.f, 0.f, 0.f};
    const float* bb = tw + cur * TF;
    float xv[NS];  // every read issued before the MFMAs
#pragma unroll
    for (int s = 0; s < NS; ++s) xv[s] = lds_at(bb, xo[s]);
#pragma unroll
    for (int s = 0; s < NS; ++s) acc = mfma4(wr[s], xv[s], acc);
    if (relu) {
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] = fmaxf(acc[j], 0.f);
    }
    if constexpr (POOL) {
      // through LDS (tile t's buffer: its MFMA operands have been read, and
      // tile t+NBUF is loaded into it only in the next iteration): lane o
      // pools group 2t + (o/16)%2 in channel n0 + o%16; lanes 32-63 repeat
      // lanes 0-31 (same address, same data: no lane goes to the dummy row,
      // which every wave of the grid would hit)
      float* ps = tw + cur * TF;
      oc::pool_put(ps, acc, lane);
      uint32_t sw;
      const float m = oc::pool_scan(ps, lane, sw);
      const int64_t g = 2 * t + ((lane >> 4) & 1);
      const bool st = g < ngroups && pq[0] >= 0;
      const int c = n0 + (lane & 15);
      gstore4(st ? (void*)(y + (int64_t)pq[0] * cout + c) : (void*)(g_cin_dummy + lane),
              __float_as_uint(m));
      gstore1(st ? (void*)(psw + g * cout + c)
                 : (void*)(reinterpret_cast<uint8_t*>(g_cin_dummy) + lane),
              sw);
#pragma unroll
      for (int j = 0; j < D; ++j) pq[j] = pq[j + 1];
    } else {
      // lane l: row l / 4 of the tile, channels n0 + 4 (l % 4) ..
      acc = store_order(acc, lane);
      const int64_t row = 16 * t + (lane >> 2);
      float* dst =
          row < 8 * ngroups ? y + row * cout + n0 + 4 * (lane & 3) : g_cin_dummy + 4 * lane;
      gstore16(dst, acc);
    }
    cur = cur + 1 == NBUF ? 0 : cur + 1;
  }
  vm_wait0();  // no DMA into LDS outlives the workgroup
  zero_share();
}

// Weight gradient: part[blockIdx.x][k][n0 + j] = sum over the workgroup's
// octants i of x[nb(i, tap)][c] dy[i][n0 + j] for pair k = CIN tap + c.
// M = 16 pairs per block (NMB blocks), N = 16 output channels, the reduction
// over octants four per MFMA step (children 4u'..4u'+3 of a group).  The
// tile's dY rows (16 x 16 channels) are DMA'd with it.  The four waves'
// sums are added in wave order through LDS.
template <int CIN>
__global__ __launch_bounds__(TB) void k_cin_dw(const int32_t* __restrict__ nbr, int64_t ngroups,
                                               const float* __restrict__ x,
                                               const float* __restrict__ dy, int cout,
                                               float* __restrict__ part) {
  constexpr int KF = 27 * CIN, NMB = (KF + 15) / 16;
  constexpr int TF = 2 * 64 * 4;  // floats of a tile's x positions
  constexpr int YF = 16 * 16;     // floats of its dY rows
  constexpr int BF = TF + YF;     // floats of a tile buffer
  __shared__ __attribute__((aligned(16))) float tiles[NWAVE][NBUF][BF];
  __shared__ __attribute__((aligned(16))) int32_t nbs[NWAVE][2][64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int li = lane & 15, q = lane >> 4;
  const int n0 = blockIdx.y * 16;
  int64_t t0, t1;
  wave_range((ngroups + 1) / 2, wave, t0, t1);

  // lane (li, q) in step u (rows 4u..4u+3 of the tile: group u / 2, children
  // 4 (u & 1) + q) of block b supplies x of pair k = 16 b + li
  int xo[NMB][4];
#pragma unroll
  for (int b = 0; b < NMB; ++b) {
    const int k = 16 * b + li;
    const bool on = k < KF;
#pragma unroll
    for (int u = 0; u < 4; ++u)
      xo[b][u] = tap_offset<false>(u >> 1, 4 * (u & 1) + q, on ? k / CIN : 0, on ? k % CIN : 0);
  }
#pragma unroll
  for (int b = 0; b < NMB; ++b)
#pragma unroll
    for (int u = 0; u < 4; ++u) asm volatile("" : "+v"(xo[b][u]));  // one register each
  bool kon[NMB];
#pragma unroll
  for (int b = 0; b < NMB; ++b) kon[b] = 16 * b + li < KF;
  v4f acc[NMB];
#pragma unroll
  for (int b = 0; b < NMB; ++b) acc[b] = v4f{0.f, 0.f, 0.f, 0.f};

  float* tw = &tiles[wave][0][0];
  int32_t* nw = &nbs[wave][0][0];
  // dY rows of tile tl: lane l takes row l / 4, columns n0 + 4 (l % 4)..
  auto dy_dma = [&](int64_t tl, float* buf) {
    const int64_t row = 16 * tl + (lane >> 2);
    const float* src =
        row < 8 * ngroups ? dy + row * cout + n0 + 4 * (lane & 3) : g_cin_zero;
    lds_load16(src, lds_addr(buf));
  };

  if (t0 < t1) {  // wave-uniform
    // as in the forward, without stores: entries of tile t+D+1, then tile
    // t+D (x positions and dY rows), then the MFMAs of tile t; every wait
    // counts 4 younger operations (tile 3, entries 1)
    nb_dma(nbr, ngroups, t0, nw, lane);
#pragma unroll
    for (int j = 0; j < D; ++j) {
      nb_dma(nbr, ngroups, t0 + j + 1, nw + 64 * ((j + 1) & 1), lane);
      if (j == 0)
        vm_wait_n<1>();
      else
        vm_wait_n<4>();
      tile_dma<CIN, false>(x, nw + 64 * (j & 1), tw + j * BF, lane);
      dy_dma(t0 + j, tw + j * BF + TF);
    }
    int cur = 0;  // buffer of tile t
    for (int64_t t = t0; t < t1; ++t) {
      const int ahead = (cur + D) % NBUF;  // buffer of tile t+D
      const int e = (int)((t - t0) & 1);   // entry slot of tile t (tile u: slot (u - t0) & 1)
      nb_dma(nbr, ngroups, t + D + 1, nw + 64 * ((e + D + 1) & 1), lane);
      vm_wait_n<4>();  // entries of tile t+D
      tile_dma<CIN, false>(x, nw + 64 * ((e + D) & 1), tw + ahead * BF, lane);
      dy_dma(t + D, tw + ahead * BF + TF);
      vm_wait_n<4 * D>();  // tile t
      const float* bb = tw + cur * BF;
      // every read of the tile issued before its MFMAs
      float bv[4], av[4][NMB];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        bv[u] = lds_at(bb, (TF + (4 * u + q) * 16 + li) * 4);  // dY[row 4u + q][n0 + li]
#pragma unroll
        for (int b = 0; b < NMB; ++b) av[u][b] = lds_at(bb, xo[b][u]);
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int b = 0; b < NMB; ++b) acc[b] = mfma4(kon[b] ? av[u][b] : 0.f, bv[u], acc[b]);
      cur = cur + 1 == NBUF ? 0 : cur + 1;
    }
    vm_wait0();  // no DMA into LDS outlives the loop
  }

  // the waves' sums in wave order: wave w adds its own to the running sum
  // left by wave w-1 (LDS reuse of the tile buffers after a barrier)
  __syncthreads();
  v4f* red = reinterpret_cast<v4f*>(&tiles[0][0][0]);  // NMB x 64 v4f
  static_assert(NMB * 64 * 4 <= NWAVE * NBUF * BF, "reduction fits the tile buffers");
  for (int w = 0; w < NWAVE; ++w) {
    if (wave == w) {
#pragma unroll
      for (int b = 0; b < NMB; ++b) {
        v4f v = acc[b];
        if (w > 0) v = red[b * 64 + lane] + v;
        red[b * 64 + lane] = v;
      }
    }
    __syncthreads();
  }
  // lane l of block b holds pairs k = 16 b + 4 (l / 16) + j, column n0 + l % 16
  if (wave == 0) {
    float* pp = part + (int64_t)blockIdx.x * KF * cout;
#pragma unroll
    for (int b = 0; b < NMB; ++b) {
      const v4f v = red[b * 64 + lane];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int k = 16 * b + 4 * q + j;
        if (k < KF) pp[(int64_t)k * cout + n0 + li] = v[j];
      }
    }
  }
}

// Resident workgroups per CU of a kernel (at least 1).
template <typename F>
int occupancy(F kernel) {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, TB, 0) != hipSuccess || n < 1)
    n = 1;
  return n;
}

// Workgroups of a launch over G groups: every resident slot of the GPU
// (divided among the column blocks), about one tile per wave at least, a
// multiple of eight (the XCD-wise ranges).
int64_t workgroups(int64_t G, int slots_per_cu, int ncb) {
  const int64_t slots = (int64_t)oc::cu_count() * slots_per_cu;
  const int64_t tiles = std::max<int64_t>(1, (G + 1) / 2);
  const int64_t n = std::max<int64_t>(1, std::min<int64_t>(slots / ncb, oc::cdiv(tiles, NWAVE)));
  return 8 * oc::cdiv(n, 8);
}

// The weight gradient keeps at most three workgroups per CU (as many as its
// LDS allows): each one writes a partial sum of every entry (27 Cin Cout
// floats), so more would add little latency hiding for more to add.
template <int CIN>
int64_t dw_workgroups(int64_t G, int cout) {
  static const int occ = std::min(3, occupancy(k_cin_dw<CIN>));
  return workgroups(G, occ, cout / 16);
}

}  // namespace

namespace oc {

bool conv_cin_supported(int K, int cin, int cout) {
  return K == 3 && (cin == 3 || cin == 4) && cout % 16 == 0 && cout > 0;
}

template <int CIN, bool POOL>
void launch_cin_fwd(const oc_octree* t, int l, const float* x, const float* w, int cout, float* y,
                    int relu, uint8_t* sw, hipStream_t s) {
  const int64_t G = t->M[l - 1];
  const int ncb = cout / 16;
  static const int occ = occupancy(k_cin_fwd<CIN, POOL>);
  const dim3 grid((unsigned)workgroups(G, occ, ncb), (unsigned)ncb);
  launch_main(k_cin_fwd<CIN, POOL>, grid, dim3(TB), s, (const int32_t*)t->nbr[l], G, x, w, cout,
              y, relu, POOL ? (const int32_t*)t->rows[l - 1] : nullptr,
              POOL ? (const int32_t*)t->labels[l - 1] : nullptr, POOL ? t->N[l - 1] : 0, sw);
}

void conv_cin_fwd(const oc_octree* t, int l, const float* x, int cin, const float* w, int cout,
                  float* y, int relu, hipStream_t s) {
  if (t->M[l - 1] <= 0) return;
  if (cin == 3)
    launch_cin_fwd<3, false>(t, l, x, w, cout, y, relu, nullptr, s);
  else
    launch_cin_fwd<4, false>(t, l, x, w, cout, y, relu, nullptr, s);
}

void conv_cin_pool_fwd(const oc_octree* t, int l, const float* x, int cin, const float* w,
                       int cout, float* yp, uint8_t* sw, int relu, hipStream_t s) {
  if (t->N[l - 1] <= 0) return;
  // with no non-empty depth-(l-1) octant the kernel still zeroes every row
  if (cin == 3)
    launch_cin_fwd<3, true>(t, l, x, w, cout, yp, relu, sw, s);
  else
    launch_cin_fwd<4, true>(t, l, x, w, cout, yp, relu, sw, s);
}

size_t conv_cin_dw_parts(const oc_octree* t, int l, int cin, int cout) {
  const int64_t G = t->M[l - 1];
  return (size_t)(cin == 3 ? dw_workgroups<3>(G, cout) : dw_workgroups<4>(G, cout));
}

void conv_cin_dw(const oc_octree* t, int l, const float* x, int cin, const float* dy, int cout,
                 float* dw, float* part, hipStream_t s, bool defer) {
  const int64_t G = t->M[l - 1];
  const int64_t entries = (int64_t)27 * cin * cout;
  const int64_t np = (int64_t)conv_cin_dw_parts(t, l, cin, cout);
  const dim3 grid((unsigned)np, (unsigned)(cout / 16));
  if (cin == 3)
    launch_main(k_cin_dw<3>, grid, dim3(TB), s, (const int32_t*)t->nbr[l], G, x, dy, cout, part);
  else
    launch_main(k_cin_dw<4>, grid, dim3(TB), s, (const int32_t*)t->nbr[l], G, x, dy, cout, part);
  if (!defer) sum_partials(part, (int)np, entries, dw, s);
}

void conv_cin_kernel_name(int cin, int pass, char* buf, size_t n) {
  if (pass == 2)
    snprintf(buf, n, "k_cin_dw<%d>", cin);
  else
    snprintf(buf, n, "k_cin_fwd<%d, %s>", cin, pass == 3 ? "true" : "false");
}

}  // namespace oc
