/*
 * oc.h -- C ABI of the MI355X (gfx950) octree-CNN hot path.
 *
 * Implements the GPU side of O-CNN (Wang et al., "O-CNN: Octree-based
 * Convolutional Neural Networks for 3D Shape Analysis", arXiv 1712.01537):
 * building the per-depth packed super-octree of a batch of oriented point
 * clouds (Sec. 3.1), and convolution, deconvolution, max-pooling,
 * max-unpooling and general pooling restricted to the octants of that
 * octree (Sec. 3.2).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Depth l has N_l octants (every child of a non-empty depth-(l-1) octant,
 *    empty or not; N_0 = batch) of which M_l are non-empty.  N_l = 8 M_{l-1}.
 *  - Feature maps are row-major [N_l][C] (one row per octant, in key order,
 *    channels contiguous), fp32 unless a dtype argument says otherwise.
 *  - Convolution weights are [K^3][Cin][Cout], fp32 (or bf16 for OC_BF16),
 *    tap index k = ((dx+r)K + (dy+r))K + (dz+r) with r = (K-1)/2 and
 *    (dx,dy,dz) the neighbour's offset; x varies slowest, matching the bit
 *    order of the shuffle key.  The operation is a cross-correlation with no
 *    bias; a neighbour that is not in the octree reads as zero (Sec. 3.2,
 *    unrolled convolution).
 *  - Every pointer named "dev" is device memory of the current HIP device;
 *    "host" pointers are host memory.  The caller owns every buffer it passes;
 *    the library never frees them.  Buffers must not alias unless stated.
 *  - Every call enqueues work on `stream` and returns without waiting, except
 *    oc_build and oc_build_finish, which wait exactly once (to read the
 *    per-depth counts), and oc_build_cancel.
 *  - Argument errors are detected before any work is enqueued and returned
 *    as a status; nothing is written in that case.  Asynchronous device
 *    faults surface as OC_ERR_DEVICE from a later call.  oc_last_error()
 *    gives a message for the calling thread's last failure.  No C++
 *    exception crosses this interface.
 *  - An octree is immutable after oc_build; calls on different streams may
 *    use it concurrently.
 */
#ifndef OC_H_
#define OC_H_

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  OC_OK = 0,
  OC_ERR_ARG = 1,          /* invalid argument, null pointer, shape mismatch */
  OC_ERR_RANGE = 2,        /* a point outside [0,1]^3 or NaN */
  OC_ERR_NOMEM = 3,        /* the allocator returned NULL */
  OC_ERR_DEVICE = 4,       /* a HIP runtime error */
  OC_ERR_UNSUPPORTED = 5   /* valid but not implemented (e.g. kernel size) */
} oc_status;

typedef enum { OC_F32 = 0, OC_BF16 = 1 } oc_dtype;

/* oc_conv_fwd / oc_conv_bwd flag: y = max(0, conv(x)); the backward then
 * masks dy with [y > 0] (Sec. 4, ReLU after each convolution). */
#define OC_FUSE_RELU 1

/* oc_conv_bwd flag: leave the weight gradient as its partial sums in the
 * workspace instead of adding them into dw, so that one oc_sum_partials
 * launch can add those of several layers (dw is then written by that call;
 * the workspace must stay untouched until it has run).  Layers whose weight
 * gradient has no deferred form still write dw; oc_conv_dw_partials tells
 * which, and where the partial sums are. */
#define OC_DEFER_DW 2

/* Device memory provider for the octree's arrays and oc_build's temporaries.
 * alloc returns device memory usable in stream order on `stream` (NULL on
 * failure); free releases it in stream order.  Pass NULL to oc_build to use
 * hipMalloc/hipFree. */
typedef struct oc_allocator {
  void* (*alloc)(void* ctx, size_t bytes, hipStream_t stream);
  void (*free)(void* ctx, void* ptr, hipStream_t stream);
  void* ctx;
} oc_allocator;

typedef struct oc_octree oc_octree; /* opaque, immutable after oc_build */

/* Per-depth arrays of a built octree (Sec. 3.1), all dev, owned by the octree.
 *   keys          [N_l]  shuffle key x1y1z1...xlylzl of each octant with the
 *                        shape index in bits 24..31 (super-octree key,
 *                        Sec. 3.1 "Mini-batch"); ascending.
 *   labels        [N_l]  0 for an empty octant, p for the p-th non-empty one
 *                        of the whole batch (1-based, Sec. 3.1 "Label").
 *   rows_of_label [M_l]  inverse of labels: the row holding label p at p-1.
 *   nbr           [M_{l-1}][27] (NULL at l = 0): for sibling group g (the
 *                        children of the g-th non-empty octant of depth l-1),
 *                        and parent offset o = (ox+1)*9 + (oy+1)*3 + (oz+1)
 *                        with ox,oy,oz in {-1,0,1}, the first-child row
 *                        8(label-1) at depth l of the depth-(l-1) octant at
 *                        that offset from the group's parent, or -1 if that
 *                        octant is outside the cube, empty or absent.  Every
 *                        neighbour of every octant of the group within
 *                        offset +-2 per axis is reachable from these 27
 *                        entries (the shared neighbourhood of the eight
 *                        siblings, Sec. 3.2 and Fig. 4). */
typedef struct oc_level {
  int32_t depth;
  int64_t num_octants;  /* N_l */
  int64_t num_nonempty; /* M_l */
  const uint32_t* keys;
  const int32_t* labels;
  const int32_t* rows_of_label;
  const int32_t* nbr;
} oc_level;

/* Build the super-octree of `batch` shapes (Sec. 3.1).
 *   points       dev f32 [P][3], every coordinate in [0,1] (else
 *                OC_ERR_RANGE); shape b owns points
 *                shape_offsets[b] .. shape_offsets[b+1]-1.
 *   normals      dev f32 [P][3], finite (else OC_ERR_RANGE), averaged per
 *                non-empty leaf into the input signal (Sec. 3.1 "Input
 *                signal"); the sums are kept in 64-bit fixed point with a
 *                step of 2^-62 times P times the largest |component|, so
 *                the signal does not depend on the order of the additions.
 *   shape_offsets host i32 [batch+1], non-decreasing, shape_offsets[0] = 0.
 *   batch        1..256 (8-bit shape index in the key).
 *   depth        1..8 (3*depth key bits must fit below the shape byte).
 *   full_depth   0..depth: octants shallower than full_depth are forced
 *                non-empty, so every octant of depth full_depth exists
 *                (Sec. 4 uses 2).
 *   alloc        NULL for hipMalloc/hipFree.
 * Quantisation: cell = min(floor(p * 2^depth), 2^depth - 1) per axis, in fp32.
 * Device scratch of about (8/7) B 8^depth / 4 bytes (occupancy bitmaps and
 * their popcount prefix) plus 32 bytes per point is taken from `alloc` for the
 * duration of the call.
 * On success *out owns its arrays until oc_octree_free.  Waits once on
 * `stream`. */
oc_status oc_build(const float* points, const float* normals, const int32_t* shape_offsets,
                   int32_t batch, int32_t depth, int32_t full_depth, const oc_allocator* alloc,
                   hipStream_t stream, oc_octree** out);

/* The two halves of oc_build, for callers that overlap building the next
 * batch's octree with other work (Sec. 3.2, last paragraph: the paper builds
 * the next batch in a separate thread).  oc_build(..., s, out) is exactly
 * oc_build_async(..., s, &job) followed by oc_build_finish(job, s, out).
 *
 * oc_build_async takes the same arguments as oc_build, checks them, takes
 * the scratch from `alloc` on `stream` and enqueues on `stream` the part of
 * the build that decides the per-depth counts: quantisation, the occupancy
 * bitmaps of every depth and their popcount scan, then a copy of the counts
 * to pinned host memory.  It returns without waiting; *job (host, opaque)
 * owns the scratch until oc_build_finish or oc_build_cancel, and
 * shape_offsets is copied, so the caller may reuse it at once.  points and
 * normals must stay valid until the work of oc_build_finish is done.
 *
 * oc_build_finish waits for the job's counts (the one wait; only the work
 * oc_build_async enqueued is waited for, not what follows it on its stream),
 * allocates the octree from the job's allocator on `stream` (which may differ
 * from the job's stream; it is made to wait for the job's work), enqueues on
 * `stream` the leaf signal and the emission of keys, labels, rows_of_label
 * and nbr, releases the scratch in stream order on `stream`, and returns
 * without waiting for that work.  The octree's arrays are released on
 * `stream` by oc_octree_free.  The job is consumed whatever the status; a
 * point outside [0,1]^3 or a non-finite normal is reported here
 * (OC_ERR_RANGE).
 *
 * oc_build_cancel waits for the job's work and releases the job without
 * building (NULL is ignored). */
typedef struct oc_build_job oc_build_job;
oc_status oc_build_async(const float* points, const float* normals, const int32_t* shape_offsets,
                         int32_t batch, int32_t depth, int32_t full_depth,
                         const oc_allocator* alloc, hipStream_t stream, oc_build_job** job);
oc_status oc_build_finish(oc_build_job* job, hipStream_t stream, oc_octree** out);
void oc_build_cancel(oc_build_job* job);

/* Sizes and device arrays of depth l (0..depth). */
oc_status oc_octree_level(const oc_octree* tree, int32_t l, oc_level* out);

/* Tree depth, full depth and batch size. */
oc_status oc_octree_info(const oc_octree* tree, int32_t* depth, int32_t* full_depth,
                         int32_t* batch);

/* Input signal, dev f32 [N_depth][3]: mean normal of the points in each
 * non-empty leaf, zero for empty leaves (Sec. 3.1 "Input signal"). */
const float* oc_octree_signal(const oc_octree* tree);

/* Release the octree's arrays (in stream order on the build stream). */
void oc_octree_free(oc_octree* tree);

/* Octree convolution forward (Sec. 3.2).
 *   depth   input depth l (1..tree depth).
 *   ksize   3 or 5 (stride 1); 3 (stride 2).
 *   stride  1: output at all N_l octants of depth l.
 *           2: output at depth l-1: the convolution is evaluated at the
 *              first sibling of every group and written to the row of its
 *              parent; rows of empty parents are zero (Sec. 3.2 stride-2
 *              paragraphs, Fig. 2(d)).
 *           2^r, r = 1 .. l: output at depth l-r (Sec. 3.2, stride 2^r):
 *              evaluated at the first depth-l position of the sub-tree of
 *              height r below every non-empty depth-(l-r) octant (2^r times
 *              its coordinates, whether or not an octant is stored there:
 *              the neighbours of that position are read as usual) and
 *              written to that octant's row; rows of empty octants are
 *              zero.  Strided convolutions take ksize 3 only.
 *   dt      OC_F32: x, w fp32.  OC_BF16: x, w bf16 (round-to-nearest-even
 *           values held as uint16); products accumulate in fp32, so the
 *           result is the fp32 convolution of the bf16 values.
 *   x       dev [N_l][cin].      w  dev [K^3][cin][cout].
 *   y       dev f32 [N_out][cout], N_out = N_l, N_{l-1} or N_{l-2}.
 *   ws      dev workspace of at least oc_conv_fwd_workspace() bytes (may be
 *           NULL when that is 0): partial sums of a reduction split across
 *           workgroups, added in a fixed order (results are reproducible);
 *           for OC_BF16 shapes the bf16 matrix-core kernels do not take
 *           (strided; channel counts not multiples of 16; rows of x or of
 *           the output gradient spanning 2 GiB or more), x and w widened to
 *           fp32; when strided, each output's eight
 *           source-group rows (32 bytes per output) and w transposed.
 *   flags   0 or OC_FUSE_RELU.
 * cin, cout in 1..1024. */
oc_status oc_conv_fwd(const oc_octree* tree, int32_t depth, int32_t ksize, int32_t stride,
                      oc_dtype dt, const void* x, int32_t cin, const void* w, int32_t cout,
                      float* y, void* ws, size_t ws_bytes, int32_t flags, hipStream_t stream);

/* Convolution, ReLU and 2x2x2 max-pooling forward in one call (the unit of
 * Sec. 4's network structure without its normalisation; operations of
 * Sec. 3.2): the stride-1 convolution at depth l, max(0, .) when flags has
 * OC_FUSE_RELU, then oc_pool_fwd's pooling to depth l-1.  Where the kernel
 * pools in its epilogue (fp32; K = 3 with cin 3 or 4 and cout a multiple of
 * 16, or cin and cout multiples of 4 with cin >= 16) the depth-l output is
 * never written to memory.
 *   depth   l, 1 .. tree depth; ksize 3 or 5; dt, x, cin, w, cout, flags
 *           as oc_conv_fwd with stride 1.
 *   y       dev f32 [N_{l-1}][cout], 16-byte aligned: the pooled features;
 *           rows of empty octants are zero.
 *   sw      dev u8 [M_{l-1}][cout], 4-byte aligned: the switches, as
 *           oc_pool_fwd (the first maximum over children 0..7).
 *   ws      dev workspace of oc_conv_pool_fwd_workspace() bytes (may be NULL
 *           when that is 0).
 * y and sw equal, bit for bit, oc_conv_fwd followed by oc_pool_fwd.  The
 * backward is oc_pool_bwd with y (which applies the ReLU's backward), then
 * oc_conv_bwd without OC_FUSE_RELU. */
size_t oc_conv_pool_fwd_workspace(const oc_octree* tree, int32_t depth, int32_t ksize,
                                  oc_dtype dt, int32_t cin, int32_t cout);
oc_status oc_conv_pool_fwd(const oc_octree* tree, int32_t depth, int32_t ksize, oc_dtype dt,
                           const void* x, int32_t cin, const void* w, int32_t cout, float* y,
                           uint8_t* sw, void* ws, size_t ws_bytes, int32_t flags,
                           hipStream_t stream);

/* oc_conv_fwd without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation): the workspace is a static device array of the
 * library, 32 MiB per device, held from the first call on a device until the
 * process ends; the call allocates nothing.  Arguments as oc_conv_fwd.
 * Returns OC_ERR_UNSUPPORTED when the call would need more workspace than
 * 32 MiB (oc_conv_fwd_workspace tells) and for strides other than 1.
 * Results are identical, bit for bit, to oc_conv_fwd's.  Every call on a
 * device shares that device's array: calls that overlap on one device (other
 * streams, other threads) race and must be ordered by the caller. */
oc_status oc_conv_fwd_noalloc(const oc_octree* tree, int32_t depth, int32_t ksize, int32_t stride,
                              oc_dtype dt, const void* x, int32_t cin, const void* w,
                              int32_t cout, float* y, int32_t flags, hipStream_t stream);

/* Name, template arguments included (as profilers such as rocprofv3 print
 * it), of the kernel that does the arithmetic of one pass of a convolution
 * call with these arguments: pass 0 = oc_conv_fwd, 1 = the input gradient and
 * 2 = the weight gradient of oc_conv_bwd, 3 = the convolution kernel of
 * oc_conv_pool_fwd (stride 1 only).  Lets a caller attribute measured
 * kernel time to the operation it belongs to.  The string lives in
 * thread-local storage until the next call on the thread; "" (and
 * oc_last_error set) for invalid arguments. */
const char* oc_conv_kernel(const oc_octree* tree, int32_t depth, int32_t ksize, int32_t stride,
                           oc_dtype dt, int32_t cin, int32_t cout, int32_t pass);

/* Bytes of device workspace oc_conv_fwd needs for these arguments. */
size_t oc_conv_fwd_workspace(const oc_octree* tree, int32_t depth, int32_t ksize, int32_t stride,
                             oc_dtype dt, int32_t cin, int32_t cout);

/* Bytes of device workspace oc_conv_bwd needs for these arguments (with or
 * without OC_FUSE_RELU). */
size_t oc_conv_bwd_workspace(const oc_octree* tree, int32_t depth, int32_t ksize, int32_t stride,
                             oc_dtype dt, int32_t cin, int32_t cout);

/* Octree convolution backward (Sec. 3.2; the transposed products of the
 * forward).  Arguments as oc_conv_fwd, plus
 *   y    dev f32 [N_out][cout], the forward output, read only when flags has
 *        OC_FUSE_RELU (then dy is masked with [y > 0]); may be NULL otherwise.
 *   dy   dev f32 [N_out][cout] upstream gradient.  OC_BF16: the
 *        matrix-core operand is dy (after the ReLU mask) rounded to bf16,
 *        nearest-even; dx and dw are the fp32-accumulated products of those
 *        bf16 values with the bf16 w and x.
 *   dx   dev f32 [N_l][cin] or NULL: gradient w.r.t. x (overwritten).
 *   dw   dev f32 [K^3][cin][cout] or NULL: gradient w.r.t. w (overwritten).
 *   ws   dev workspace of at least oc_conv_bwd_workspace() bytes.
 *   flags   0, OC_FUSE_RELU, OC_DEFER_DW or both.
 * Deterministic: no floating-point atomics; repeated calls give identical
 * bits.  The strided workspace holds each output's eight source-group rows,
 * the upstream gradient gathered at the evaluated outputs and the weight
 * gradient's partial sums over ranges of outputs. */
oc_status oc_conv_bwd(const oc_octree* tree, int32_t depth, int32_t ksize, int32_t stride,
                      oc_dtype dt, const void* x, int32_t cin, const void* w, int32_t cout,
                      const float* y, const float* dy, float* dx, float* dw, void* ws,
                      size_t ws_bytes, int32_t flags, hipStream_t stream);

/* Where oc_conv_bwd with OC_DEFER_DW leaves the weight gradient of these
 * arguments (the same as oc_conv_bwd's): *nparts partial sums of *count =
 * K^3 cin cout floats each, one after another at byte *offset of its
 * workspace (256-byte aligned); dw = their sum in index order, which
 * oc_sum_partials forms.  *nparts = 0: the layer writes dw itself (strided,
 * bf16 on the bf16 kernels, or no octants).  The first layer's and the
 * matrix-core kernels' reductions over ranges of groups (the transposed
 * products of Sec. 3.2) are what is deferred. */
oc_status oc_conv_dw_partials(const oc_octree* tree, int32_t depth, int32_t ksize, int32_t stride,
                              oc_dtype dt, int32_t cin, int32_t cout, size_t* offset,
                              int32_t* nparts, int64_t* count);

/* outs[i][e] = sum over p < nparts[i] of parts[i][p counts[i] + e], for every
 * set i < n, in one launch per eight sets whose buffers are 16-byte aligned
 * and whose counts are multiples of 4 (others alone).  Each entry gets its
 * terms in the same fixed order as inside oc_conv_bwd, so the bits equal a
 * call without OC_DEFER_DW.  Host arrays of device pointers; outs may not
 * overlap parts.  OC_ERR_ARG for n < 0, NULL arrays, nparts < 1 or
 * counts < 0. */
oc_status oc_sum_partials(int32_t n, const float* const* parts, const int32_t* nparts,
                          const int64_t* counts, float* const* outs, hipStream_t stream);

/* y[e] = x[e] rounded to bf16 (nearest, ties to even; NaN stays NaN), for
 * e < n: the operand of an OC_BF16 layer that follows a layer with f32
 * output (oc_conv_fwd always writes f32).  x dev f32 [n], y dev u16 [n]
 * (the bf16 bit patterns), not overlapping; 16-byte aligned buffers
 * take vector accesses.  OC_ERR_ARG for n < 0 or a NULL buffer (n > 0). */
oc_status oc_round_bf16(int64_t n, const float* x, uint16_t* y, hipStream_t stream);

/* The input gradient of a stride-1 fp32 convolution whose input x is the
 * output of a 2x2x2 max-pooling from depth l+1, carried on through that
 * pooling's backward (Sec. 3.2 "Pooling" and the transposed products of the
 * convolution): oc_conv_bwd's input gradient followed by oc_pool_bwd, in one
 * call that never stores the depth-l gradient (the partial sums of its
 * split reduction go straight into the routing).
 *   depth   l, the convolution's depth (depth l+1 must exist).
 *   w, cin, cout, y, dy, flags   as oc_conv_bwd (OC_FUSE_RELU masks dy with
 *           [y > 0], the convolution's own ReLU).
 *   xp      dev f32 [N_l][cin] or NULL: the pooled values (x itself); the
 *           routed gradient is kept only where xp > 0, the backward of a
 *           ReLU below the pooling, as oc_pool_bwd's y.
 *   sw      dev u8 [M_l][cin], the pooling's switches (oc_pool_fwd or
 *           oc_conv_pool_fwd at depth l+1).
 *   dxf     dev f32 [N_{l+1}][cin]: overwritten with the gradient w.r.t. the
 *           pooling's input (the pre-activation of the layer below when xp
 *           is given).
 *   dym     dev f32 [N_l][cout] or NULL: with OC_FUSE_RELU, receives dy
 *           masked with [y > 0] (the operand the weight gradient needs: a
 *           following oc_conv_bwd for dw can take it without OC_FUSE_RELU).
 *   ws      dev workspace of oc_conv_bwd_pool_workspace() bytes.
 * dxf equals, bit for bit, oc_conv_bwd (dx only, same flags) followed by
 * oc_pool_bwd(depth + 1, dx, sw, xp).  The weight gradient is a separate
 * oc_conv_bwd call (dx NULL). */
size_t oc_conv_bwd_pool_workspace(const oc_octree* tree, int32_t depth, int32_t ksize,
                                  int32_t cin, int32_t cout);
oc_status oc_conv_bwd_pool(const oc_octree* tree, int32_t depth, int32_t ksize, const float* w,
                           int32_t cin, int32_t cout, const float* y, const float* dy,
                           const float* xp, const uint8_t* sw, float* dxf, float* dym, void* ws,
                           size_t ws_bytes, int32_t flags, hipStream_t stream);

/* Octree deconvolution, also called transposed convolution (Sec. 3.2
 * "Deconvolution"): the transpose of the convolution cout -> cin with the
 * same weight tensor, obtained as the paper does by swapping that
 * convolution's forward and backward passes.
 *   depth   l, the depth of the output (the finer depth when strided).
 *   ksize   3 or 5 (stride 1); 3 (stride 2^r).
 *   stride  1: x dev [N_l][cin] -> y dev f32 [N_l][cout];
 *             y[n] = sum over the rows i and taps k whose neighbour is n of
 *             w[k] x[i] (the input gradient of oc_conv_fwd, cout -> cin).
 *           2^r (r = 1 .. depth): x dev [N_{l-r}][cin] -> y dev f32
 *             [N_l][cout], the transpose of the stride-2^r convolution at
 *             depth l: row i of x counts only when its octant is non-empty
 *             (label p > 0), and then reaches the depth-l neighbourhood of
 *             the first depth-l position below octant p-1.
 *   dt      OC_F32: x, w fp32.  OC_BF16: x, w bf16; products accumulate in
 *           fp32 (y is the fp32 deconvolution of the bf16 values).
 *   w       dev [K^3][cout][cin], the weight of the convolution it
 *           transposes (its index order: tap, that convolution's input
 *           channel = this call's output channel, output channel).
 *   ws      dev workspace of at least oc_deconv_fwd_workspace() bytes.
 *   flags   0 (a deconvolution is followed by normalisation before its
 *           ReLU in the paper's decoder unit, so none is fused).
 * Each pass runs on the convolution's kernels: the forward on the kernel
 * oc_conv_kernel(tree, depth, ksize, stride, dt, cout, cin, 1) names, the
 * input gradient on pass 0 and the weight gradient on pass 2 of the same
 * call.  Deterministic, as the convolution.  cin, cout in 1..1024. */
oc_status oc_deconv_fwd(const oc_octree* tree, int32_t depth, int32_t ksize, int32_t stride,
                        oc_dtype dt, const void* x, int32_t cin, const void* w, int32_t cout,
                        float* y, void* ws, size_t ws_bytes, int32_t flags, hipStream_t stream);

/* Bytes of device workspace oc_deconv_fwd needs for these arguments. */
size_t oc_deconv_fwd_workspace(const oc_octree* tree, int32_t depth, int32_t ksize,
                               int32_t stride, oc_dtype dt, int32_t cin, int32_t cout);

/* Bytes of device workspace oc_deconv_bwd needs for these arguments. */
size_t oc_deconv_bwd_workspace(const oc_octree* tree, int32_t depth, int32_t ksize,
                               int32_t stride, oc_dtype dt, int32_t cin, int32_t cout);

/* Backward of oc_deconv_fwd.  Arguments as oc_deconv_fwd, plus
 *   x    the forward input (read only when dw is requested).
 *   dy   dev f32 [N_l][cout] upstream gradient.  OC_BF16: the matrix-core
 *        operand is dy rounded to bf16, nearest-even.
 *   dx   dev f32, shaped as x, or NULL: the convolution cout -> cin of dy
 *        (strided: rows of empty depth-(l-r) octants are 0).
 *   dw   dev f32 [K^3][cout][cin] or NULL:
 *        dw[k][co][ci] = sum over rows i of x and taps k of dy[nb(i,k)][co]
 *        x[i][ci] (strided: rows of non-empty octants, at the first depth-l
 *        position below them).
 *   ws   dev workspace of at least oc_deconv_bwd_workspace() bytes; both
 *        passes use it in stream order.
 * Every argument is checked before either pass is enqueued. */
oc_status oc_deconv_bwd(const oc_octree* tree, int32_t depth, int32_t ksize, int32_t stride,
                        oc_dtype dt, const void* x, int32_t cin, const void* w, int32_t cout,
                        const float* dy, float* dx, float* dw, void* ws, size_t ws_bytes,
                        int32_t flags, hipStream_t stream);

/* 2x2x2 max-pooling from depth l to l-1 (Sec. 3.2 "Pooling", Fig. 5): for
 * every row i of depth l-1 with label p > 0, y[i] = channel-wise max of the
 * 8 rows 8(p-1)..8(p-1)+7 of depth l, sw[p-1][c] = the child index 0..7 of
 * that maximum (the first one on ties); rows with label 0 get y = 0.
 *   x  dev f32 [N_l][c];  y dev f32 [N_{l-1}][c];  sw dev u8 [M_{l-1}][c]. */
oc_status oc_pool_fwd(const oc_octree* tree, int32_t depth, const float* x, int32_t c, float* y,
                      uint8_t* sw, hipStream_t stream);

/* Gradient of oc_pool_fwd: dx[8(p-1) + sw[p-1][c]][c] = dy[i][c] for the row
 * i of label p at depth l-1; every other entry of dx is 0.
 *   dy dev f32 [N_{l-1}][c];  sw as produced by oc_pool_fwd;
 *   y  NULL, or dev f32 [N_{l-1}][c], the pooled output of oc_pool_fwd when
 *      its input came out of a ReLU (an oc_conv_fwd with OC_FUSE_RELU): the
 *      ReLU's backward is then applied as well, dx[...][c] = 0 where
 *      y[i][c] <= 0 (the routed child holds the value y[i][c]), so that dx is
 *      the gradient w.r.t. the convolution's pre-activation output;
 *   dx dev f32 [N_l][c]. */
oc_status oc_pool_bwd(const oc_octree* tree, int32_t depth, const float* dy, const uint8_t* sw,
                      int32_t c, const float* y, float* dx, hipStream_t stream);

/* 2x2x2 max-unpooling from depth l-1 to l (Sec. 3.2 "Unpooling", Fig. 5):
 * y[8(p-1) + sw[p-1][c]][c] = x[i][c] for the row i of label p at depth
 * l-1; every other entry of y is 0 (rows of empty parents have no children).
 *   depth  target depth l.  x dev f32 [N_{l-1}][c];  y dev f32 [N_l][c]. */
oc_status oc_unpool_fwd(const oc_octree* tree, int32_t depth, const float* x, const uint8_t* sw,
                        int32_t c, float* y, hipStream_t stream);

/* Gradient of oc_unpool_fwd: dx[i][c] = dy[8(p-1) + sw[p-1][c]][c] for the
 * row i of label p > 0 at depth l-1, 0 for label 0.
 *   dy dev f32 [N_l][c];  dx dev f32 [N_{l-1}][c]. */
oc_status oc_unpool_bwd(const oc_octree* tree, int32_t depth, const float* dy, const uint8_t* sw,
                        int32_t c, float* dx, hipStream_t stream);

/* General pooling (Sec. 3.2, last paragraph of "Pooling": pooling with other
 * kernel or stride sizes finds the neighbouring octants as the convolution
 * does and applies the pooling operation to them).  Over the K^3 taps k of
 * the convolution's neighbourhood (index as the convolution's weights), where
 * a neighbour that is not in the octree reads as 0, for every channel c:
 *   OC_POOL_MAX  y = the maximum; sw = the tap of its first occurrence in tap
 *                order, or 255 when that is an absent neighbour (whose zero
 *                then gets no gradient);
 *   OC_POOL_AVG  y = the sum over the K^3 taps / K^3 (sw unused).
 *   depth   l, the input depth (1..depth of the tree).
 *   ksize   3 or 5 (stride 1); 3 (stride 2^r).
 *   stride  1: y, sw [N_l][c], one output per octant of depth l.
 *           2^r, r = 1 .. l: y, sw [N_{l-r}][c]: evaluated where the
 *             stride-2^r convolution is (the first depth-l position below
 *             every non-empty depth-(l-r) octant, written to its row); rows
 *             of empty depth-(l-r) octants get y = 0 and sw = 255.
 *   x  dev f32 [N_l][c];  y dev f32;  sw dev u8 (max) or NULL (average). */
#define OC_POOL_MAX 0
#define OC_POOL_AVG 1
oc_status oc_gpool_fwd(const oc_octree* tree, int32_t depth, int32_t ksize, int32_t stride,
                       int32_t mode, const float* x, int32_t c, float* y, uint8_t* sw,
                       hipStream_t stream);

/* Gradient of oc_gpool_fwd: dx[n][c] = the sum over the outputs i whose tap k
 * reaches n of dy[i][c] if sw[i][c] == k (max), or of dy[i][c] / K^3
 * (average).  Stride 1: a gather in tap order (the average is the forward
 * applied to dy: i reaches n at offset d exactly when n reaches i at -d).
 * Stride 2: a gather per input row over its at most eight readers.  Stride
 * 2^r, r >= 2: every input row has at most one reader, which writes it; the
 * others are 0.  No atomics: deterministic.
 *   dy dev f32, shaped as y;  sw as produced by oc_gpool_fwd (max) or NULL;
 *   dx dev f32 [N_l][c]. */
oc_status oc_gpool_bwd(const oc_octree* tree, int32_t depth, int32_t ksize, int32_t stride,
                       int32_t mode, const float* dy, const uint8_t* sw, int32_t c, float* dx,
                       hipStream_t stream);

/* ---- The rest of the O-CNN(d) training iteration (Sec. 4 "Network
 * structure": units of convolution + batch normalisation + ReLU + pooling,
 * then dropout, fully connected layers and softmax; Sec. 5 "Training
 * details": SGD with momentum and weight decay).  Plain device buffers, fp32,
 * enqueued on `stream`; no floating-point atomics (reproducible bit for bit).
 *
 * Batch normalisation in training mode over the n rows of x [n][c] (all
 * octants of a depth, empty children included): per channel mean and biased
 * variance (double precision, one pass: per-block counts, means and sums of
 * squared deviations merged pairwise in a fixed order), y = (x - mean) invstd
 * gamma + beta, invstd = 1 / sqrt(var + eps); flags OC_FUSE_RELU applies
 * max(0, .) to y.  mean, invstd: dev f32 [c], written for the backward.
 * ws: dev, at least oc_bn_workspace(n, c) bytes. */
size_t oc_bn_workspace(int64_t n, int32_t c);
oc_status oc_bn_fwd(int64_t n, int32_t c, const float* x, const float* gamma, const float* beta,
                    float eps, int32_t flags, float* y, float* mean, float* invstd, void* ws,
                    size_t ws_bytes, hipStream_t stream);

/* Batch normalisation, optional ReLU and 2x2x2 max-pooling forward in one
 * call (the unit of Sec. 4 after its convolution): the statistics of
 * oc_bn_fwd over the N_l rows of z; the normalised values (ReLU'd with
 * OC_FUSE_RELU) are pooled to depth l-1 as oc_pool_fwd does, and never
 * written at depth l.  The backward is oc_pool_bwd with y (which applies the
 * ReLU's backward), then oc_bn_bwd on z.
 *   depth   l, 1 .. tree depth, with N_l > 0.
 *   z       dev f32 [N_l][c].  gamma, beta dev f32 [c].  eps > 0.
 *   y       dev f32 [N_{l-1}][c]: pooled features, empty octants' rows zero.
 *   sw      dev u8 [M_{l-1}][c]: switches, as oc_pool_fwd.
 *   mean, invstd  dev f32 [c], written for the backward.
 *   ws      dev, at least oc_bn_workspace(N_l, c) bytes.
 * y and sw equal oc_bn_fwd followed by oc_pool_fwd bit for bit. */
oc_status oc_bn_pool_fwd(const oc_octree* tree, int32_t depth, int32_t c, const float* z,
                         const float* gamma, const float* beta, float eps, int32_t flags, float* y,
                         uint8_t* sw, float* mean, float* invstd, void* ws, size_t ws_bytes,
                         hipStream_t stream);

/* Gradients of oc_bn_fwd (without the ReLU: dy is the gradient w.r.t. the
 * normalised output): dbeta = sum dy, dgamma = sum dy x_hat, dx = gamma
 * invstd (dy - dbeta / n - x_hat dgamma / n); dev f32, dx [n][c], dgamma and
 * dbeta [c]. */
oc_status oc_bn_bwd(int64_t n, int32_t c, const float* x, const float* dy, const float* gamma,
                    const float* mean, const float* invstd, float* dx, float* dgamma,
                    float* dbeta, void* ws, size_t ws_bytes, hipStream_t stream);

/* Fully connected layer: y [B][cout] = x [B][cin] w [cin][cout] + bias [cout]
 * (bias may be NULL).  Backward: dx = dy w^T, dw = x^T dy, dbias = sum of dy
 * over the batch; dx and dbias may be NULL. */
oc_status oc_fc_fwd(int32_t batch, int32_t cin, int32_t cout, const float* x, const float* w,
                    const float* bias, float* y, hipStream_t stream);
oc_status oc_fc_bwd(int32_t batch, int32_t cin, int32_t cout, const float* x, const float* w,
                    const float* dy, float* dx, float* dw, float* dbias, hipStream_t stream);

/* Dropout with ratio p in [0, 1): y = keep ? x / (1 - p) : 0, keep dev u8 [n]
 * (the mask is an input: the caller draws it).  The backward is the same call
 * on dy. */
oc_status oc_dropout(int64_t n, const float* x, const uint8_t* keep, float p, float* y,
                     hipStream_t stream);

/* Softmax cross-entropy over the batch: loss (dev f32 scalar) = mean over
 * the rows b of -log softmax(z[b])[labels[b]], dz [B][nc] = (softmax(z) -
 * onehot(labels)) / B.  z dev f32 [B][nc], labels dev i32 [B] in 0..nc-1.
 * ws: dev, at least oc_softmax_ce_workspace(B) bytes. */
size_t oc_softmax_ce_workspace(int32_t batch);
oc_status oc_softmax_ce(int32_t batch, int32_t nc, const float* z, const int32_t* labels,
                        float* loss, float* dz, void* ws, size_t ws_bytes, hipStream_t stream);

/* SGD step with momentum and weight decay, in place over n parameters:
 * v = momentum v + lr (g + decay w), w = w - v. */
oc_status oc_sgd(int64_t n, float* w, const float* g, float* v, float lr, float momentum,
                 float decay, hipStream_t stream);

/* Profiling: the next launch, on the calling thread, of the kernel that does
 * the main work of an entry point (the kernel oc_conv_kernel names for a
 * convolution pass; the pooling, routing or unpooling kernel of oc_pool_* /
 * oc_unpool_*) is bracketed by these events, recorded at the start and the
 * end of that kernel on its stream (as hipExtLaunchKernelGGL does), so that
 * its duration is measured without host-side gaps.  Both NULL clears a
 * pending pair.  The caller owns the events. */
oc_status oc_profile_next(hipEvent_t start, hipEvent_t stop);

/* Profiling: while armed, every kernel the library launches from the calling
 * thread is bracketed by the next pair starts[i], stops[i] (recorded at the
 * start and the end of that kernel on its stream, as hipExtLaunchKernelGGL
 * does), i = the value of *used before the launch, which is then incremented;
 * launches past cap are not bracketed.  A kernel that oc_profile_next
 * brackets takes that pair instead.  The sum of the pairs' durations is the
 * kernel time of the calls made while armed, without host-side gaps.
 * Arming sets *used = 0.  All four NULL/0 disarms.  The arrays and *used are
 * the caller's and must stay valid while armed.  Host-side only: no device
 * work is enqueued by this call. */
oc_status oc_profile_calls(hipEvent_t* starts, hipEvent_t* stops, int32_t cap, int32_t* used);

const char* oc_status_str(oc_status s);
const char* oc_last_error(void); /* thread-local message of the last failure */

#ifdef __cplusplus
}
#endif

#endif /* OC_H_ */
