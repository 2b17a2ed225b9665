"""GPU parity of convolution, pooling and unpooling against the CPU oracle.

Small cases compare every output element.  The full-size workloads, in the
launch configuration the bench uses, compare every output row, input-gradient
row and weight-gradient entry, except the 5x5x5 64->64 layer of wide_d7,
whose every row and entry is checked through random channel projections
(each implied by the elementwise rule) beside exact contiguous tiles and
exact entries of every (tap, 16 x 16 channel) block of dW."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import (assert_bf16_close, assert_dw_close, assert_f32_close, bf16_round)

pytestmark = pytest.mark.gpu


def _oc():
    import paper_1712_01537_amd as oc
    return oc


def _trees(pts, nrm, offs, depth, full=2):
    oc = _oc()
    ref = oracle.Octree(pts, nrm, offs, depth, full)
    tree = oc.oc_build(torch.as_tensor(pts).cuda(), torch.as_tensor(nrm).cuda(), offs, depth, full)
    assert [tree.num(l) for l in range(depth + 1)] == [ref.num(l) for l in range(depth + 1)]
    return ref, tree


def _cuda(a, dtype=torch.float32):
    return torch.as_tensor(np.ascontiguousarray(a)).to(dtype).cuda()


def _mask_ambiguous(dy, yref, relu):
    """Zero the upstream gradient where the fp32 sign of the pre-activation is
    not decided by the oracle's float64 value within the forward tolerance, so
    both sides take the same ReLU decision (float64 decides, rounded to fp32)."""
    if not relu:
        return dy
    dy = dy.copy()
    dy[np.abs(yref) <= 1e-4] = 0.0
    return dy


SMALL = [  # seed, B, n, depth, K, stride, cin, cout, relu
    (1, 2, 400, 4, 3, 1, 5, 7, False),
    (2, 3, 300, 4, 3, 1, 16, 32, True),
    (3, 1, 800, 5, 5, 1, 8, 8, False),
    (4, 2, 500, 4, 3, 2, 6, 10, False),
    (5, 2, 500, 5, 3, 2, 16, 16, True),
    (6, 1, 300, 3, 3, 1, 3, 16, True),
    (7, 4, 300, 4, 5, 1, 12, 20, True),
    (8, 2, 900, 5, 3, 1, 64, 128, False),
    (9, 3, 400, 4, 3, 1, 4, 32, True),  # 4-channel input, two column blocks
    (10, 2, 300, 5, 3, 1, 3, 20, False),  # 3-channel input, ragged column block
]


@pytest.mark.parametrize("seed,B,n,depth,K,stride,cin,cout,relu", SMALL)
def test_conv_small_fp32(seed, B, n, depth, K, stride, cin, cout, relu):
    oc = _oc()
    print(f"[conv] seed={seed} B={B} d={depth} K={K} s={stride} {cin}->{cout} relu={relu}", flush=True)
    pts, nrm, offs = synth.random_cloud(seed, B, n, "union")
    ref, tree = _trees(pts, nrm, offs, depth)
    l = depth
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((ref.num(l), cin)).astype(np.float32)
    w = (rng.standard_normal((K ** 3, cin, cout)) / np.sqrt(K ** 3 * cin)).astype(np.float32)
    n_out = ref.num(l) if stride == 1 else ref.num(l - 1)
    if stride == 1:
        nb = ref.neighbors(l, K)
        yref = oracle.conv_fwd(nb, x, w)
    else:
        nb = ref.neighbors(l, K, stride=2)
        yref = oracle.renew(ref.labels(l - 1), oracle.conv_fwd(nb, x, w))
    dy = _mask_ambiguous(rng.standard_normal((n_out, cout)).astype(np.float32), yref, relu)
    y = oc.oc_conv_fwd(tree, l, K, stride, _cuda(x), _cuda(w), relu=relu)
    yr = oracle.relu_fwd(yref) if relu else yref
    assert_f32_close(y.cpu().numpy(), yr, "y")
    dx, dw = oc.oc_conv_bwd(tree, l, K, stride, _cuda(x), _cuda(w), _cuda(dy), y=y, relu=relu)
    dye = oracle.relu_bwd(yref, dy) if relu else dy
    if stride == 1:
        dxr = oracle.conv_bwd_data(nb, dye, w, ref.num(l))
        dwr = oracle.conv_bwd_weight(nb, x, dye, K ** 3)
    else:
        dxr, dwr = oracle.conv_s2_bwd(ref, l, x, w, dye)
    assert_f32_close(dx.cpu().numpy(), dxr, "dx")
    assert_dw_close(dw.cpu().numpy(), dwr, "dw")
    # deterministic: identical bits on a second call
    dx2, dw2 = oc.oc_conv_bwd(tree, l, K, stride, _cuda(x), _cuda(w), _cuda(dy), y=y, relu=relu)
    assert torch.equal(dx.view(torch.int32), dx2.view(torch.int32))
    assert torch.equal(dw.view(torch.int32), dw2.view(torch.int32))


SR_SMALL = [  # seed, B, n, depth, stride, cin, cout, relu, bf16
    (101, 2, 400, 4, 4, 5, 7, False, False),
    (102, 3, 600, 5, 4, 16, 32, True, False),
    (103, 1, 900, 5, 4, 64, 16, False, False),
    (104, 2, 500, 4, 4, 8, 12, False, True),
    (105, 2, 800, 5, 4, 32, 32, True, True),
    (106, 3, 700, 5, 8, 16, 48, True, False),  # r = 3: depth 5 -> 2
    (107, 2, 900, 5, 8, 24, 16, False, True),
    (108, 2, 600, 5, 16, 32, 64, False, False),  # r = 4: depth 5 -> 1
    (109, 2, 500, 4, 16, 16, 16, True, True),   # r = 4: depth 4 -> 0 (the roots)
    (110, 4, 400, 4, 2, 80, 96, True, True),    # several output-column tiles, 3 reduction chunks
    (111, 2, 700, 5, 2, 3, 20, False, False),   # rows of 12 bytes (element-wise loads)
    (112, 2, 700, 5, 2, 36, 130, True, False),  # ragged channel chunks and columns
]


@pytest.mark.parametrize("seed,B,n,depth,stride,cin,cout,relu,bf16", SR_SMALL)
def test_conv_stride_pow2(seed, B, n, depth, stride, cin, cout, relu, bf16):
    """Stride 2^r (Sec. 3.2): depth l -> depth l-r, evaluated at the first
    depth-l position below every non-empty depth-(l-r) octant."""
    oc = _oc()
    print(f"[sr] seed={seed} B={B} d={depth} s={stride} {cin}->{cout} relu={relu} bf16={bf16}",
          flush=True)
    r = stride.bit_length() - 1
    pts, nrm, offs = synth.random_cloud(seed, B, n, "union")
    ref, tree = _trees(pts, nrm, offs, depth)
    l = depth
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((ref.num(l), cin)).astype(np.float32)
    w = (rng.standard_normal((27, cin, cout)) / np.sqrt(27 * cin)).astype(np.float32)
    dt = torch.bfloat16 if bf16 else torch.float32
    xq, wq = (bf16_round(x), bf16_round(w)) if bf16 else (x, w)
    pre = oracle.conv_sr_fwd(ref, l, xq, wq, stride)
    dy = _mask_ambiguous(rng.standard_normal((ref.num(l - r), cout)).astype(np.float32), pre,
                         relu)
    y = oc.oc_conv_fwd(tree, l, 3, stride, _cuda(x, dt), _cuda(w, dt), relu=relu)
    assert_f32_close(y.cpu().numpy(), oracle.relu_fwd(pre) if relu else pre, "y")
    dx, dw = oc.oc_conv_bwd(tree, l, 3, stride, _cuda(x, dt), _cuda(w, dt), _cuda(dy), y=y,
                            relu=relu)
    dye = oracle.relu_bwd(pre, dy) if relu else dy
    if bf16:  # the bf16 backward multiplies dy rounded to bf16
        dye = bf16_round(dye)
    dxr, dwr = oracle.conv_sr_bwd(ref, l, xq, wq, dye, stride)
    assert_f32_close(dx.cpu().numpy(), dxr, "dx")
    assert_dw_close(dw.cpu().numpy(), dwr, "dw")
    dx2, dw2 = oc.oc_conv_bwd(tree, l, 3, stride, _cuda(x, dt), _cuda(w, dt), _cuda(dy), y=y,
                              relu=relu)
    assert torch.equal(dx.view(torch.int32), dx2.view(torch.int32))
    assert torch.equal(dw.view(torch.int32), dw2.view(torch.int32))
    with pytest.raises(oc.OcError):  # strided convolution takes K = 3 only
        oc.oc_conv_fwd(tree, l, 5, stride, _cuda(x), _cuda(np.zeros((125, cin, cout))))


DECONV_SMALL = [  # seed, B, n, depth, K, stride, cin, cout (deconv channels), bf16
    (81, 2, 400, 4, 3, 1, 7, 5, False),
    (82, 2, 900, 5, 3, 1, 128, 64, False),  # split reduction in the forward (input-gradient kernel)
    (83, 1, 800, 5, 5, 1, 8, 8, False),
    (84, 2, 500, 4, 3, 2, 10, 6, False),
    (85, 2, 500, 5, 3, 2, 32, 16, False),
    (86, 3, 300, 4, 3, 1, 16, 3, False),  # down to 3 channels
    (87, 2, 700, 5, 3, 4, 24, 16, False),  # stride 4: depth 3 -> 5
    (88, 2, 600, 5, 3, 8, 16, 32, False),  # stride 8: depth 2 -> 5
    (89, 2, 700, 5, 3, 1, 32, 48, True),   # bf16 matrix-core kernels
    (90, 2, 500, 4, 5, 1, 12, 20, True),   # bf16 on widened operands
    (91, 3, 600, 5, 3, 2, 64, 32, True),
    (92, 2, 600, 5, 3, 4, 16, 16, True),
]


@pytest.mark.parametrize("seed,B,n,depth,K,stride,cin,cout,bf16", DECONV_SMALL)
def test_deconv_small(seed, B, n, depth, K, stride, cin, cout, bf16):
    oc = _oc()
    print(f"[deconv] seed={seed} B={B} d={depth} K={K} s={stride} {cin}->{cout} bf16={bf16}",
          flush=True)
    pts, nrm, offs = synth.random_cloud(seed, B, n, "union")
    ref, tree = _trees(pts, nrm, offs, depth)
    l = depth
    r = stride.bit_length() - 1
    rng = np.random.default_rng(seed)
    n_in = ref.num(l - r)
    x = rng.standard_normal((n_in, cin)).astype(np.float32)
    w = (rng.standard_normal((K ** 3, cout, cin)) / np.sqrt(K ** 3 * cin)).astype(np.float32)
    dy = rng.standard_normal((ref.num(l), cout)).astype(np.float32)
    dt = torch.bfloat16 if bf16 else torch.float32
    if bf16:  # the same bf16 values on both sides; the backward rounds dy to bf16
        x, w = bf16_round(x), bf16_round(w)
    dyq = bf16_round(dy) if bf16 else dy
    y = oc.oc_deconv_fwd(tree, l, K, stride, _cuda(x, dt), _cuda(w, dt))
    dx, dw = oc.oc_deconv_bwd(tree, l, K, stride, _cuda(x, dt), _cuda(w, dt), _cuda(dy))
    if stride == 1:
        nb = ref.neighbors(l, K)
        yr = oracle.deconv_fwd(nb, x, w, ref.num(l))
        dxr, dwr = oracle.deconv_bwd(nb, x, w, dyq)
    else:
        yr = oracle.deconv_sr_fwd(ref, l, x, w, stride)
        dxr, dwr = oracle.deconv_sr_bwd(ref, l, x, w, dyq, stride)
    assert_f32_close(y.cpu().numpy(), yr, "y")
    assert_f32_close(dx.cpu().numpy(), dxr, "dx")
    assert_dw_close(dw.cpu().numpy(), dwr, "dw")
    # deterministic: identical bits on a second call; each gradient alone equals the pair
    y2 = oc.oc_deconv_fwd(tree, l, K, stride, _cuda(x, dt), _cuda(w, dt))
    dx2, _ = oc.oc_deconv_bwd(tree, l, K, stride, _cuda(x, dt), _cuda(w, dt), _cuda(dy),
                              need_dw=False)
    _, dw2 = oc.oc_deconv_bwd(tree, l, K, stride, _cuda(x, dt), _cuda(w, dt), _cuda(dy),
                              need_dx=False)
    assert torch.equal(y.view(torch.int32), y2.view(torch.int32))
    assert torch.equal(dx.view(torch.int32), dx2.view(torch.int32))
    assert torch.equal(dw.view(torch.int32), dw2.view(torch.int32))


def test_deconv_argument_errors():
    oc = _oc()
    pts = np.array([[0.3, 0.6, 0.9]], np.float32)
    ref, tree = _trees(pts, np.ones((1, 3), np.float32), [0, 1], 3, 0)
    x = _cuda(np.zeros((ref.num(3), 4)))
    with pytest.raises(oc.OcError):  # x and w of different dtypes
        oc.oc_deconv_fwd(tree, 3, 3, 1, x.to(torch.bfloat16), _cuda(np.zeros((27, 2, 4))))
    with pytest.raises(oc.OcError):  # stride 16 from depth 3
        oc.oc_deconv_fwd(tree, 3, 3, 16, _cuda(np.zeros((ref.num(0), 4))),
                         _cuda(np.zeros((27, 2, 4))))
    with pytest.raises(oc.OcError):  # kernel size 7
        oc.oc_deconv_fwd(tree, 3, 7, 1, x, _cuda(np.zeros((343, 2, 4))))
    with pytest.raises(oc.OcError):  # stride 2 with K = 5
        oc.oc_deconv_bwd(tree, 3, 5, 2, _cuda(np.zeros((ref.num(2), 4))),
                         _cuda(np.zeros((125, 2, 4))), _cuda(np.zeros((ref.num(3), 2))))


@pytest.mark.parametrize("K,stride", [(3, 1), (5, 1), (3, 2)])
def test_conv_small_bf16(K, stride):
    oc = _oc()
    pts, nrm, offs = synth.random_cloud(20 + K, 2, 600, "union")
    ref, tree = _trees(pts, nrm, offs, 5)
    l, cin, cout = 5, 32, 48
    rng = np.random.default_rng(K)
    x32 = rng.standard_normal((ref.num(l), cin)).astype(np.float32)
    w32 = (rng.standard_normal((K ** 3, cin, cout)) / np.sqrt(K ** 3 * cin)).astype(np.float32)
    x, w = bf16_round(x32), bf16_round(w32)
    nb = ref.neighbors(l, K, stride=stride)

    def fwd(a, b):
        r = oracle.conv_fwd(nb, a, b)
        return oracle.renew(ref.labels(l - 1), r) if stride == 2 else r

    yref = fwd(x, w)
    y = oc.oc_conv_fwd(tree, l, K, stride, _cuda(x, torch.bfloat16), _cuda(w, torch.bfloat16))
    # same bf16 values on both sides: only the fp32 accumulation differs
    assert_f32_close(y.cpu().numpy(), yref, "y bf16 inputs")
    # against the fp32-input oracle: the bf16 rounding of inputs and weights
    assert_bf16_close(y.cpu().numpy(), fwd(x32, w32), "y vs fp32 oracle")
    dy = rng.standard_normal(yref.shape).astype(np.float32)
    dx, dw = oc.oc_conv_bwd(tree, l, K, stride, _cuda(x, torch.bfloat16), _cuda(w, torch.bfloat16), _cuda(dy))
    if stride == 1:
        # the stride-1 bf16 backward multiplies dy rounded to bf16
        dyq = bf16_round(dy)
        dxr = oracle.conv_bwd_data(nb, dyq, w, ref.num(l))
        dwr = oracle.conv_bwd_weight(nb, x, dyq, K ** 3)
        assert_bf16_close(dx.cpu().numpy(), oracle.conv_bwd_data(nb, dy, w32, ref.num(l)),
                          "dx vs fp32 oracle")
        assert_bf16_close(dw.cpu().numpy(), oracle.conv_bwd_weight(nb, x32, dy, K ** 3),
                          "dw vs fp32 oracle")
    else:  # the stride-2 bf16 backward multiplies dy rounded to bf16 as well
        dxr, dwr = oracle.conv_s2_bwd(ref, l, x, w, bf16_round(dy))
        dx32, dw32 = oracle.conv_s2_bwd(ref, l, x32, w32, dy)
        assert_bf16_close(dx.cpu().numpy(), dx32, "dx vs fp32 oracle")
        assert_bf16_close(dw.cpu().numpy(), dw32, "dw vs fp32 oracle")
    assert_f32_close(dx.cpu().numpy(), dxr, "dx bf16 weights")
    assert_dw_close(dw.cpu().numpy(), dwr, "dw bf16 inputs")


DEFER_LAYERS = [  # K, stride, dtype, cin, cout: every weight-gradient path, and layers
    # without a deferred form (strided; bf16 on the bf16 kernels)
    (3, 1, torch.float32, 3, 16),     # first layer (Cin 3)
    (3, 1, torch.float32, 4, 32),     # first layer (Cin 4)
    (3, 1, torch.float32, 16, 32),    # matrix-core weight gradient, K = 3
    (3, 1, torch.float32, 5, 7),      # ragged channels
    (5, 1, torch.float32, 8, 16),     # K = 5
    (3, 1, torch.bfloat16, 8, 24),    # bf16 widened to fp32
    (3, 2, torch.float32, 16, 16),    # strided: dw written by the call
    (3, 1, torch.bfloat16, 16, 32),   # bf16 kernels: dw written by the call
    (3, 1, torch.float32, 32, 64),
    (3, 1, torch.float32, 64, 128),
    (3, 1, torch.float32, 16, 16),    # a ninth deferred set: a second launch
]


def test_conv_bwd_deferred_dw():
    """oc_conv_bwd with OC_DEFER_DW leaves the weight gradient's partial sums
    in its workspace; one oc_sum_partials over all layers gives the same bits
    as the calls without it."""
    oc = _oc()
    pts, nrm, offs = synth.random_cloud(151, 2, 600, "union")
    ref, tree = _trees(pts, nrm, offs, 5)
    rng = np.random.default_rng(151)
    pending, direct, deferred, nparts = [], [], [], []
    for K, stride, dt, cin, cout in DEFER_LAYERS:
        l = 5
        n_out = ref.num(l) if stride == 1 else ref.num(l - 1)
        x = _cuda(rng.standard_normal((ref.num(l), cin)).astype(np.float32), dt)
        w = _cuda((rng.standard_normal((K ** 3, cin, cout)) / np.sqrt(K ** 3 * cin)).astype(np.float32), dt)
        dy = _cuda(rng.standard_normal((n_out, cout)).astype(np.float32))
        _, dw = oc.oc_conv_bwd(tree, l, K, stride, x, w, dy, need_dx=False)
        before = len(pending)
        _, dwd = oc.oc_conv_bwd(tree, l, K, stride, x, w, dy, need_dx=False, defer=pending)
        nparts.append(len(pending) - before)
        print(f"[defer] K{K} s{stride} {dt} {cin}->{cout}: deferred {nparts[-1]}", flush=True)
        direct.append(dw)
        deferred.append(dwd)
    # every stride-1 layer off the bf16 kernels has a deferred form
    assert nparts == [1, 1, 1, 1, 1, 1, 0, 0, 1, 1, 1]
    oc.oc_sum_partials(pending)
    assert pending == []
    for (K, stride, dt, cin, cout), a, b in zip(DEFER_LAYERS, direct, deferred):
        assert torch.equal(a, b), (K, stride, dt, cin, cout)


BF16_NATIVE = [  # seed, B, n, depth, K, cin, cout, relu: tiles with ragged tails, one or two
    # 64-channel chunks of the reduction, one or two 64-column output blocks
    (41, 2, 700, 5, 5, 64, 64, False),
    (42, 3, 400, 4, 3, 16, 48, True),
    (43, 1, 900, 5, 5, 80, 32, True),
    (44, 2, 300, 4, 3, 128, 96, False),
    (45, 1, 200, 3, 5, 32, 16, False),
    # 16-group tiles (K = 5, whole 32-channel halves, 64-column blocks): two
    # chunks of 64, two column blocks, a 64 + 32 split
    (46, 2, 500, 4, 5, 128, 64, True),
    (47, 1, 600, 5, 5, 96, 128, False),
]


@pytest.mark.parametrize("seed,B,n,depth,K,cin,cout,relu", BF16_NATIVE)
def test_conv_bf16_matrix_core(seed, B, n, depth, K, cin, cout, relu):
    """bf16 stride-1 shapes with channel counts that are multiples of 16 (the
    bf16 matrix-core kernels), against the oracle on the same bf16 values."""
    oc = _oc()
    pts, nrm, offs = synth.random_cloud(seed, B, n, "union")
    ref, tree = _trees(pts, nrm, offs, depth)
    l = depth
    rng = np.random.default_rng(seed)
    x = bf16_round(rng.standard_normal((ref.num(l), cin)).astype(np.float32))
    w = bf16_round((rng.standard_normal((K ** 3, cin, cout)) / np.sqrt(K ** 3 * cin)).astype(np.float32))
    nb = ref.neighbors(l, K)
    pre = oracle.conv_fwd(nb, x, w)
    print(f"[bf16 {seed}] d{l} K{K} {cin}->{cout} rows {ref.num(l)} relu {relu}", flush=True)
    y = oc.oc_conv_fwd(tree, l, K, 1, _cuda(x, torch.bfloat16), _cuda(w, torch.bfloat16), relu=relu)
    assert_f32_close(y.cpu().numpy(), oracle.relu_fwd(pre) if relu else pre, "y")
    dy = _mask_ambiguous(rng.standard_normal(pre.shape).astype(np.float32), pre, relu)
    dye = bf16_round(oracle.relu_bwd(pre, dy) if relu else dy)
    dx, dw = oc.oc_conv_bwd(tree, l, K, 1, _cuda(x, torch.bfloat16), _cuda(w, torch.bfloat16),
                            _cuda(dy), y=y, relu=relu)
    assert_f32_close(dx.cpu().numpy(), oracle.conv_bwd_data(nb, dye, w, ref.num(l)), "dx")
    rule = assert_dw_close(dw.cpu().numpy(), oracle.conv_bwd_weight(nb, x, dye, K ** 3), "dw")
    print(f"[bf16 {seed}] dw rule: {rule}", flush=True)
    # reproducible bit for bit
    dx2, dw2 = oc.oc_conv_bwd(tree, l, K, 1, _cuda(x, torch.bfloat16), _cuda(w, torch.bfloat16),
                              _cuda(dy), y=y, relu=relu)
    assert torch.equal(dx, dx2) and torch.equal(dw, dw2)


GPOOL_SMALL = [  # seed, B, n, depth, K, stride, c, relu (inputs through a ReLU: exact zeros, ties)
    (91, 2, 400, 4, 3, 1, 16, False),
    (92, 3, 300, 4, 5, 1, 5, False),
    (93, 1, 800, 5, 3, 1, 7, True),
    (94, 2, 500, 4, 5, 1, 32, True),
    (95, 2, 600, 5, 3, 2, 16, False),
    (96, 3, 500, 4, 3, 2, 7, True),
    (97, 2, 700, 5, 3, 4, 12, True),
    (98, 2, 700, 5, 3, 8, 5, False),
    (99, 1, 400, 4, 3, 16, 8, True),  # depth 4 -> the roots
]


@pytest.mark.parametrize("seed,B,n,depth,K,stride,c,relu", GPOOL_SMALL)
def test_gpool_small(seed, B, n, depth, K, stride, c, relu):
    oc = _oc()
    print(f"[gpool] seed={seed} B={B} d={depth} K={K} s={stride} c={c} relu={relu}", flush=True)
    pts, nrm, offs = synth.random_cloud(seed, B, n, "union")
    ref, tree = _trees(pts, nrm, offs, depth)
    l = depth
    r = stride.bit_length() - 1
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((ref.num(l), c)).astype(np.float32)
    if relu:
        x = np.maximum(x, 0)
    dy = rng.standard_normal((ref.num(l - r), c)).astype(np.float32)
    if stride == 1:
        nb = ref.neighbors(l, K)
        fwd = lambda a, m: oracle.gpool_fwd(nb, a, m)  # noqa: E731
        bwd = lambda g, s_, m: oracle.gpool_bwd(nb, g, s_, ref.num(l), m)  # noqa: E731
    else:
        fwd = lambda a, m: oracle.gpool_sr_fwd(ref, l, a, m, stride)  # noqa: E731
        bwd = lambda g, s_, m: oracle.gpool_sr_bwd(ref, l, g, s_, ref.num(l), m, stride)  # noqa: E731
    # max: values and switches bit-exact, the gradient within the fp32 rule
    y, sw = oc.oc_gpool_fwd(tree, l, K, oc.OC_POOL_MAX, _cuda(x), stride=stride)
    yr, swr = fwd(x, oracle.POOL_MAX)
    np.testing.assert_array_equal(y.cpu().numpy(), yr)
    np.testing.assert_array_equal(sw.cpu().numpy(), swr)
    dx = oc.oc_gpool_bwd(tree, l, K, oc.OC_POOL_MAX, _cuda(dy), sw, stride=stride)
    assert_f32_close(dx.cpu().numpy(), bwd(dy, swr, oracle.POOL_MAX), "max dx")
    # average
    ya, _ = oc.oc_gpool_fwd(tree, l, K, oc.OC_POOL_AVG, _cuda(x), stride=stride)
    assert_f32_close(ya.cpu().numpy(), fwd(x, oracle.POOL_AVG)[0], "avg y")
    dxa = oc.oc_gpool_bwd(tree, l, K, oc.OC_POOL_AVG, _cuda(dy), None, stride=stride)
    assert_f32_close(dxa.cpu().numpy(), bwd(dy, None, oracle.POOL_AVG), "avg dx")
    # deterministic
    dx2 = oc.oc_gpool_bwd(tree, l, K, oc.OC_POOL_MAX, _cuda(dy), sw, stride=stride)
    assert torch.equal(dx.view(torch.int32), dx2.view(torch.int32))
    if stride > 1:
        with pytest.raises(oc.OcError):  # strided pooling takes K = 3 only
            oc.oc_gpool_fwd(tree, l, 5, oc.OC_POOL_MAX, _cuda(x), stride=stride)


@pytest.mark.parametrize("seed,B,n,depth,c", [(31, 2, 500, 4, 8), (32, 3, 300, 5, 3), (33, 1, 100, 3, 32)])
def test_pool_unpool_small(seed, B, n, depth, c):
    oc = _oc()
    pts, nrm, offs = synth.random_cloud(seed, B, n, "union")
    ref, tree = _trees(pts, nrm, offs, depth)
    l = depth
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((ref.num(l), c)).astype(np.float32)
    x[::5] = np.round(x[::5])  # plenty of ties among siblings
    y, sw = oc.oc_pool_fwd(tree, l, _cuda(x))
    yr, swr = oracle.pool_fwd(ref.labels(l - 1), x)
    np.testing.assert_array_equal(y.cpu().numpy(), yr)
    np.testing.assert_array_equal(sw.cpu().numpy(), swr)
    dy = rng.standard_normal((ref.num(l - 1), c)).astype(np.float32)
    np.testing.assert_array_equal(oc.oc_pool_bwd(tree, l, _cuda(dy), sw).cpu().numpy(),
                                  oracle.pool_bwd(ref.labels(l - 1), dy, swr, ref.num(l)))
    np.testing.assert_array_equal(oc.oc_unpool_fwd(tree, l, _cuda(dy), sw).cpu().numpy(),
                                  oracle.unpool_fwd(ref.labels(l - 1), dy, swr, ref.num(l)))
    # ReLU before the pooling: pool_bwd with y applies the ReLU's backward too
    z = x.copy()
    z[1::7] = 0.0
    a = np.maximum(z, 0.0)
    ya, swa = oc.oc_pool_fwd(tree, l, _cuda(a))
    _, swar = oracle.pool_fwd(ref.labels(l - 1), a)
    np.testing.assert_array_equal(
        oc.oc_pool_bwd(tree, l, _cuda(dy), swa, y=ya).cpu().numpy(),
        oracle.relu_bwd(z, oracle.pool_bwd(ref.labels(l - 1), dy, swar, ref.num(l))))
    g = rng.standard_normal((ref.num(l), c)).astype(np.float32)
    np.testing.assert_array_equal(oc.oc_unpool_bwd(tree, l, _cuda(g), sw).cpu().numpy(),
                                  oracle.unpool_bwd(ref.labels(l - 1), g, swr))


def _check_conv_pool(ref, tree, l, K, x, w, relu, tag, dtype=torch.float32, yref=None):
    """oc_conv_pool_fwd against oc_conv_fwd + oc_pool_fwd (bit for bit), the
    oracle's pooling of the GPU's own depth-l output (bit for bit: the same
    fp32 values decide) and, when yref (the oracle's float64 convolution) is
    given, the oracle's conv + ReLU + pooling within the fp32 tolerance."""
    oc = _oc()
    xg, wg = _cuda(x, dtype), _cuda(w, dtype)
    y, sw = oc.oc_conv_pool_fwd(tree, l, K, xg, wg, relu=relu)
    yl = oc.oc_conv_fwd(tree, l, K, 1, xg, wg, relu=relu)
    yu, swu = oc.oc_pool_fwd(tree, l, yl)
    assert torch.equal(y.view(torch.int32), yu.view(torch.int32)), f"{tag}: fused y != unfused"
    assert torch.equal(sw, swu), f"{tag}: fused switches != unfused"
    yo, swo = oracle.pool_fwd(ref.labels(l - 1), yl.cpu().numpy())
    np.testing.assert_array_equal(y.cpu().numpy(), yo)
    np.testing.assert_array_equal(sw.cpu().numpy(), swo)
    if yref is not None:
        yr = oracle.relu_fwd(yref) if relu else yref
        assert_f32_close(y.cpu().numpy(), oracle.pool_fwd(ref.labels(l - 1), yr)[0], f"{tag} y")
    # a second call gives the same bits (fixed-order sums, no atomics)
    y2, sw2 = oc.oc_conv_pool_fwd(tree, l, K, xg, wg, relu=relu)
    assert torch.equal(y.view(torch.int32), y2.view(torch.int32)) and torch.equal(sw, sw2)


CONV_POOL_SMALL = [  # seed, B, n, depth, K, cin, cout, relu, bf16
    (121, 2, 500, 4, 3, 3, 16, True, False),    # first-layer kernel, pooled epilogue
    (122, 3, 300, 5, 3, 4, 32, True, False),    # two column blocks
    (123, 1, 700, 5, 3, 3, 48, False, False),   # no ReLU
    (124, 2, 600, 5, 3, 16, 32, True, False),   # group-tile kernel, pooled epilogue
    (125, 3, 400, 4, 3, 16, 16, False, False),
    (126, 2, 900, 5, 3, 32, 64, True, False),   # split reduction: pooled split sum
    (127, 2, 500, 4, 3, 64, 128, True, False),
    (128, 2, 400, 4, 3, 5, 7, True, False),     # other shapes: conv, then pooling
    (129, 1, 500, 4, 5, 8, 8, True, False),
    (130, 2, 500, 4, 3, 16, 32, True, True),
]


@pytest.mark.parametrize("seed,B,n,depth,K,cin,cout,relu,bf16", CONV_POOL_SMALL)
def test_conv_pool_small(seed, B, n, depth, K, cin, cout, relu, bf16):
    """Convolution + ReLU + 2x2x2 max-pool in one call (Sec. 3.2, Sec. 4)."""
    print(f"[conv_pool] seed={seed} B={B} d={depth} K={K} {cin}->{cout} relu={relu} bf16={bf16}",
          flush=True)
    pts, nrm, offs = synth.random_cloud(seed, B, n, "union")
    ref, tree = _trees(pts, nrm, offs, depth)
    l = depth
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((ref.num(l), cin)).astype(np.float32)
    w = (rng.standard_normal((K ** 3, cin, cout)) / np.sqrt(K ** 3 * cin)).astype(np.float32)
    if bf16:
        x, w = bf16_round(x), bf16_round(w)
    yref = oracle.conv_fwd(ref.neighbors(l, K), x, w)
    _check_conv_pool(ref, tree, l, K, x, w, relu, f"conv_pool {seed}",
                     torch.bfloat16 if bf16 else torch.float32, yref)


CONV_BWD_POOL_SMALL = [  # seed, B, n, fine depth, K, cin, cout, conv ReLU, pooled-value mask
    (141, 2, 500, 5, 3, 16, 16, False, True),   # one reduction chunk: no split
    (142, 2, 600, 5, 3, 16, 32, True, True),    # two splits, the convolution's own ReLU
    (143, 3, 400, 4, 3, 32, 64, False, True),   # four splits
    (144, 2, 500, 4, 3, 64, 128, True, True),   # eight splits
    (145, 2, 400, 4, 3, 6, 8, False, True),     # cin % 4 != 0: gradient, then routing
    (146, 1, 500, 4, 5, 8, 8, False, True),     # K = 5 group-tile kernel
    (147, 2, 300, 4, 3, 4, 16, True, False),    # no mask
]


@pytest.mark.parametrize("seed,B,n,depth,K,cin,cout,relu,masked", CONV_BWD_POOL_SMALL)
def test_conv_bwd_pool_small(seed, B, n, depth, K, cin, cout, relu, masked):
    """Input gradient of a convolution routed on through the max-pool that
    produced its input (Sec. 3.2 "Pooling"): bit for bit oc_conv_bwd's input
    gradient followed by oc_pool_bwd, and the oracle's gradient within the
    fp32 tolerance."""
    print(f"[conv_bwd_pool] seed={seed} B={B} d={depth} K={K} {cin}->{cout} relu={relu} "
          f"masked={masked}", flush=True)
    oc = _oc()
    pts, nrm, offs = synth.random_cloud(seed, B, n, "union")
    ref, tree = _trees(pts, nrm, offs, depth)
    lf, l = depth, depth - 1
    rng = np.random.default_rng(seed)
    # the layer below: ReLU'd activations at depth lf, pooled to depth l
    z = rng.standard_normal((ref.num(lf), cin)).astype(np.float32)
    z[1::7] = 0.0
    a = np.maximum(z, 0.0)
    p, sw = oc.oc_pool_fwd(tree, lf, _cuda(a))
    _, swr = oracle.pool_fwd(ref.labels(l), a)
    w = (rng.standard_normal((K ** 3, cin, cout)) / np.sqrt(K ** 3 * cin)).astype(np.float32)
    dy = rng.standard_normal((ref.num(l), cout)).astype(np.float32)
    y = rng.standard_normal((ref.num(l), cout)).astype(np.float32)
    y[::3] = 0.0
    wg, dyg, yg = _cuda(w), _cuda(dy), _cuda(y)
    xp = p if masked else None
    dym = torch.full_like(dyg, float("nan")) if relu else None
    dxf = oc.oc_conv_bwd_pool(tree, l, K, wg, dyg, sw, xp=xp, y=yg, relu=relu, dym=dym)
    if relu:  # the masked upstream gradient handed out for the weight gradient
        np.testing.assert_array_equal(dym.cpu().numpy(), np.where(y > 0, dy, np.float32(0)))
    dx, _ = oc.oc_conv_bwd(tree, l, K, 1, p, wg, dyg, y=yg, relu=relu, need_dx=True,
                           need_dw=False)
    dxu = oc.oc_pool_bwd(tree, lf, dx, sw, y=xp)
    assert torch.equal(dxf.view(torch.int32), dxu.view(torch.int32)), "fused != unfused"
    g = oracle.relu_bwd(y, dy) if relu else dy
    dxo = oracle.conv_bwd_data(ref.neighbors(l, K), g, w, ref.num(l))
    ro = oracle.pool_bwd(ref.labels(l), dxo, swr, ref.num(lf))
    if masked:
        ro = oracle.relu_bwd(z, ro)
    assert_f32_close(dxf.cpu().numpy(), ro, f"conv_bwd_pool {seed}")
    dxf2 = oc.oc_conv_bwd_pool(tree, l, K, wg, dyg, sw, xp=xp, y=yg, relu=relu)
    assert torch.equal(dxf.view(torch.int32), dxf2.view(torch.int32)), "not reproducible"


def test_conv_pool_one_point_tree():
    """A one-point tree (one sibling group per depth) down to depth 1."""
    pts = np.array([[0.3, 0.6, 0.9]], np.float32)
    ref, tree = _trees(pts, np.ones((1, 3), np.float32), [0, 1], 3, 0)
    rng = np.random.default_rng(17)
    for l in (1, 2, 3):
        for cin, cout in ((3, 16), (16, 16), (32, 32)):
            x = rng.standard_normal((ref.num(l), cin)).astype(np.float32)
            w = rng.standard_normal((27, cin, cout)).astype(np.float32)
            _check_conv_pool(ref, tree, l, 3, x, w, True, f"one point l={l} {cin}->{cout}",
                             yref=oracle.conv_fwd(ref.neighbors(l, 3), x, w))


def test_conv_edge_cases():
    oc = _oc()
    # a single shape with one point, full depth 0: depth-1 has 8 octants, one group
    pts = np.array([[0.3, 0.6, 0.9]], np.float32)
    nrm = np.ones((1, 3), np.float32)
    ref, tree = _trees(pts, nrm, [0, 1], 3, 0)
    for l in (1, 2, 3):
        x = np.arange(ref.num(l) * 2, dtype=np.float32).reshape(-1, 2) / 7
        w = np.linspace(-1, 1, 27 * 2 * 3, dtype=np.float32).reshape(27, 2, 3)
        y = oc.oc_conv_fwd(tree, l, 3, 1, _cuda(x), _cuda(w))
        assert_f32_close(y.cpu().numpy(), oracle.conv_fwd(ref.neighbors(l, 3), x, w), f"y l={l}")
    # argument errors are reported, nothing launched
    with pytest.raises(oc.OcError):
        oc.oc_conv_fwd(tree, 0, 3, 1, _cuda(np.zeros((1, 2))), _cuda(np.zeros((27, 2, 3))))
    with pytest.raises(oc.OcError):
        oc.oc_conv_fwd(tree, 3, 7, 1, _cuda(np.zeros((ref.num(3), 2))), _cuda(np.zeros((343, 2, 3))))


def test_new_ops_degenerate_trees():
    """Deconvolution, general pooling and stride 4 on a one-point tree with
    full depth 0 (one sibling group per depth, most neighbours outside the
    cube) and at the shallowest depths they accept."""
    oc = _oc()
    pts = np.array([[0.3, 0.6, 0.9]], np.float32)
    ref, tree = _trees(pts, np.ones((1, 3), np.float32), [0, 1], 3, 0)
    rng = np.random.default_rng(7)
    for l in (1, 2, 3):
        n = ref.num(l)
        for K in (3, 5):
            x = rng.standard_normal((n, 4)).astype(np.float32)
            nb = ref.neighbors(l, K)
            for mode, rmode in ((oc.OC_POOL_MAX, oracle.POOL_MAX), (oc.OC_POOL_AVG, oracle.POOL_AVG)):
                y, sw = oc.oc_gpool_fwd(tree, l, K, mode, _cuda(x))
                yr, swr = oracle.gpool_fwd(nb, x, rmode)
                assert_f32_close(y.cpu().numpy(), yr, f"gpool y l={l} K={K}")
                if sw is not None:
                    np.testing.assert_array_equal(sw.cpu().numpy(), swr)
                dx = oc.oc_gpool_bwd(tree, l, K, mode, _cuda(x), sw)
                assert_f32_close(dx.cpu().numpy(), oracle.gpool_bwd(nb, x, swr, n, rmode),
                                 f"gpool dx l={l} K={K}")
        w = rng.standard_normal((27, 3, 4)).astype(np.float32)  # deconv 4 -> 3
        x = rng.standard_normal((n, 4)).astype(np.float32)
        nb = ref.neighbors(l, 3)
        assert_f32_close(oc.oc_deconv_fwd(tree, l, 3, 1, _cuda(x), _cuda(w)).cpu().numpy(),
                         oracle.deconv_fwd(nb, x, w, n), f"deconv l={l}")
        xs = rng.standard_normal((ref.num(l - 1), 4)).astype(np.float32)
        assert_f32_close(oc.oc_deconv_fwd(tree, l, 3, 2, _cuda(xs), _cuda(w)).cpu().numpy(),
                         oracle.deconv_s2_fwd(ref, l, xs, w), f"deconv s2 l={l}")
    for l, st in ((2, 4), (3, 4), (3, 8)):  # strides 4 and 8 down to depths 0 and 1
        r = st.bit_length() - 1
        x = rng.standard_normal((ref.num(l), 16)).astype(np.float32)
        w = rng.standard_normal((27, 16, 16)).astype(np.float32)
        y = oc.oc_conv_fwd(tree, l, 3, st, _cuda(x), _cuda(w))
        assert_f32_close(y.cpu().numpy(), oracle.conv_sr_fwd(ref, l, x, w, st), f"s{st} l={l}")
        dy = rng.standard_normal((ref.num(l - r), 16)).astype(np.float32)
        dx, dw = oc.oc_conv_bwd(tree, l, 3, st, _cuda(x), _cuda(w), _cuda(dy))
        dxr, dwr = oracle.conv_sr_bwd(ref, l, x, w, dy, st)
        assert_f32_close(dx.cpu().numpy(), dxr, f"s{st} dx l={l}")
        assert_dw_close(dw.cpu().numpy(), dwr, f"s{st} dw l={l}")
    with pytest.raises(oc.OcError):  # stride 4 from depth 1
        oc.oc_conv_fwd(tree, 1, 3, 4, _cuda(np.zeros((ref.num(1), 16))), _cuda(np.zeros((27, 16, 16))))


# ----------------------------------------------------------------------------
# full-size workloads: every output row, input-gradient row and weight-gradient
# entry against the oracle; for the 5x5x5 64->64 layer of wide_d7 (about 1.2
# TFLOP per pass, minutes for the float64 oracle) every row and entry through
# random channel projections plus exact contiguous tiles, as below


def _proj_tol(g, b, atol):
    """Bound on |g.b - r.b| implied by the elementwise rule |g - r| <= atol +
    RTOL |r| for every entry of the row (then |g - r| <= (atol + RTOL |g|) /
    (1 - RTOL))."""
    from helpers import RTOL
    return (np.abs(g) * RTOL + atol) @ np.abs(b) / (1 - RTOL) + 1e-12


def _assert_proj(g, b, ref_proj, what, atol=None):
    """Every row of g projected on b (a random channel vector) against the
    oracle's projection ref_proj [rows].  atol: the absolute term of the
    elementwise rule (the fp32 rule's by default; the scaled weight-gradient
    rule's 1e-5 max(1, rms) for dW)."""
    from helpers import ATOL
    g = np.asarray(g, np.float64)
    got = g @ b
    tol = _proj_tol(g, b, ATOL if atol is None else atol)
    err = np.abs(got - ref_proj)
    bad = err > tol
    if bad.any():
        i = int(np.argmax(err - tol))
        raise AssertionError(f"{what}: {int(bad.sum())} of {len(err)} rows fail the projected "
                             f"rule; worst row {i}: got {got[i]!r} ref {ref_proj[i]!r}")


def _tiles(n_rows, every, tile=64):
    """Rows of every `every`-th tile of `tile` rows (with the first and last
    two tiles), as a bool mask and as a sorted index array."""
    nt = -(-n_rows // tile)
    pick = set(range(0, nt, every)) | {0, 1, max(nt - 2, 0), nt - 1}
    want = np.zeros(n_rows, bool)
    for t in pick:
        want[t * tile:(t + 1) * tile] = True
    return want, np.nonzero(want)[0]


def _dw_block_entries(K3, cin, cout, rng, per=2):
    """`per` random entries of every (tap, 16 input x 16 output channel)
    block of dW, as flat indices into [K3][cin][cout]."""
    out = []
    for k in range(K3):
        for c0 in range(0, cin, 16):
            for n0 in range(0, cout, 16):
                ci = rng.integers(c0, min(c0 + 16, cin), size=per)
                co = rng.integers(n0, min(n0 + 16, cout), size=per)
                out.append((k * cin + ci) * cout + co)
    return np.unique(np.concatenate(out))


def _check_conv_full(ref, tree, l, K, stride, x, w, relu, dy, tag, dtype=torch.float32):
    oc = _oc()
    n_in = ref.num(l)
    nb = ref.neighbors(l, K, stride=stride)
    xq, wq = (x, w) if dtype == torch.float32 else (bf16_round(x), bf16_round(w))
    K3, cin, cout = w.shape
    big = K3 * cin * cout * nb.shape[0] > 6e10  # float64 oracle minutes per pass
    print(f"[{tag}] conv d{l} K{K} s{stride} {cin}->{cout} rows {n_in} "
          f"{'projected + tiles' if big else 'every element'}", flush=True)
    y = oc.oc_conv_fwd(tree, l, K, stride, _cuda(xq, dtype), _cuda(wq, dtype), relu=relu)
    yg = y.cpu().numpy()
    r = stride.bit_length() - 1  # stride 2^r
    rng = np.random.default_rng(7)
    if not big:
        pre = oracle.conv_fwd(nb, xq, wq)
        if stride > 1:
            pre = oracle.renew(ref.labels(l - r), pre)
        dy = _mask_ambiguous(dy, pre, relu)
        assert_f32_close(yg, oracle.relu_fwd(pre) if relu else pre, f"{tag} y")
        dye = oracle.relu_bwd(pre, dy) if relu else dy
    else:
        assert stride == 1 and not relu
        want, rows = _tiles(n_in, 16)
        assert_f32_close(yg[rows], oracle.conv_fwd(nb, xq, wq, rows=rows), f"{tag} y tiles")
        b = rng.standard_normal(cout)
        _assert_proj(yg, b, oracle.conv_fwd(nb, xq, wq @ b[:, None])[:, 0], f"{tag} y proj")
        dye = dy
    dx, dw = oc.oc_conv_bwd(tree, l, K, stride, _cuda(xq, dtype), _cuda(wq, dtype), _cuda(dy),
                            y=y, relu=relu)
    dxg, dwg = dx.cpu().numpy(), dw.cpu().numpy()
    if dtype == torch.bfloat16:  # the bf16 backward multiplies dy rounded to bf16
        dye = bf16_round(dye)
    dyh = dye if stride == 1 else oracle.renew_bwd(ref.labels(l - r), dye, nb.shape[0])
    if not big:
        assert_f32_close(dxg, oracle.conv_bwd_data(nb, dyh, wq, n_in), f"{tag} dx")
        rule = assert_dw_close(dwg, oracle.conv_bwd_weight(nb, xq, dyh, K3), f"{tag} dw")
    else:
        assert_f32_close(dxg[rows], oracle.conv_bwd_data(nb, dyh, wq, n_in, want=want)[rows],
                         f"{tag} dx tiles")
        bi = rng.standard_normal(cin)
        wb = np.einsum("kio,i->ko", wq.astype(np.float64), bi)[:, None, :]  # [K3][1][cout]
        _assert_proj(dxg, bi, oracle.conv_bwd_data(nb, dyh, wb, n_in)[:, 0], f"{tag} dx proj")
        # every entry of dW through both channel projections, and exact entries
        # in every (tap, 16 x 16 channel) block
        bo = rng.standard_normal(cout)
        datol = 1e-5 * max(1.0, float(np.sqrt(np.mean(dwg.astype(np.float64) ** 2))))
        _assert_proj(dwg.reshape(-1, cout), bo,
                     oracle.conv_bwd_weight(nb, xq, dyh @ bo[:, None], K3).reshape(-1),
                     f"{tag} dw proj out", atol=datol)
        _assert_proj(dwg.transpose(0, 2, 1).reshape(-1, cin), bi,
                     oracle.conv_bwd_weight(nb, xq @ bi[:, None], dyh, K3).reshape(-1),
                     f"{tag} dw proj in", atol=datol)
        ent = _dw_block_entries(K3, cin, cout, rng)
        rule = assert_dw_close(dwg.ravel()[ent],
                               oracle.conv_bwd_weight(nb, xq, dyh, K3, entries=ent),
                               f"{tag} dw blocks")
    print(f"[{tag}] dw rule: {rule}", flush=True)
    return y


def _check_deconv_full(ref, tree, l, K, stride, x, w, dy, tag):
    oc = _oc()
    n_out = ref.num(l)
    print(f"[{tag}] deconv d{l} K{K} s{stride} {x.shape[1]}->{w.shape[1]} rows {n_out}", flush=True)
    y = oc.oc_deconv_fwd(tree, l, K, stride, _cuda(x), _cuda(w))
    dx, dw = oc.oc_deconv_bwd(tree, l, K, stride, _cuda(x), _cuda(w), _cuda(dy))
    if stride == 1:
        nb = ref.neighbors(l, K)
        yr = oracle.deconv_fwd(nb, x, w, n_out)
        dxr, dwr = oracle.deconv_bwd(nb, x, w, dy)
    else:
        yr = oracle.deconv_s2_fwd(ref, l, x, w)
        dxr, dwr = oracle.deconv_s2_bwd(ref, l, x, w, dy)
    assert_f32_close(y.cpu().numpy(), yr, f"{tag} y")
    assert_f32_close(dx.cpu().numpy(), dxr, f"{tag} dx")
    rule = assert_dw_close(dw.cpu().numpy(), dwr, f"{tag} dw")
    print(f"[{tag}] dw rule: {rule}", flush=True)


@pytest.mark.parametrize("name", ["sphere_d5", "net_d5", "net_d6", "deep_d8", "wide_d7", "seg_d6",
                                  "gpool_d6", "s4_d6"])
def test_workload_full_size(name):
    oc = _oc()
    w_ = synth.WORKLOADS[name]
    pts, nrm, offs = synth.make_points(w_)
    ref, tree = _trees(pts, nrm, offs, w_.depth, w_.full_depth)
    first = True
    for li, L in enumerate(w_.layers):
        l = L.depth
        if L.op == "conv":
            if first and w_.signal_input:
                x = ref.signal  # the oracle's averaged normals
            else:
                x = synth.make_features([w_.seed_id, 3000 + li], ref.num(l), L.cin)
            first = False
            K = L.ksize
            w = synth.make_weights(w_, li, K, L.cin, L.cout)
            n_out = ref.num(l - (L.stride.bit_length() - 1))
            dy = synth.make_upstream(w_, li, n_out, L.cout)
            _check_conv_full(ref, tree, l, K, L.stride, x, w, L.relu, dy, f"{name}/{li}")
            nxt = w_.layers[li + 1] if li + 1 < len(w_.layers) else None
            if nxt is not None and nxt.op == "pool" and L.stride == 1 and L.dtype != "bf16":
                # the network runs this pair as one conv + pool call
                print(f"[{name}/{li}] conv + pool d{l}", flush=True)
                _check_conv_pool(ref, tree, l, K, x, w, L.relu, f"{name}/{li}+pool")
            if L.dtype == "bf16":
                _check_conv_full(ref, tree, l, K, L.stride, x, w, L.relu, dy, f"{name}/{li}/bf16",
                                 dtype=torch.bfloat16)
        elif L.op == "deconv":
            n_in = ref.num(l) if L.stride == 1 else ref.num(l - 1)
            x = synth.make_features([w_.seed_id, 3000 + li], n_in, L.cin)
            w = synth.make_weights(w_, li, L.ksize, L.cout, L.cin)
            dy = synth.make_upstream(w_, li, ref.num(l), L.cout)
            _check_deconv_full(ref, tree, l, L.ksize, L.stride, x, w, dy, f"{name}/{li}")
        elif L.op == "gpool":
            x = np.maximum(synth.make_features([w_.seed_id, 3000 + li], ref.num(l), L.cin), 0)
            r = L.stride.bit_length() - 1
            print(f"[{name}/{li}] gpool {L.mode} K{L.ksize} s{L.stride} d{l} C{L.cin}", flush=True)
            mode = oc.OC_POOL_MAX if L.mode == "max" else oc.OC_POOL_AVG
            rmode = oracle.POOL_MAX if L.mode == "max" else oracle.POOL_AVG
            y, sw = oc.oc_gpool_fwd(tree, l, L.ksize, mode, _cuda(x), stride=L.stride)
            dy = synth.make_upstream(w_, li, ref.num(l - r), L.cin)
            dx = oc.oc_gpool_bwd(tree, l, L.ksize, mode, _cuda(dy), sw, stride=L.stride)
            if r == 0:
                nb = ref.neighbors(l, L.ksize)
                yr, swr = oracle.gpool_fwd(nb, x, rmode)
                dxr = oracle.gpool_bwd(nb, dy, swr, ref.num(l), rmode)
            else:
                yr, swr = oracle.gpool_sr_fwd(ref, l, x, rmode, L.stride)
                dxr = oracle.gpool_sr_bwd(ref, l, dy, swr, ref.num(l), rmode, L.stride)
            if L.mode == "max":
                np.testing.assert_array_equal(y.cpu().numpy(), yr)
                np.testing.assert_array_equal(sw.cpu().numpy(), swr)
            else:
                assert_f32_close(y.cpu().numpy(), yr, f"{name}/{li} y")
            assert_f32_close(dx.cpu().numpy(), dxr, f"{name}/{li} dx")
        elif L.op == "pool":
            x = synth.make_features([w_.seed_id, 3000 + li], ref.num(l), L.cin)
            print(f"[{name}/{li}] pool d{l} C{L.cin}", flush=True)
            y, sw = oc.oc_pool_fwd(tree, l, _cuda(x))
            yr, swr = oracle.pool_fwd(ref.labels(l - 1), x)
            np.testing.assert_array_equal(y.cpu().numpy(), yr)
            np.testing.assert_array_equal(sw.cpu().numpy(), swr)
            dy = synth.make_upstream(w_, li, ref.num(l - 1), L.cin)
            np.testing.assert_array_equal(oc.oc_pool_bwd(tree, l, _cuda(dy), sw).cpu().numpy(),
                                          oracle.pool_bwd(ref.labels(l - 1), dy, swr, ref.num(l)))
            # the ReLU-masked routing the network's backward uses (pool_bwd with
            # the pooled output of a ReLU'd input)
            a = np.maximum(x, 0.0)
            ya, swa = oc.oc_pool_fwd(tree, l, _cuda(a))
            _, swar = oracle.pool_fwd(ref.labels(l - 1), a)
            np.testing.assert_array_equal(swa.cpu().numpy(), swar)
            np.testing.assert_array_equal(
                oc.oc_pool_bwd(tree, l, _cuda(dy), swa, y=ya).cpu().numpy(),
                oracle.relu_bwd(x, oracle.pool_bwd(ref.labels(l - 1), dy, swar, ref.num(l))))
        elif L.op == "unpool":
            x = synth.make_features([w_.seed_id, 3000 + li], ref.num(l), L.cin)
            _, sw = oc.oc_pool_fwd(tree, l, _cuda(x))
            _, swr = oracle.pool_fwd(ref.labels(l - 1), x)
            xp = synth.make_features([w_.seed_id, 4000 + li], ref.num(l - 1), L.cin)
            print(f"[{name}/{li}] unpool d{l} C{L.cin}", flush=True)
            np.testing.assert_array_equal(oc.oc_unpool_fwd(tree, l, _cuda(xp), sw).cpu().numpy(),
                                          oracle.unpool_fwd(ref.labels(l - 1), xp, swr, ref.num(l)))
            g = synth.make_upstream(w_, li, ref.num(l), L.cin)
            np.testing.assert_array_equal(oc.oc_unpool_bwd(tree, l, _cuda(g), sw).cpu().numpy(),
                                          oracle.unpool_bwd(ref.labels(l - 1), g, swr))


@pytest.mark.parametrize("n,offset", [(0, 0), (1, 0), (4099, 0), (4099, 1), (1 << 20, 0)])
def test_round_bf16(n, offset):
    """oc_round_bf16 against torch's own f32 -> bf16 conversion (round to
    nearest, ties to even) on the CPU: bit-exact for every non-NaN value,
    ties, subnormals, signed zeros, values that round up to infinity and the
    infinities included; NaN stays NaN.  offset 1 takes the element path."""
    g = torch.Generator().manual_seed(n + offset)
    v = torch.randn(n + offset, generator=g) * torch.exp2(torch.randint(-140, 128, (n + offset,),
                                                                          generator=g).float())
    special = torch.tensor([0.0, -0.0, float("inf"), float("-inf"), float("nan"),
                            3.4028235e38, -3.4028235e38, 1e-45, -1e-45, 1.0 + 2 ** -8,
                            1.0 + 3 * 2 ** -8, 1.0 + 2 ** -8 + 2 ** -20])
    k = min(len(special), n)
    v[offset:offset + k] = special[:k]
    ties = torch.randint(0, 1 << 31, (n + offset,), generator=g, dtype=torch.int64)
    v = torch.where(torch.arange(n + offset) % 5 == 4,  # exact ties of both parities
                    ((ties & ~0xffff) | 0x8000).to(torch.int32).view(torch.float32), v)
    x = v.cuda()[offset:]
    y = _oc().oc_round_bf16(x)
    assert y.dtype == torch.bfloat16 and y.shape == x.shape
    got = y.cpu()
    want = v[offset:].to(torch.bfloat16)
    nan = torch.isnan(want)
    assert torch.equal(torch.isnan(got), nan)
    assert torch.equal(got[~nan].view(torch.int16), want[~nan].view(torch.int16))
