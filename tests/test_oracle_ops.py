"""Pins of the CPU oracle's neighbour search, convolution, pooling and
unpooling (Sec. 3.2) against brute force and dense float64 torch routines.

Octree convolution with absent neighbours read as zero is a dense 3D
cross-correlation evaluated at the octants that exist, with zeros wherever no
octant exists; 2x2x2 max-pooling is dense max_pool3d read at the non-empty
parents.  These dense forms are computed here with torch on the CPU in float64.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth



def _coords(tree, l):
    keys = tree.keys(l).astype(np.int64)
    b = keys >> 24
    k = keys & 0xFFFFFF
    x = np.zeros_like(k)
    y = np.zeros_like(k)
    z = np.zeros_like(k)
    for i in range(l):
        g = (k >> (3 * (l - 1 - i))) & 7
        x, y, z = 2 * x + (g >> 2), 2 * y + ((g >> 1) & 1), 2 * z + (g & 1)
    return b, x, y, z


def _scatter(tree, l, feat):
    """Dense grid [B][C][2^l]^3 holding feat at the existing octants, 0 elsewhere."""
    b, x, y, z = _coords(tree, l)
    s = 2 ** l
    g = torch.zeros((tree.batch, feat.shape[1], s, s, s), dtype=torch.float64)
    g[b, :, x, y, z] = feat
    return g


def _gather(tree, l, grid):
    b, x, y, z = _coords(tree, l)
    return grid[b, :, x, y, z]


def _torch_weight(w):
    K = round(w.shape[0] ** (1 / 3))
    wt = torch.as_tensor(np.asarray(w, np.float64))  # [K^3][cin][cout]
    return wt.reshape(K, K, K, w.shape[1], w.shape[2]).permute(4, 3, 0, 1, 2).contiguous()


def _tree(seed, B=2, depth=4, full=2, n=150, spread="union"):
    pts, nrm, offs = synth.random_cloud(seed, B, n, spread)
    return oracle.Octree(pts, nrm, offs, depth, full)


CASES = [  # seed, B, depth, full, K
    (11, 2, 4, 2, 3),
    (12, 1, 3, 0, 3),
    (13, 3, 4, 1, 5),
    (14, 1, 3, 3, 3),  # complete octree: dense conv everywhere
]


@pytest.mark.parametrize("seed,B,depth,full,K", CASES)
def test_neighbors_brute_force(seed, B, depth, full, K):
    t = _tree(seed, B, depth, full)
    l = depth
    nb = t.neighbors(l, K)
    b, x, y, z = _coords(t, l)
    r = (K - 1) // 2
    offs = [(dx, dy, dz) for dx in range(-r, r + 1) for dy in range(-r, r + 1) for dz in range(-r, r + 1)]
    for i in range(len(b)):
        for k, (dx, dy, dz) in enumerate(offs):
            hit = np.nonzero((b == b[i]) & (x == x[i] + dx) & (y == y[i] + dy) & (z == z[i] + dz))[0]
            assert nb[i, k] == (hit[0] if len(hit) else -1)
    # stride 2 rows are the stride-1 rows of the first siblings
    nb2 = t.neighbors(l, K, stride=2)
    np.testing.assert_array_equal(nb2, nb[::8])


def test_union_neighbourhood_size():
    # Sec. 3.2: the 8 siblings of a group touch (K+1)^3 distinct positions
    t = _tree(21, 1, 3, 3)  # complete: interior groups see every position
    for K in (3, 5):
        nb = t.neighbors(3, K)
        b, x, y, z = _coords(t, 3)
        sizes = []
        for g in range(len(nb) // 8):
            gx, gy, gz = x[8 * g] // 2, y[8 * g] // 2, z[8 * g] // 2
            if 1 <= gx <= 2 and 1 <= gy <= 2 and 1 <= gz <= 2:
                sizes.append(len(set(nb[8 * g:8 * g + 8].ravel().tolist()) - {-1}))
        assert sizes and all(s == (K + 1) ** 3 for s in sizes)


@pytest.mark.parametrize("seed,B,depth,full,K", CASES)
def test_conv_fwd_equals_dense_conv3d(seed, B, depth, full, K):
    t = _tree(seed, B, depth, full)
    l = depth
    cin, cout = 5, 7
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((t.num(l), cin))
    w = rng.standard_normal((K ** 3, cin, cout))
    y = oracle.conv_fwd(t.neighbors(l, K), x, w)
    dense = F.conv3d(_scatter(t, l, torch.as_tensor(x)), _torch_weight(w), padding=(K - 1) // 2)
    ref = _gather(t, l, dense).numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)
    # row subset
    rows = rng.choice(t.num(l), size=min(17, t.num(l)), replace=False)
    np.testing.assert_allclose(oracle.conv_fwd(t.neighbors(l, K), x, w, rows=rows), ref[rows], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed,B,depth,full,K", CASES)
def test_conv_bwd_equals_dense_autograd(seed, B, depth, full, K):
    t = _tree(seed, B, depth, full)
    l = depth
    cin, cout = 4, 6
    rng = np.random.default_rng(100 + seed)
    x = rng.standard_normal((t.num(l), cin))
    w = rng.standard_normal((K ** 3, cin, cout))
    dy = rng.standard_normal((t.num(l), cout))
    nb = t.neighbors(l, K)
    dx = oracle.conv_bwd_data(nb, dy, w, t.num(l))
    dw = oracle.conv_bwd_weight(nb, x, dy, K ** 3)

    xt = torch.as_tensor(x).requires_grad_(True)
    wt = torch.as_tensor(w).requires_grad_(True)
    K_ = K
    wd = wt.reshape(K_, K_, K_, cin, cout).permute(4, 3, 0, 1, 2)
    out = _gather(t, l, F.conv3d(_scatter(t, l, xt), wd, padding=(K - 1) // 2))
    out.backward(torch.as_tensor(dy))
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-11, atol=1e-11)
    # want-mask and entry subsets agree with the full results
    want = rng.random(t.num(l)) < 0.3
    dxm = oracle.conv_bwd_data(nb, dy, w, t.num(l), want=want)
    np.testing.assert_array_equal(dxm[want], dx[want])
    assert np.all(dxm[~want] == 0)
    ent = rng.choice(w.size, size=11, replace=False)
    np.testing.assert_allclose(oracle.conv_bwd_weight(nb, x, dy, K ** 3, entries=ent), dw.ravel()[ent], rtol=1e-12, atol=1e-12)


def test_conv_adjoint_and_finite_difference():
    t = _tree(31, 2, 4, 2)
    l, K, cin, cout = 4, 3, 3, 4
    rng = np.random.default_rng(5)
    nb = t.neighbors(l, K)
    x = rng.standard_normal((t.num(l), cin))
    w = rng.standard_normal((K ** 3, cin, cout))
    v = rng.standard_normal((t.num(l), cout))
    # <conv(x), v> = <x, conv_bwd_data(v)> = <w, conv_bwd_weight(x, v)>
    lhs = np.sum(oracle.conv_fwd(nb, x, w) * v)
    assert np.isclose(lhs, np.sum(x * oracle.conv_bwd_data(nb, v, w, t.num(l))), rtol=1e-12)
    assert np.isclose(lhs, np.sum(w * oracle.conv_bwd_weight(nb, x, v, K ** 3)), rtol=1e-12)
    # central differences of L = <conv(x), v> along random directions
    dx = oracle.conv_bwd_data(nb, v, w, t.num(l))
    h = 1e-6
    for _ in range(3):
        e = rng.standard_normal(x.shape)
        fd = (np.sum(oracle.conv_fwd(nb, x + h * e, w) * v) - np.sum(oracle.conv_fwd(nb, x - h * e, w) * v)) / (2 * h)
        assert np.isclose(fd, np.sum(dx * e), rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("seed,B,depth,full", [(41, 2, 4, 2), (42, 1, 3, 0), (43, 3, 4, 1)])
def test_stride2_equals_dense_strided_conv(seed, B, depth, full):
    t = _tree(seed, B, depth, full)
    l, K, cin, cout = depth, 3, 4, 5
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((t.num(l), cin))
    w = rng.standard_normal((K ** 3, cin, cout))
    y = oracle.conv_s2_fwd(t, l, x, w)
    dense = F.conv3d(_scatter(t, l, torch.as_tensor(x)), _torch_weight(w), stride=2, padding=1)
    ref = _gather(t, l - 1, dense).numpy()
    ref[t.labels(l - 1) == 0] = 0  # empty parents get no output (Sec. 3.2, Fig. 2(d))
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)
    # backward vs autograd of the same dense form
    dy = rng.standard_normal((t.num(l - 1), cout))
    dx, dw = oracle.conv_s2_bwd(t, l, x, w, dy)
    xt = torch.as_tensor(x).requires_grad_(True)
    wt = torch.as_tensor(w).requires_grad_(True)
    wd = wt.reshape(K, K, K, cin, cout).permute(4, 3, 0, 1, 2)
    out = _gather(t, l - 1, F.conv3d(_scatter(t, l, xt), wd, stride=2, padding=1))
    mask = torch.as_tensor((t.labels(l - 1) > 0).astype(np.float64))[:, None]
    (out * mask).backward(torch.as_tensor(dy))
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("seed,B,depth,full", [(51, 2, 4, 2), (52, 1, 3, 0), (53, 3, 3, 1)])
def test_pool_unpool_equal_dense(seed, B, depth, full):
    t = _tree(seed, B, depth, full)
    l, c = depth, 6
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((t.num(l), c))  # continuous: no ties
    y, sw = oracle.pool_fwd(t.labels(l - 1), x)
    dense, idx = F.max_pool3d(_scatter(t, l, torch.as_tensor(x)), 2, return_indices=True)
    ref = _gather(t, l - 1, dense).numpy()
    nz = t.labels(l - 1) > 0
    ref[~nz] = 0
    np.testing.assert_array_equal(y, ref)
    # switch = child index 4 (x&1) + 2 (y&1) + (z&1) of the dense argmax
    s = 2 ** l
    fi = _gather(t, l - 1, idx).numpy()[nz]
    ix, iy, iz = fi // (s * s), (fi // s) % s, fi % s
    np.testing.assert_array_equal(sw[t.labels(l - 1)[nz] - 1], 4 * (ix & 1) + 2 * (iy & 1) + (iz & 1))
    # pooling backward and unpooling vs dense max_unpool3d / autograd
    dy = rng.standard_normal((t.num(l - 1), c))
    dx = oracle.pool_bwd(t.labels(l - 1), dy, sw, t.num(l))
    xt = torch.as_tensor(x).requires_grad_(True)
    out = _gather(t, l - 1, F.max_pool3d(_scatter(t, l, xt), 2))
    (out * torch.as_tensor(nz.astype(np.float64))[:, None]).backward(torch.as_tensor(dy))
    np.testing.assert_array_equal(dx, xt.grad.numpy())
    u = oracle.unpool_fwd(t.labels(l - 1), dy, sw, t.num(l))
    dyz = dy.copy()
    dyz[~nz] = 0
    up = F.max_unpool3d(_scatter(t, l - 1, torch.as_tensor(dyz)), idx, 2, output_size=(s, s, s))
    np.testing.assert_array_equal(u, _gather(t, l, up).numpy())
    # unpool backward is the adjoint of unpool forward
    g = rng.standard_normal((t.num(l), c))
    ub = oracle.unpool_bwd(t.labels(l - 1), g, sw)
    assert np.isclose(np.sum(u * g), np.sum(dyz * ub), rtol=1e-12)
    assert np.all(ub[~nz] == 0)


def test_pool_tie_takes_first_child():
    # one group of 8 siblings, with equal maxima at children 2 and 5
    pts = np.array([[0.3, 0.3, 0.3]], np.float32)
    t = oracle.Octree(pts, np.ones((1, 3), np.float32), [0, 1], 1, 0)
    x = np.array([[0.], [1.], [3.], [-1.], [2.], [3.], [0.], [3.]])
    y, sw = oracle.pool_fwd(t.labels(0), x)
    assert y.tolist() == [[3.0]] and sw.tolist() == [[2]]


def test_relu():
    x = np.array([-1.0, 0.0, 2.0])
    assert oracle.relu_fwd(x).tolist() == [0.0, 0.0, 2.0]
    assert oracle.relu_bwd(x, np.array([5.0, 6.0, 7.0])).tolist() == [0.0, 0.0, 7.0]


# Deconvolution (Sec. 3.2): the transpose of the octree convolution.  Dense
# form: conv_transpose3d of the input scattered to the grid (zero where no
# octant exists), read at the existing octants; its weight tensor is the one
# of the convolution cout -> cin it transposes.

@pytest.mark.parametrize("seed,B,depth,full,K", CASES)
def test_deconv_equals_dense_conv_transpose3d(seed, B, depth, full, K):
    t = _tree(seed, B, depth, full)
    l = depth
    cin, cout = 6, 5  # deconv channels; w [K^3][cout][cin]
    rng = np.random.default_rng(200 + seed)
    x = rng.standard_normal((t.num(l), cin))
    w = rng.standard_normal((K ** 3, cout, cin))
    nb = t.neighbors(l, K)
    y = oracle.deconv_fwd(nb, x, w, t.num(l))
    xt = torch.as_tensor(x).requires_grad_(True)
    wt = torch.as_tensor(w).requires_grad_(True)
    wd = wt.reshape(K, K, K, cout, cin).permute(4, 3, 0, 1, 2)  # [cin][cout][K][K][K]
    out = _gather(t, l, F.conv_transpose3d(_scatter(t, l, xt), wd, padding=(K - 1) // 2))
    np.testing.assert_allclose(y, out.detach().numpy(), rtol=1e-12, atol=1e-12)
    dy = rng.standard_normal((t.num(l), cout))
    out.backward(torch.as_tensor(dy))
    dx, dw = oracle.deconv_bwd(nb, x, w, dy)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-11, atol=1e-11)
    # subsets agree with the full results
    want = rng.random(t.num(l)) < 0.3
    np.testing.assert_array_equal(oracle.deconv_fwd(nb, x, w, t.num(l), want=want)[want], y[want])
    rows = rng.choice(t.num(l), size=min(9, t.num(l)), replace=False)
    ent = rng.choice(w.size, size=7, replace=False)
    dxs, dws = oracle.deconv_bwd(nb, x, w, dy, rows=rows, entries=ent)
    np.testing.assert_allclose(dxs, dx[rows], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dws, dw.ravel()[ent], rtol=1e-12, atol=1e-12)


def test_deconv_is_adjoint_of_conv():
    # <conv(a; w), b> = <a, deconv(b; w)> for the same weight tensor
    t = _tree(61, 2, 4, 2)
    l, K, c1, c2 = 4, 3, 3, 5
    rng = np.random.default_rng(61)
    nb = t.neighbors(l, K)
    w = rng.standard_normal((K ** 3, c1, c2))  # conv c1 -> c2, deconv c2 -> c1
    a = rng.standard_normal((t.num(l), c1))
    b = rng.standard_normal((t.num(l), c2))
    lhs = np.sum(oracle.conv_fwd(nb, a, w) * b)
    assert np.isclose(lhs, np.sum(a * oracle.deconv_fwd(nb, b, w, t.num(l))), rtol=1e-12)


@pytest.mark.parametrize("seed,B,depth,full,stride", [
    (71, 2, 4, 2, 2), (72, 1, 3, 0, 2), (73, 3, 4, 1, 2),
    (74, 2, 4, 2, 4), (75, 2, 4, 0, 8), (76, 1, 3, 1, 8)])
def test_deconv_sr_equals_dense_strided_transpose(seed, B, depth, full, stride):
    """Stride 2^r deconvolution (depth l-r -> l): dense conv_transpose3d with
    stride 2^r, padding 1 and output_padding 2^r - 1 (the transpose of the
    dense conv3d(stride=2^r, padding=1) that pins the strided convolution)."""
    t = _tree(seed, B, depth, full)
    r = stride.bit_length() - 1
    l, K, cin, cout = depth, 3, 5, 4
    rng = np.random.default_rng(300 + seed)
    x = rng.standard_normal((t.num(l - r), cin))
    w = rng.standard_normal((K ** 3, cout, cin))
    y = oracle.deconv_sr_fwd(t, l, x, w, stride)
    nz = torch.as_tensor((t.labels(l - r) > 0).astype(np.float64))[:, None]
    xt = torch.as_tensor(x).requires_grad_(True)
    wt = torch.as_tensor(w).requires_grad_(True)
    wd = wt.reshape(K, K, K, cout, cin).permute(4, 3, 0, 1, 2)
    # rows of empty octants carry nothing (the strided convolution has no output there)
    out = _gather(t, l, F.conv_transpose3d(_scatter(t, l - r, xt * nz), wd, stride=stride,
                                           padding=1, output_padding=stride - 1))
    np.testing.assert_allclose(y, out.detach().numpy(), rtol=1e-12, atol=1e-12)
    dy = rng.standard_normal((t.num(l), cout))
    out.backward(torch.as_tensor(dy))
    dx, dw = oracle.deconv_sr_bwd(t, l, x, w, dy, stride)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-11, atol=1e-11)
    assert np.all(dx[t.labels(l - r) == 0] == 0)
    if stride == 2:  # the stride-2 names are the same functions
        np.testing.assert_array_equal(oracle.deconv_s2_fwd(t, l, x, w), y)


# General pooling (Sec. 3.2, last paragraph of "Pooling"): the stride-1 K^3
# neighbourhood with absent neighbours read as zero.  Dense forms: the grid of
# the octants' features (zeros elsewhere), zero-padded, then max_pool3d /
# avg_pool3d (count_include_pad) with stride 1, read at the octants.

@pytest.mark.parametrize("seed,B,depth,full,K", CASES)
def test_gpool_equals_dense_pooling(seed, B, depth, full, K):
    t = _tree(seed, B, depth, full)
    l, c, r = depth, 5, (K - 1) // 2
    rng = np.random.default_rng(400 + seed)
    x = rng.standard_normal((t.num(l), c))  # continuous: ties only among zeros
    nb = t.neighbors(l, K)
    dy = rng.standard_normal((t.num(l), c))
    # max
    y, sw = oracle.gpool_fwd(nb, x, oracle.POOL_MAX)
    xt = torch.as_tensor(x).requires_grad_(True)
    g = F.pad(_scatter(t, l, xt), (r,) * 6, value=0.0)
    dense, idx = F.max_pool3d(g, K, stride=1, return_indices=True)
    out = _gather(t, l, dense)
    np.testing.assert_array_equal(y, out.detach().numpy())
    # the switch names the dense argmax cell (a zero cell when POOL_ABSENT)
    s = 2 ** l + 2 * r
    b, X, Y, Z = _coords(t, l)
    fi = _gather(t, l, idx).numpy()
    ix, iy, iz = fi // (s * s), (fi // s) % s, fi % s
    tap = ((ix - X[:, None]) * K + (iy - Y[:, None])) * K + (iz - Z[:, None])
    present = sw != oracle.POOL_ABSENT
    np.testing.assert_array_equal(sw[present], tap[present])
    assert np.all(y[~present] == 0)
    out.backward(torch.as_tensor(dy))
    np.testing.assert_allclose(oracle.gpool_bwd(nb, dy, sw, t.num(l), oracle.POOL_MAX),
                               xt.grad.numpy(), rtol=1e-12, atol=1e-12)
    # average
    ya, swa = oracle.gpool_fwd(nb, x, oracle.POOL_AVG)
    assert swa is None
    xt = torch.as_tensor(x).requires_grad_(True)
    out = _gather(t, l, F.avg_pool3d(_scatter(t, l, xt), K, stride=1, padding=r,
                                     count_include_pad=True))
    np.testing.assert_allclose(ya, out.detach().numpy(), rtol=1e-12, atol=1e-12)
    out.backward(torch.as_tensor(dy))
    np.testing.assert_allclose(oracle.gpool_bwd(nb, dy, None, t.num(l), oracle.POOL_AVG),
                               xt.grad.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed,B,depth,full,stride", [
    (41, 2, 4, 2, 2), (42, 1, 3, 0, 2), (43, 3, 4, 1, 4), (44, 2, 4, 2, 8), (45, 1, 3, 3, 2)])
def test_gpool_strided_equals_dense_pooling(seed, B, depth, full, stride):
    """Strided general pooling: dense zero-padded max_pool3d / avg_pool3d
    (count_include_pad) with kernel 3 and stride 2^r, read at the non-empty
    depth-(l-r) octants (zero rows at empty ones), and their autograd."""
    t = _tree(seed, B, depth, full)
    l, c = depth, 4
    r = stride.bit_length() - 1
    rng = np.random.default_rng(500 + seed)
    x = rng.standard_normal((t.num(l), c))
    dy = rng.standard_normal((t.num(l - r), c))
    nz = t.labels(l - r) > 0
    y, sw = oracle.gpool_sr_fwd(t, l, x, oracle.POOL_MAX, stride)
    xt = torch.as_tensor(x).requires_grad_(True)
    g = F.pad(_scatter(t, l, xt), (1,) * 6, value=0.0)
    dense, idx = F.max_pool3d(g, 3, stride=stride, return_indices=True)
    out = _gather(t, l - r, dense) * torch.as_tensor(nz.astype(np.float64))[:, None]
    np.testing.assert_array_equal(y, out.detach().numpy())
    sp = 2 ** l + 2
    b, X, Y, Z = _coords(t, l - r)
    fi = _gather(t, l - r, idx).numpy()
    ix, iy, iz = fi // (sp * sp), (fi // sp) % sp, fi % sp
    tap = ((ix - stride * X[:, None]) * 3 + (iy - stride * Y[:, None])) * 3 + (iz - stride * Z[:, None])
    present = sw != oracle.POOL_ABSENT
    np.testing.assert_array_equal(sw[present], tap[present])
    assert np.all(y[~present] == 0) and np.all(sw[~nz] == oracle.POOL_ABSENT)
    out.backward(torch.as_tensor(dy))
    np.testing.assert_allclose(oracle.gpool_sr_bwd(t, l, dy, sw, t.num(l), oracle.POOL_MAX, stride),
                               xt.grad.numpy(), rtol=1e-12, atol=1e-12)
    ya, swa = oracle.gpool_sr_fwd(t, l, x, oracle.POOL_AVG, stride)
    assert swa is None
    xt = torch.as_tensor(x).requires_grad_(True)
    out = _gather(t, l - r, F.avg_pool3d(_scatter(t, l, xt), 3, stride=stride, padding=1,
                                         count_include_pad=True))
    out = out * torch.as_tensor(nz.astype(np.float64))[:, None]
    np.testing.assert_allclose(ya, out.detach().numpy(), rtol=1e-12, atol=1e-12)
    out.backward(torch.as_tensor(dy))
    np.testing.assert_allclose(oracle.gpool_sr_bwd(t, l, dy, None, t.num(l), oracle.POOL_AVG,
                                                   stride),
                               xt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_gpool_hand_case():
    # one group of 8 siblings at depth 1 (the whole cube): every child sees the
    # other seven plus 19 absent (outside-cube) neighbours
    pts = np.array([[0.3, 0.3, 0.3]], np.float32)
    t = oracle.Octree(pts, np.ones((1, 3), np.float32), [0, 1], 1, 0)
    x = np.array([[-1.], [-2.], [-3.], [-4.], [-5.], [-6.], [-7.], [-0.5]])
    nb = t.neighbors(1, 3)
    y, sw = oracle.gpool_fwd(nb, x, oracle.POOL_MAX)
    assert np.all(y == 0) and np.all(sw == oracle.POOL_ABSENT)  # an absent zero beats them
    ya, _ = oracle.gpool_fwd(nb, x, oracle.POOL_AVG)
    np.testing.assert_allclose(ya[:, 0], np.full(8, x.sum() / 27))  # all 8 in every window
    y2, sw2 = oracle.gpool_fwd(nb, x + 10, oracle.POOL_MAX)
    # child 7 (x=y=z=1) is the maximum; seen from child 0 at offset (+1,+1,+1): tap 26
    assert y2[0, 0] == 9.5 and sw2[0, 0] == 26 and sw2[7, 0] == 13


# Stride 2^r (Sec. 3.2): the convolution at the first depth-l position of the
# sub-tree of height r below each non-empty octant of depth l-r, i.e. dense
# conv3d with stride 2^r read at the depth-(l-r) octants, 0 at empty ones.

@pytest.mark.parametrize("seed,B,depth,full,stride", [(81, 2, 4, 2, 4), (82, 1, 4, 0, 4),
                                                      (83, 3, 5, 1, 4), (84, 2, 5, 2, 8)])
def test_stride_2r_equals_dense_strided_conv(seed, B, depth, full, stride):
    t = _tree(seed, B, depth, full, n=300)
    r = stride.bit_length() - 1
    l, K, cin, cout = depth, 3, 3, 4
    rng = np.random.default_rng(500 + seed)
    x = rng.standard_normal((t.num(l), cin))
    w = rng.standard_normal((K ** 3, cin, cout))
    y = oracle.conv_sr_fwd(t, l, x, w, stride)
    xt = torch.as_tensor(x).requires_grad_(True)
    wt = torch.as_tensor(w).requires_grad_(True)
    wd = wt.reshape(K, K, K, cin, cout).permute(4, 3, 0, 1, 2)
    out = _gather(t, l - r, F.conv3d(_scatter(t, l, xt), wd, stride=stride, padding=1))
    nz = torch.as_tensor((t.labels(l - r) > 0).astype(np.float64))[:, None]
    np.testing.assert_allclose(y, (out * nz).detach().numpy(), rtol=1e-12, atol=1e-12)
    dy = rng.standard_normal((t.num(l - r), cout))
    (out * nz).backward(torch.as_tensor(dy))
    dx, dw = oracle.conv_sr_bwd(t, l, x, w, dy, stride)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-11, atol=1e-11)
    if stride == 2:  # the same as the first-sibling form
        np.testing.assert_array_equal(t.neighbors(l, K, 2), t.neighbors(l, K)[::8])


def test_stride_2_neighbors_are_first_siblings():
    t = _tree(85, 2, 4, 2)
    np.testing.assert_array_equal(t.neighbors(4, 3, stride=2), t.neighbors(4, 3)[::8])
    np.testing.assert_array_equal(t.neighbors(4, 5, stride=2), t.neighbors(4, 5)[::8])
