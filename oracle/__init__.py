"""ctypes wrapper of the plain CPU oracle (``ocref.cpp``).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by the package smoke check
and by the bench's CPU-baseline leg, never by the product path.  It shares
no code with the HIP library.  Inputs are numpy arrays; floating-point inputs
are widened to float64 and every result is float64 (integers stay exact).
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ocref.cpp")
_LIB = os.path.join(_HERE, "libocref.so")

OK, ERR_ARG, ERR_RANGE = 0, 1, 2


def build(force: bool = False) -> str:
    """Compile the oracle with the host compiler (g++), never hipcc."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["g++", "-O3", "-std=c++17", "-fopenmp", "-shared", "-fPIC", _SRC, "-o", tmp]
        )
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = C.CDLL(_LIB)
        p, i32, i64 = C.c_void_p, C.c_int32, C.c_int64
        sig = {
            "ocref_build": [p, p, p, i32, i32, i32, C.POINTER(p)],
            "ocref_level_size": [p, i32, C.POINTER(i64), C.POINTER(i64)],
            "ocref_level": [p, i32, p, p, p],
            "ocref_signal": [p, p],
            "ocref_neighbors": [p, i32, i32, i32, p],
            "ocref_conv_fwd": [p, i64, i32, p, i64, i32, p, i32, p, i64, p],
            "ocref_conv_bwd_data": [p, i64, i32, p, i32, p, i32, i64, p, p],
            "ocref_conv_bwd_weight": [p, i64, i32, p, i64, i32, p, i32, p, i64, p],
            "ocref_renew": [p, i64, p, i32, p],
            "ocref_renew_bwd": [p, i64, p, i32, i64, p],
            "ocref_pool_fwd": [p, i64, p, i64, i32, p, p],
            "ocref_pool_bwd": [p, i64, p, p, i32, i64, p],
            "ocref_unpool_fwd": [p, i64, p, p, i32, i64, p],
            "ocref_unpool_bwd": [p, i64, p, p, i32, p],
            "ocref_relu_fwd": [p, i64, p],
            "ocref_relu_bwd": [p, p, i64, p],
        }
        for name, args in sig.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = C.c_int
        L.ocref_num_threads.argtypes = []
        L.ocref_num_threads.restype = C.c_int
        L.ocref_set_num_threads.argtypes = [C.c_int32]
        L.ocref_set_num_threads.restype = C.c_int
        L.ocref_free.argtypes = [p]
        L.ocref_free.restype = None
        _lib = L
    return _lib


def num_threads() -> int:
    """OpenMP threads the oracle's parallel loops use."""
    return int(lib().ocref_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on (timing only)."""
    _check(lib().ocref_set_num_threads(int(n)))


def _ptr(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


class OracleError(RuntimeError):
    def __init__(self, code):
        super().__init__(f"oracle status {code}")
        self.code = code


def _check(rc):
    if rc != OK:
        raise OracleError(rc)


class Octree:
    """Super-octree built by breadth-first subdivision (Sec. 3.1)."""

    def __init__(self, points, normals, offsets, depth, full_depth=2):
        points = np.ascontiguousarray(points, dtype=np.float32).reshape(-1, 3)
        normals = np.ascontiguousarray(normals, dtype=np.float32).reshape(-1, 3)
        offsets = _i32(offsets)
        self.batch = len(offsets) - 1
        self.depth = depth
        self.full_depth = full_depth
        h = C.c_void_p()
        _check(lib().ocref_build(_ptr(points), _ptr(normals), _ptr(offsets), self.batch, depth,
                                 full_depth, C.byref(h)))
        self._h = h
        self.levels = []
        for l in range(depth + 1):
            n, m = C.c_int64(), C.c_int64()
            _check(lib().ocref_level_size(h, l, C.byref(n), C.byref(m)))
            keys = np.zeros(n.value, np.uint32)
            labels = np.zeros(n.value, np.int32)
            rows = np.zeros(m.value, np.int32)
            _check(lib().ocref_level(h, l, _ptr(keys), _ptr(labels), _ptr(rows)))
            self.levels.append({"keys": keys, "labels": labels, "rows": rows})
        sig = np.zeros((len(self.levels[depth]["keys"]), 3), np.float32)
        _check(lib().ocref_signal(h, _ptr(sig)))
        self.signal = sig

    def __del__(self):
        h = getattr(self, "_h", None)
        if h is not None and h.value and _lib is not None:
            _lib.ocref_free(h)
            self._h = None

    def num(self, l):
        return len(self.levels[l]["keys"])

    def nonempty(self, l):
        return len(self.levels[l]["rows"])

    def keys(self, l):
        return self.levels[l]["keys"]

    def labels(self, l):
        return self.levels[l]["labels"]

    def rows(self, l):
        return self.levels[l]["rows"]

    def neighbors(self, l, K=3, stride=1):
        r = int(stride).bit_length() - 1  # stride 2^r
        n = self.num(l) if stride == 1 else self.nonempty(l - r)
        nb = np.zeros((n, K ** 3), np.int32)
        _check(lib().ocref_neighbors(self._h, l, K, stride, _ptr(nb)))
        return nb


def conv_fwd(nb, x, w, rows=None):
    """Y = im2col(X; nb) . W, w [K^3][cin][cout]; rows: optional subset of outputs."""
    nb = _i32(nb)
    x = _f64(x)
    w = _f64(w)
    K3, cin, cout = w.shape
    assert nb.shape[1] == K3 and x.shape[1] == cin
    n_out = nb.shape[0]
    if rows is not None:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        y = np.zeros((len(rows), cout))
        _check(lib().ocref_conv_fwd(_ptr(nb), n_out, K3, _ptr(x), x.shape[0], cin, _ptr(w), cout,
                                    _ptr(rows), len(rows), _ptr(y)))
    else:
        y = np.zeros((n_out, cout))
        _check(lib().ocref_conv_fwd(_ptr(nb), n_out, K3, _ptr(x), x.shape[0], cin, _ptr(w), cout,
                                    None, 0, _ptr(y)))
    return y


def conv_bwd_data(nb, dy, w, n_in, want=None):
    """dX = col2im(dY . W^T; nb); want: optional bool mask of input rows to compute."""
    nb = _i32(nb)
    dy = _f64(dy)
    w = _f64(w)
    K3, cin, cout = w.shape
    dx = np.zeros((n_in, cin))
    wm = None if want is None else np.ascontiguousarray(want, dtype=np.uint8)
    _check(lib().ocref_conv_bwd_data(_ptr(nb), nb.shape[0], K3, _ptr(dy), cout, _ptr(w), cin, n_in,
                                     _ptr(wm), _ptr(dx)))
    return dx


def conv_bwd_weight(nb, x, dy, K3, entries=None):
    """dW = col^T . dY, [K^3][cin][cout]; entries: optional flat indices to compute."""
    nb = _i32(nb)
    x = _f64(x)
    dy = _f64(dy)
    cin, cout = x.shape[1], dy.shape[1]
    if entries is not None:
        entries = np.ascontiguousarray(entries, dtype=np.int64)
        dw = np.zeros(len(entries))
        _check(lib().ocref_conv_bwd_weight(_ptr(nb), nb.shape[0], K3, _ptr(x), x.shape[0], cin,
                                           _ptr(dy), cout, _ptr(entries), len(entries), _ptr(dw)))
        return dw
    dw = np.zeros((K3, cin, cout))
    _check(lib().ocref_conv_bwd_weight(_ptr(nb), nb.shape[0], K3, _ptr(x), x.shape[0], cin,
                                       _ptr(dy), cout, None, 0, _ptr(dw)))
    return dw


def renew(labels_lm1, yhat):
    labels_lm1 = _i32(labels_lm1)
    yhat = _f64(yhat)
    y = np.zeros((len(labels_lm1), yhat.shape[1]))
    _check(lib().ocref_renew(_ptr(labels_lm1), len(labels_lm1), _ptr(yhat), yhat.shape[1], _ptr(y)))
    return y


def renew_bwd(labels_lm1, dy, m):
    labels_lm1 = _i32(labels_lm1)
    dy = _f64(dy)
    dyhat = np.zeros((m, dy.shape[1]))
    _check(lib().ocref_renew_bwd(_ptr(labels_lm1), len(labels_lm1), _ptr(dy), dy.shape[1], m,
                                 _ptr(dyhat)))
    return dyhat


def conv_s2_fwd(tree: Octree, l, x, w):
    """Stride-2 conv (Sec. 3.2): conv at the first sibling of each group, renewed into T_{l-1}."""
    K = round(w.shape[0] ** (1 / 3))
    nb = tree.neighbors(l, K, stride=2)
    return renew(tree.labels(l - 1), conv_fwd(nb, x, w))


def conv_s2_bwd(tree: Octree, l, x, w, dy):
    K = round(w.shape[0] ** (1 / 3))
    nb = tree.neighbors(l, K, stride=2)
    dyhat = renew_bwd(tree.labels(l - 1), dy, nb.shape[0])
    dx = conv_bwd_data(nb, dyhat, w, x.shape[0])
    dw = conv_bwd_weight(nb, x, dyhat, w.shape[0])
    return dx, dw


def deconv_fwd(nb, x, w, n_out, want=None):
    """Stride-1 octree deconvolution (Sec. 3.2 "Deconvolution"): the
    convolution with its forward and backward passes swapped, so its forward
    is the convolution's input gradient.  w [K^3][cout][cin] is the weight of
    the convolution cout -> cin that it transposes; x [N_l][cin] -> [N_l][cout].
    want: optional bool mask of output rows to compute."""
    return conv_bwd_data(nb, x, w, n_out, want=want)


def deconv_bwd(nb, x, w, dy, rows=None, entries=None):
    """Backward of deconv_fwd, the convolution's forward and weight gradient:
    dx = conv(dy; w) [N_l][cin]; dw[k][co][ci] = sum_i dy[nb(i,k)][co] x[i][ci].
    rows / entries: optional subsets of dx rows and flat dw entries."""
    dx = conv_fwd(nb, dy, w, rows=rows)
    dw = conv_bwd_weight(nb, dy, x, w.shape[0], entries=entries)
    return dx, dw


def deconv_sr_fwd(tree: Octree, l, x, w, stride=2, want=None):
    """Strided deconvolution from depth l-r to depth l (stride 2^r): the
    transpose of the stride-2^r convolution at depth l (Sec. 3.2).  Row i of
    x [N_{l-r}][cin] counts only when its octant is non-empty (label p > 0);
    it reaches the depth-l neighbourhood of the first depth-l position below
    octant p-1.  -> [N_l][cout]."""
    r = int(stride).bit_length() - 1
    K = round(w.shape[0] ** (1 / 3))
    nb = tree.neighbors(l, K, stride=stride)
    xhat = renew_bwd(tree.labels(l - r), x, nb.shape[0])
    return conv_bwd_data(nb, xhat, w, tree.num(l), want=want)


def deconv_sr_bwd(tree: Octree, l, x, w, dy, stride=2, entries=None):
    """Backward of deconv_sr_fwd: dx = the stride-2^r convolution of dy
    [N_l][cout] ([N_{l-r}][cin], zero at empty octants), dw as in deconv_bwd
    over the evaluated positions."""
    r = int(stride).bit_length() - 1
    K = round(w.shape[0] ** (1 / 3))
    nb = tree.neighbors(l, K, stride=stride)
    dx = renew(tree.labels(l - r), conv_fwd(nb, dy, w))
    xhat = renew_bwd(tree.labels(l - r), x, nb.shape[0])
    dw = conv_bwd_weight(nb, dy, xhat, w.shape[0], entries=entries)
    return dx, dw


def deconv_s2_fwd(tree: Octree, l, x, w, want=None):
    """Stride-2 deconvolution (depth l-1 -> l): deconv_sr_fwd with stride 2."""
    return deconv_sr_fwd(tree, l, x, w, 2, want=want)


def deconv_s2_bwd(tree: Octree, l, x, w, dy, entries=None):
    """Backward of deconv_s2_fwd: deconv_sr_bwd with stride 2."""
    return deconv_sr_bwd(tree, l, x, w, dy, 2, entries=entries)


def conv_sr_fwd(tree: Octree, l, x, w, stride):
    """Convolution with stride 2^r (Sec. 3.2): evaluated at the first depth-l
    position of the sub-tree of height r below each non-empty octant of depth
    l-r, renewed into T_{l-r} through L_{l-r} (empty octants get 0)."""
    r = int(stride).bit_length() - 1
    K = round(w.shape[0] ** (1 / 3))
    nb = tree.neighbors(l, K, stride=stride)
    return renew(tree.labels(l - r), conv_fwd(nb, x, w))


def conv_sr_bwd(tree: Octree, l, x, w, dy, stride):
    r = int(stride).bit_length() - 1
    K = round(w.shape[0] ** (1 / 3))
    nb = tree.neighbors(l, K, stride=stride)
    dyhat = renew_bwd(tree.labels(l - r), dy, nb.shape[0])
    dx = conv_bwd_data(nb, dyhat, w, x.shape[0])
    dw = conv_bwd_weight(nb, x, dyhat, w.shape[0])
    return dx, dw


def pool_fwd(labels_lm1, x):
    labels_lm1 = _i32(labels_lm1)
    x = _f64(x)
    c = x.shape[1]
    y = np.zeros((len(labels_lm1), c))
    sw = np.zeros((x.shape[0] // 8, c), np.uint8)
    _check(lib().ocref_pool_fwd(_ptr(labels_lm1), len(labels_lm1), _ptr(x), x.shape[0], c, _ptr(y),
                                _ptr(sw)))
    return y, sw


def pool_bwd(labels_lm1, dy, sw, n_l):
    labels_lm1 = _i32(labels_lm1)
    dy = _f64(dy)
    sw = np.ascontiguousarray(sw, dtype=np.uint8)
    c = dy.shape[1]
    dx = np.zeros((n_l, c))
    _check(lib().ocref_pool_bwd(_ptr(labels_lm1), len(labels_lm1), _ptr(dy), _ptr(sw), c, n_l,
                                _ptr(dx)))
    return dx


def unpool_fwd(labels_lm1, x, sw, n_l):
    labels_lm1 = _i32(labels_lm1)
    x = _f64(x)
    sw = np.ascontiguousarray(sw, dtype=np.uint8)
    c = x.shape[1]
    y = np.zeros((n_l, c))
    _check(lib().ocref_unpool_fwd(_ptr(labels_lm1), len(labels_lm1), _ptr(x), _ptr(sw), c, n_l,
                                  _ptr(y)))
    return y


def unpool_bwd(labels_lm1, dy, sw):
    labels_lm1 = _i32(labels_lm1)
    dy = _f64(dy)
    sw = np.ascontiguousarray(sw, dtype=np.uint8)
    c = dy.shape[1]
    dx = np.zeros((len(labels_lm1), c))
    _check(lib().ocref_unpool_bwd(_ptr(labels_lm1), len(labels_lm1), _ptr(dy), _ptr(sw), c,
                                  _ptr(dx)))
    return dx


POOL_MAX, POOL_AVG = 0, 1
POOL_ABSENT = 255  # switch value: the maximum was an absent neighbour's zero


def gpool_fwd(nb, x, mode, rows=None):
    """General pooling (Sec. 3.2 "Pooling", last paragraph): the K^3
    neighbourhood of every octant is found as for the stride-1 convolution,
    and each channel takes the max (mode POOL_MAX) or the average (POOL_AVG)
    over it.  A neighbour that is not in the octree counts as a zero, as in
    the convolution (so the average divides by K^3).  Returns y [N][C] and,
    for max, the switch sw [N][C] u8: the tap of the first maximum in tap
    order, or POOL_ABSENT when that maximum is an absent neighbour.
    rows: optional subset of output rows.  Rows are taken in chunks so that
    the gathered [rows][K^3][C] block stays near 256 MB."""
    nb = _i32(nb)
    x = _f64(x)
    if rows is not None:
        nb = nb[np.asarray(rows, dtype=np.int64)]
    n, K3 = nb.shape
    C = x.shape[1]
    ext = np.vstack([x, np.zeros((1, C))])
    y = np.zeros((n, C))
    sw = None if mode == POOL_AVG else np.zeros((n, C), np.uint8)
    step = max(1, (1 << 25) // max(1, K3 * C))
    for r0 in range(0, n, step):
        part = nb[r0:r0 + step]
        vals = ext[np.where(part >= 0, part, x.shape[0])]  # [rows][K^3][C]
        if mode == POOL_AVG:
            y[r0:r0 + step] = vals.sum(axis=1) / K3
            continue
        k = np.argmax(vals, axis=1)  # first maximum
        y[r0:r0 + step] = np.take_along_axis(vals, k[:, None, :], axis=1)[:, 0, :]
        absent = np.take_along_axis(part, k, axis=1) < 0
        sw[r0:r0 + step] = np.where(absent, POOL_ABSENT, k)
    return y, sw


def gpool_bwd(nb, dy, sw, n_in, mode):
    """Gradient of gpool_fwd w.r.t. x [n_in][C]: every output's gradient goes
    to its switch's neighbour (max; nowhere for POOL_ABSENT) or, divided by
    K^3, to each of its present neighbours (average).  Added tap by tap; within
    one tap no two octants share a neighbour (the neighbour at a fixed offset
    is a position shift), so each tap is a plain indexed add."""
    nb = _i32(nb)
    dy = _f64(dy)
    n, K3 = nb.shape
    dx = np.zeros((n_in, dy.shape[1]))
    for k in range(K3):
        rows = np.nonzero(nb[:, k] >= 0)[0]
        idx = nb[rows, k]
        assert len(np.unique(idx)) == len(idx)
        if mode == POOL_AVG:
            dx[idx] += dy[rows] / K3
        else:
            dx[idx] += dy[rows] * (sw[rows] == k)
    return dx


def gpool_sr_fwd(tree: Octree, l, x, mode, stride):
    """General pooling with stride 2^r (Sec. 3.2, pooling as a special kind of
    convolution, here with another stride): the 3x3x3 neighbourhood the
    stride-2^r convolution reads, evaluated at the first depth-l position
    below every non-empty depth-(l-r) octant and written to that octant's
    row; absent neighbours count as zeros (as at stride 1).  Rows of empty
    depth-(l-r) octants get 0 and, for max, the switch POOL_ABSENT.
    Returns y [N_{l-r}][C] and sw [N_{l-r}][C] u8 (max) or None."""
    r = int(stride).bit_length() - 1
    nb = tree.neighbors(l, 3, stride=stride)
    yh, swh = gpool_fwd(nb, x, mode)
    lab = tree.labels(l - r)
    y = renew(lab, yh)
    if mode == POOL_AVG:
        return y, None
    sw = np.full((len(lab), yh.shape[1]), POOL_ABSENT, np.uint8)
    sw[lab > 0] = swh[lab[lab > 0] - 1]
    return y, sw


def gpool_sr_bwd(tree: Octree, l, dy, sw, n_in, mode, stride):
    """Gradient of gpool_sr_fwd w.r.t. x [n_in][C]: the rows of the
    non-empty depth-(l-r) octants carry their gradient (and switch) to the
    stride-1 rule of gpool_bwd over the strided neighbourhood."""
    r = int(stride).bit_length() - 1
    nb = tree.neighbors(l, 3, stride=stride)
    dyh = renew_bwd(tree.labels(l - r), dy, nb.shape[0])
    swh = None if mode == POOL_AVG else np.asarray(sw)[tree.rows(l - r)]
    return gpool_bwd(nb, dyh, swh, n_in, mode)


def relu_fwd(x):
    x = _f64(x)
    y = np.zeros_like(x)
    _check(lib().ocref_relu_fwd(_ptr(x), x.size, _ptr(y)))
    return y


def relu_bwd(x, dy):
    x = _f64(x)
    dy = _f64(dy)
    dx = np.zeros_like(x)
    _check(lib().ocref_relu_bwd(_ptr(x), _ptr(dy), x.size, _ptr(dx)))
    return dx
