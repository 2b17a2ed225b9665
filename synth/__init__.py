"""Seeded synthetic inputs shared by the tests, the CPU oracle's callers and the bench.

This module only draws random numbers: oriented surface point clouds inside
the unit cube, dense feature maps, convolution weights and upstream
gradients.  It holds none of the octree method's arithmetic (no keys, no
octants, no convolution), so the CPU oracle and the HIP library can both be
fed from it without sharing any code path.

The point clouds stand in for the paper's ray-shot ModelNet40 samples
(Sec. 5, "Octree data preparation"): closed surfaces inside the unit cube,
densely sampled, with normals pointing outwards.

Workloads (sizes are the batch's; a "shape" is one point cloud):

==========  =====  =====  ========  ===============================================
name        depth  batch  pts/shape  network on the octree
==========  =====  =====  ========  ===============================================
sphere_d5   5      1      20k       conv3 3->32, pool d5->d4
net_d5      5      32     20k       conv3 3->32 @5, pool, 32->64 @4, pool, 64->128 @3, pool, 128->256 @2
net_d6      6      32     20k       conv3+ReLU+pool: 3->16 @6, 16->32 @5, 32->64 @4, 64->128 @3; conv3+ReLU 128->256 @2
deep_d8     8      8      100k      conv3 16->16 @8, pool d8->d7, unpool d7->d8
wide_d7     7      16     100k      conv5 64->64 @7 (bf16 and fp32), stride-2 conv3 64->128 d7->d6
seg_d6      6      32     20k       conv3+ReLU+pool 3->16 @6, 16->32 @5; stride-2 deconv3 32->16
                                    d4->d5; unpool d5->d6; deconv3 16->16 @6
gpool_d6    6      32     20k       conv3+ReLU 3->16 @6; 3x3x3 max-pool and 5x5x5 average-pool,
                                    stride 1, @6; 2x2x2 max-pool d6->d5; 3x3x3 max-pool
                                    stride 2 d5->d4; 3x3x3 average-pool stride 4 d4->d2
ocnn_d6     6      32     20k       O-CNN(6) training iteration: U_6 .. U_2 (conv3 + BN + ReLU +
                                    pool; 3->8, 8->16, 16->32, 32->64, 64->128), dropout,
                                    FC(128), dropout, FC(40), softmax loss, SGD (synthetic labels)
s4_d6       6      32     20k       conv3+ReLU 3->16 @6; stride-4 conv3+ReLU 16->64 d6->d4;
                                    conv3 64->128 @4
==========  =====  =====  ========  ===============================================

seg_d6 is the decoder side of the paper's segmentation network (Sec. 4,
the deconvolution units that mirror the encoder) on the depth-6 shapes: an
encoder of two conv+ReLU+pool stages, then a stride-2 deconvolution back up
one depth and an unpooling + deconvolution unit.  Normalisation and the
ReLU between the units are left out (not octree operations).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "Layer",
    "Workload",
    "WORKLOADS",
    "sphere_cloud",
    "primitive_union_cloud",
    "make_points",
    "make_weights",
    "make_features",
    "make_train_inputs",
    "make_upstream",
    "random_cloud",
]


@dataclass(frozen=True)
class Layer:
    """One operation of a workload's network."""

    op: str  # "conv", "deconv", "pool", "unpool", "gpool"
    depth: int  # input depth of the op (deconv and unpool: its output depth)
    cin: int = 0
    cout: int = 0
    ksize: int = 3
    stride: int = 1
    relu: bool = False
    dtype: str = "f32"  # "f32" or "bf16"
    mode: str = "max"  # gpool: "max" or "avg"


@dataclass(frozen=True)
class Workload:
    name: str
    seed_id: int
    depth: int
    batch: int
    points_per_shape: int
    kind: str  # "sphere" or "union"
    layers: tuple = field(default_factory=tuple)
    weight_sigma: float | None = None  # None: He-normal sqrt(2/(K^3 Cin))
    signal_input: bool = True  # first conv reads the averaged-normal signal
    full_depth: int = 2
    train: bool = False  # the O-CNN(d) classification training iteration around the convs
    classes: int = 40


WORKLOADS = {
    "sphere_d5": Workload(
        "sphere_d5", 1, 5, 1, 20_000, "sphere",
        (Layer("conv", 5, 3, 32), Layer("pool", 5, 32, 32)),
        weight_sigma=0.1,
    ),
    "net_d5": Workload(
        "net_d5", 2, 5, 32, 20_000, "union",
        (
            Layer("conv", 5, 3, 32), Layer("pool", 5, 32, 32),
            Layer("conv", 4, 32, 64), Layer("pool", 4, 64, 64),
            Layer("conv", 3, 64, 128), Layer("pool", 3, 128, 128),
            Layer("conv", 2, 128, 256),
        ),
    ),
    "net_d6": Workload(
        "net_d6", 3, 6, 32, 20_000, "union",
        (
            Layer("conv", 6, 3, 16, relu=True), Layer("pool", 6, 16, 16),
            Layer("conv", 5, 16, 32, relu=True), Layer("pool", 5, 32, 32),
            Layer("conv", 4, 32, 64, relu=True), Layer("pool", 4, 64, 64),
            Layer("conv", 3, 64, 128, relu=True), Layer("pool", 3, 128, 128),
            Layer("conv", 2, 128, 256, relu=True),
        ),
    ),
    "deep_d8": Workload(
        "deep_d8", 4, 8, 8, 100_000, "union",
        (Layer("conv", 8, 16, 16), Layer("pool", 8, 16, 16), Layer("unpool", 8, 16, 16)),
        signal_input=False,
    ),
    "wide_d7": Workload(
        "wide_d7", 5, 7, 16, 100_000, "union",
        (
            Layer("conv", 7, 64, 64, ksize=5, dtype="bf16"),
            Layer("conv", 7, 64, 128, ksize=3, stride=2, dtype="bf16"),
        ),
        signal_input=False,
    ),
    "seg_d6": Workload(
        "seg_d6", 6, 6, 32, 20_000, "union",
        (
            Layer("conv", 6, 3, 16, relu=True), Layer("pool", 6, 16, 16),
            Layer("conv", 5, 16, 32, relu=True), Layer("pool", 5, 32, 32),
            Layer("deconv", 5, 32, 16, stride=2),
            Layer("unpool", 6, 16, 16),
            Layer("deconv", 6, 16, 16),
        ),
    ),
    "gpool_d6": Workload(
        "gpool_d6", 7, 6, 32, 20_000, "union",
        (
            Layer("conv", 6, 3, 16, relu=True),
            Layer("gpool", 6, 16, 16, ksize=3, mode="max"),
            Layer("gpool", 6, 16, 16, ksize=5, mode="avg"),
            Layer("pool", 6, 16, 16),
            Layer("gpool", 5, 16, 16, ksize=3, stride=2, mode="max"),
            Layer("gpool", 4, 16, 16, ksize=3, stride=4, mode="avg"),
        ),
    ),
    # O-CNN(6) (units U_6 .. U_2: conv + BN + ReLU + pool, C_l = 2^max(1, 9-l)),
    # dropout, FC(128), dropout, FC(40), softmax loss, SGD: one training iteration
    "ocnn_d6": Workload(
        "ocnn_d6", 9, 6, 32, 20_000, "union",
        (
            Layer("conv", 6, 3, 8), Layer("conv", 5, 8, 16), Layer("conv", 4, 16, 32),
            Layer("conv", 3, 32, 64), Layer("conv", 2, 64, 128),
        ),
        train=True,
    ),
    "s4_d6": Workload(
        "s4_d6", 8, 6, 32, 20_000, "union",
        (
            Layer("conv", 6, 3, 16, relu=True),
            Layer("conv", 6, 16, 64, stride=4, relu=True),
            Layer("conv", 4, 64, 128),
        ),
    ),
}


# ----------------------------------------------------------------------------
# surface samplers


def sphere_cloud(n: int, rng: np.random.Generator, centre=(0.5, 0.5, 0.5), radius=0.4):
    """n points uniform on a sphere (normalised Gaussian directions); normal = radial."""
    d = rng.standard_normal((n, 3))
    d /= np.linalg.norm(d, axis=1, keepdims=True)
    pts = np.asarray(centre, dtype=np.float64) + radius * d
    return pts, d


def _sample_sphere_surface(c, r, m, rng):
    d = rng.standard_normal((m, 3))
    d /= np.linalg.norm(d, axis=1, keepdims=True)
    return c + r * d, d


def _sample_box_surface(c, h, m, rng):
    # face areas: the two faces normal to axis a have area 4 * h_b * h_c each
    areas = np.array([h[1] * h[2], h[0] * h[2], h[0] * h[1]])
    axis = rng.choice(3, size=m, p=areas / areas.sum())
    sign = np.where(rng.random(m) < 0.5, -1.0, 1.0)
    u = rng.uniform(-1.0, 1.0, size=(m, 3)) * h
    idx = np.arange(m)
    u[idx, axis] = sign * h[axis]
    nrm = np.zeros((m, 3))
    nrm[idx, axis] = sign
    return c + u, nrm


def _strictly_inside(prim, p):
    kind, c, s = prim
    if kind == "sphere":
        return np.sum((p - c) ** 2, axis=1) < s * s
    return np.all(np.abs(p - c) < s, axis=1)


def primitive_union_cloud(n: int, rng: np.random.Generator):
    """n points on the boundary of a union of 1-4 spheres / axis-aligned boxes.

    Each primitive is a sphere or a box with probability 1/2; the radius and the
    three box half-extents are U[0.1, 0.4]; the centre is uniform on the range
    that keeps the primitive inside the unit cube.  Points are drawn from a
    primitive in proportion to its surface area, uniformly on its surface, and
    rejected when strictly inside another primitive.  Normals are outward.
    """
    nprim = int(rng.integers(1, 5))
    prims = []
    for _ in range(nprim):
        if rng.random() < 0.5:
            r = rng.uniform(0.1, 0.4)
            c = rng.uniform(r, 1.0 - r, size=3)
            prims.append(("sphere", c, r))
        else:
            h = rng.uniform(0.1, 0.4, size=3)
            c = rng.uniform(h, 1.0 - h)
            prims.append(("box", c, h))
    area = np.array(
        [4 * math.pi * s * s if k == "sphere" else 8 * (s[0] * s[1] + s[1] * s[2] + s[0] * s[2])
         for k, _, s in prims]
    )
    pts_out, nrm_out, have = [], [], 0
    while have < n:
        m = max(2 * (n - have), 1024)
        which = rng.choice(nprim, size=m, p=area / area.sum())
        for i, (kind, c, s) in enumerate(prims):
            cnt = int(np.sum(which == i))
            if cnt == 0:
                continue
            if kind == "sphere":
                p, q = _sample_sphere_surface(c, s, cnt, rng)
            else:
                p, q = _sample_box_surface(c, s, cnt, rng)
            keep = np.ones(cnt, dtype=bool)
            for j, other in enumerate(prims):
                if j != i:
                    keep &= ~_strictly_inside(other, p)
            pts_out.append(p[keep])
            nrm_out.append(q[keep])
            have += int(keep.sum())
    pts = np.concatenate(pts_out)[:n]
    nrm = np.concatenate(nrm_out)[:n]
    return pts, nrm


def _to_f32_cube(pts, nrm):
    pts = np.clip(pts.astype(np.float32), np.float32(0.0), np.float32(1.0))
    return np.ascontiguousarray(pts), np.ascontiguousarray(nrm.astype(np.float32))


def make_points(w: Workload | str, batch: int | None = None):
    """Points f32 [P][3] in [0,1]^3, normals f32 [P][3], shape offsets i32 [B+1]."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    B = w.batch if batch is None else batch
    P, N = [], []
    for b in range(B):
        if w.kind == "sphere":
            rng = np.random.default_rng(0 if B == 1 else [w.seed_id, b])
            p, q = sphere_cloud(w.points_per_shape, rng)
        else:
            rng = np.random.default_rng([w.seed_id, b])
            p, q = primitive_union_cloud(w.points_per_shape, rng)
        p, q = _to_f32_cube(p, q)
        P.append(p)
        N.append(q)
    offs = np.zeros(B + 1, dtype=np.int32)
    offs[1:] = np.cumsum([len(p) for p in P])
    return np.concatenate(P), np.concatenate(N), offs


def random_cloud(seed: int, shapes: int, pts_per_shape, spread: str = "uniform"):
    """Small random clouds for the CPU pins: uniform in the cube or on a union surface."""
    rng = np.random.default_rng(seed)
    P, N = [], []
    for b in range(shapes):
        n = pts_per_shape if np.isscalar(pts_per_shape) else pts_per_shape[b]
        if spread == "uniform":
            p = rng.random((n, 3))
            q = rng.standard_normal((n, 3))
        else:
            p, q = primitive_union_cloud(max(n, 1), rng)
            p, q = p[:n], q[:n]
        p, q = _to_f32_cube(p, q)
        P.append(p)
        N.append(q)
    offs = np.zeros(shapes + 1, dtype=np.int32)
    offs[1:] = np.cumsum([len(p) for p in P])
    pts = np.concatenate(P) if P else np.zeros((0, 3), np.float32)
    nrm = np.concatenate(N) if N else np.zeros((0, 3), np.float32)
    return pts.reshape(-1, 3), nrm.reshape(-1, 3), offs


def make_weights(w: Workload | str, layer: int, ksize: int, cin: int, cout: int):
    """Weights f32 [K^3][cin][cout]: N(0, sigma^2), sigma fixed by the workload or He-normal.
    A deconvolution cin -> cout takes make_weights(..., cout, cin): the weight of
    the convolution it transposes."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    rng = np.random.default_rng([w.seed_id, 1000 + layer])
    sigma = w.weight_sigma if w.weight_sigma is not None else math.sqrt(2.0 / (ksize ** 3 * cin))
    return (sigma * rng.standard_normal((ksize ** 3, cin, cout))).astype(np.float32)


def make_train_inputs(w: Workload | str, batch: int | None = None, p_drop: float = 0.5):
    """Draws of a training iteration (the random numbers the method uses):
    class labels i32 [B] in [0, classes), the two dropout keep masks u8
    [B][8 C_2] and [B][128] (keep with probability 1 - p_drop), and the head's
    initial parameters: BN gamma = 1, beta = 0 per conv layer, FC weights
    N(0, 1/fan_in), FC biases 0."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    B = w.batch if batch is None else batch
    rng = np.random.default_rng([w.seed_id, 5000])
    c2 = w.layers[-1].cout
    out = {
        "labels": rng.integers(0, w.classes, B).astype(np.int32),
        "keep1": (rng.random((B, 8 * c2)) >= p_drop).astype(np.uint8),
        "keep2": (rng.random((B, 128)) >= p_drop).astype(np.uint8),
        "bn": [(np.ones(L.cout, np.float32), np.zeros(L.cout, np.float32)) for L in w.layers],
        "fc1_w": (rng.standard_normal((8 * c2, 128)) / math.sqrt(8 * c2)).astype(np.float32),
        "fc1_b": np.zeros(128, np.float32),
        "fc2_w": (rng.standard_normal((128, w.classes)) / math.sqrt(128)).astype(np.float32),
        "fc2_b": np.zeros(w.classes, np.float32),
    }
    return out


def make_features(seed, rows: int, channels: int):
    """Dense N(0,1) features f32 [rows][channels]."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal((rows, channels), dtype=np.float32)


def make_upstream(w: Workload | str, layer: int, rows: int, channels: int):
    """Upstream gradient N(0,1) f32 [rows][channels]."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    rng = np.random.default_rng([w.seed_id, 2000 + layer])
    return rng.standard_normal((rows, channels), dtype=np.float32)
