"""Pins of the CPU oracle's octree build (Sec. 3.1) against hand-worked values,
the Fig. 2 example carried to 3D, and invariants the paper fixes."""
import os

import numpy as np
import pytest

import oracle
import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _single_point_tree(depth, x, y, z, full_depth=0):
    side = 2 ** depth
    p = (np.array([[x, y, z]], np.float64) + 0.5) / side
    return oracle.Octree(p.astype(np.float32), np.ones((1, 3), np.float32), [0, 1], depth, full_depth)


def test_hand_keys():
    rows = [l.split() for l in open(os.path.join(GOLD, "keys.txt")) if l.strip() and l[0] != "#"]
    assert len(rows) >= 8
    for d, x, y, z, key in ([int(v) for v in r] for r in rows):
        t = _single_point_tree(d, x, y, z)
        lab = t.labels(d)
        keys = t.keys(d)[lab > 0]
        assert keys.tolist() == [key], (d, x, y, z)


def _load_fig2():
    spec = {"point": [], "signal": []}
    for line in open(os.path.join(GOLD, "fig2_3d.txt")):
        if not line.strip() or line[0] == "#":
            continue
        k, *v = line.split()
        if k in ("point", "signal"):
            spec[k].append([float(a) for a in v])
        else:
            spec[k] = [int(a) for a in v]
    return spec


def test_fig2_worked_example_3d():
    s = _load_fig2()
    pts = np.array([p[:3] for p in s["point"]], np.float32)
    nrm = np.array([p[3:] for p in s["point"]], np.float32)
    t = oracle.Octree(pts, nrm, [0, len(pts)], s["depth"][0], s["full_depth"][0])
    assert t.keys(1).tolist() == s["S1"]
    assert t.labels(1).tolist() == s["L1"]
    assert t.keys(2).tolist() == s["S2"]
    assert t.labels(2).tolist() == s["L2"]
    assert t.num(2) == 24
    # the first child of the node at index 2 (label 3) is row 8 * (3 - 1) = 16
    assert t.keys(2)[16] == 8 * t.keys(1)[2]
    sig = np.zeros((24, 3), np.float32)
    for r, *v in s["signal"]:
        sig[int(r)] = v
    np.testing.assert_array_equal(t.signal, sig)


def _decode(key, l):
    """Test-local decode of a super key into (b, x, y, z) by reading digits."""
    b = key >> 24
    k = key & 0xFFFFFF
    x = y = z = 0
    for i in range(l):
        g = (k >> (3 * (l - 1 - i))) & 7
        x, y, z = 2 * x + (g >> 2), 2 * y + ((g >> 1) & 1), 2 * z + (g & 1)
    return b, x, y, z


@pytest.mark.parametrize("seed,B,depth,full", [(1, 1, 3, 0), (2, 3, 4, 2), (3, 2, 5, 1), (4, 4, 4, 4)])
def test_build_invariants_and_occupancy(seed, B, depth, full):
    pts, nrm, offs = synth.random_cloud(seed, B, [200, 0, 57, 1][:B] if B > 1 else 300, "union")
    t = oracle.Octree(pts, nrm, offs, depth, full)
    q = np.minimum(np.floor(pts * np.float32(2 ** depth)).astype(np.int64), 2 ** depth - 1)
    shape = np.repeat(np.arange(B), np.diff(offs))
    for l in range(depth + 1):
        keys, lab, rows = t.keys(l), t.labels(l), t.rows(l)
        # sorted ascending (Sec. 3.1), batch byte in the top 8 bits
        assert np.all(np.diff(keys.astype(np.int64)) > 0)
        # labels: running 1-based count over the non-empty octants
        nz = lab > 0
        assert lab[nz].tolist() == list(range(1, nz.sum() + 1))
        assert rows.tolist() == np.nonzero(nz)[0].tolist()
        # occupancy: octant non-empty iff a point falls in it, or forced
        dec = [_decode(int(k), l) for k in keys]
        occ = {(int(b), *map(int, c)) for b, c in zip(shape, q >> (depth - l))}
        for (b, x, y, z), e in zip(dec, nz):
            assert e == ((b, x, y, z) in occ or l < full), (l, b, x, y, z)
        if l == 0:
            assert keys.tolist() == [b << 24 for b in range(B)]
            continue
        # child rule (Sec. 3.1 "Label"): first child of j at 8 (L_{l-1}[j] - 1)
        pk, pl = t.keys(l - 1), t.labels(l - 1)
        assert len(keys) == 8 * int((pl > 0).sum())
        for j in np.nonzero(pl > 0)[0]:
            k0 = 8 * (pl[j] - 1)
            b, kk = int(pk[j]) >> 24, int(pk[j]) & 0xFFFFFF
            assert keys[k0:k0 + 8].tolist() == [(b << 24) | (8 * kk + c) for c in range(8)]


def test_signal_is_mean_normal():
    # three points in one leaf, one in another, depth 3
    side = 8
    pts = (np.array([[1, 2, 3], [1, 2, 3], [1, 2, 3], [6, 0, 7]], np.float64) + [[.1, .2, .3], [.5, .5, .5], [.9, .9, .1], [.5, .5, .5]]) / side
    nrm = np.array([[1, 0, 0], [0, 2, 0], [0, 0, 3], [-1, -1, -1]], np.float32)
    t = oracle.Octree(pts.astype(np.float32), nrm, [0, 4], 3, 0)
    keys, lab = t.keys(3), t.labels(3)
    got = {_decode(int(k), 3)[1:]: tuple(t.signal[i]) for i, k in enumerate(keys) if lab[i] > 0}
    assert got == {(1, 2, 3): (np.float32(1 / 3), np.float32(2 / 3), np.float32(1.0)), (6, 0, 7): (-1, -1, -1)}
    assert np.all(t.signal[lab == 0] == 0)


def test_boundary_and_errors():
    # 1.0 is clamped into the last octant; 0.0 lands in the first
    t = oracle.Octree(np.array([[1.0, 0.0, 1.0]], np.float32), np.ones((1, 3), np.float32), [0, 1], 2, 0)
    keys = t.keys(2)[t.labels(2) > 0]
    assert [_decode(int(k), 2)[1:] for k in keys] == [(3, 0, 3)]
    for bad in ([[1.5, 0, 0]], [[-0.1, 0, 0]], [[np.nan, 0, 0]]):
        with pytest.raises(oracle.OracleError) as e:
            oracle.Octree(np.array(bad, np.float32), np.ones((1, 3), np.float32), [0, 1], 2, 0)
        assert e.value.code == oracle.ERR_RANGE
    with pytest.raises(oracle.OracleError):
        oracle.Octree(np.zeros((1, 3), np.float32), np.ones((1, 3), np.float32), [0, 1], 9, 0)
    # normals are averaged into the signal, so they must be finite
    for bad in ([[np.inf, 0, 0]], [[0, np.nan, 0]]):
        with pytest.raises(oracle.OracleError) as e:
            oracle.Octree(np.full((1, 3), 0.5, np.float32), np.array(bad, np.float32), [0, 1], 2, 0)
        assert e.value.code == oracle.ERR_RANGE


def test_empty_shape_and_full_depth():
    pts, nrm, offs = synth.random_cloud(7, 3, [0, 40, 0], "uniform")
    t = oracle.Octree(pts, nrm, offs, 3, 2)
    # full depth 2: every depth-1 octant of every shape is non-empty, so
    # N_2 = 64 per shape; the empty shapes have nothing deeper
    assert t.num(1) == 24 and t.nonempty(1) == 24 and t.num(2) == 192
    l2 = t.labels(2).reshape(3, 64)
    assert l2[0].max() == 0 and l2[2].max() == 0 and l2[1].max() > 0
    t0 = oracle.Octree(pts, nrm, offs, 3, 0)
    assert t0.labels(0).tolist() == [0, 1, 0]
    assert t0.num(1) == 8
