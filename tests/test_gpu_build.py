"""GPU parity of the octree build: keys, labels, label->row maps and the
sibling-group neighbour tables bit-exact against the CPU oracle; the input
signal within fp32 tolerance."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_f32_close, per_octant_neighbors

pytestmark = pytest.mark.gpu


def _gpu():
    import paper_1712_01537_amd as oc
    return oc


def _build_both(pts, nrm, offs, depth, full):
    oc = _gpu()
    print(f"[build] P={len(pts)} B={len(offs) - 1} depth={depth} full={full}", flush=True)
    ref = oracle.Octree(pts, nrm, offs, depth, full)
    tree = oc.oc_build(torch.as_tensor(pts).cuda(), torch.as_tensor(nrm).cuda(), offs, depth, full)
    torch.cuda.synchronize()
    return ref, tree


def _compare_tree(ref, tree, nb_depths=None, K=3):
    assert tree.depth == ref.depth and tree.batch == ref.batch
    for l in range(ref.depth + 1):
        assert tree.num(l) == ref.num(l), l
        assert tree.nonempty(l) == ref.nonempty(l), l
        np.testing.assert_array_equal(tree.keys(l).cpu().numpy().view(np.uint32), ref.keys(l), err_msg=f"keys {l}")
        np.testing.assert_array_equal(tree.labels(l).cpu().numpy(), ref.labels(l), err_msg=f"labels {l}")
        np.testing.assert_array_equal(tree.rows(l).cpu().numpy(), ref.rows(l), err_msg=f"rows {l}")
    for l in (nb_depths if nb_depths is not None else range(1, ref.depth + 1)):
        if ref.num(l) == 0:
            continue
        got = per_octant_neighbors(tree.nbr(l).cpu().numpy(), K)
        np.testing.assert_array_equal(got, ref.neighbors(l, K), err_msg=f"neighbours depth {l} K {K}")
    assert_f32_close(tree.signal().cpu().numpy(), ref.signal, "signal", rtol=1e-6, atol=1e-7)


SMALL = [  # seed, shapes, points per shape, depth, full depth, spread
    (1, 1, 300, 3, 0, "uniform"),
    (2, 3, [200, 0, 57], 4, 2, "union"),
    (3, 2, 500, 5, 1, "union"),
    (4, 4, [1, 2, 3, 0], 4, 4, "uniform"),
    (5, 5, 2000, 6, 2, "union"),
    (6, 2, 40000, 8, 2, "union"),
    (7, 17, 300, 5, 2, "union"),
]


@pytest.mark.parametrize("seed,B,n,depth,full,spread", SMALL)
def test_build_small(seed, B, n, depth, full, spread):
    pts, nrm, offs = synth.random_cloud(seed, B, n, spread)
    ref, tree = _build_both(pts, nrm, offs, depth, full)
    _compare_tree(ref, tree)
    # K = 5 neighbourhoods come from the same 27-entry tables
    _compare_tree(ref, tree, nb_depths=[depth], K=5)


def test_build_fig2_example():
    pts = np.array([[.1, .1, .1], [.1, .1, .6], [.1, .6, .1], [.4, .9, .4], [.2, .2, .05]], np.float32)
    nrm = np.array([[1, 0, 0], [0, 1, 0], [0, 0, 1], [0, 0, -1], [0, 1, 0]], np.float32)
    ref, tree = _build_both(pts, nrm, [0, 5], 2, 1)
    _compare_tree(ref, tree)
    assert tree.labels(1).cpu().tolist() == [1, 2, 3, 0, 0, 0, 0, 0]


def test_build_all_empty_and_errors():
    oc = _gpu()
    pts = np.zeros((0, 3), np.float32)
    ref, tree = _build_both(pts, pts, [0, 0, 0], 4, 2)
    _compare_tree(ref, tree)
    ref0, tree0 = _build_both(pts, pts, [0, 0], 3, 0)
    _compare_tree(ref0, tree0)
    bad = torch.tensor([[0.5, 1.5, 0.2]], dtype=torch.float32, device="cuda")
    with pytest.raises(oc.OcError) as e:
        oc.oc_build(bad, bad, [0, 1], 3, 2)
    assert e.value.code == 2
    nan = torch.tensor([[0.5, float("nan"), 0.2]], dtype=torch.float32, device="cuda")
    with pytest.raises(oc.OcError) as e:
        oc.oc_build(nan, nan, [0, 1], 3, 2)
    assert e.value.code == 2
    good = torch.tensor([[0.5, 0.25, 0.2]], dtype=torch.float32, device="cuda")
    inf = torch.tensor([[0.0, float("inf"), 0.0]], dtype=torch.float32, device="cuda")
    with pytest.raises(oc.OcError) as e:
        oc.oc_build(good, inf, [0, 1], 3, 2)
    assert e.value.code == 2 and "normal" in str(e.value)
    # the library stays usable after a rejected build
    ref, tree = _build_both(good.cpu().numpy(), good.cpu().numpy(), [0, 1], 3, 2)
    _compare_tree(ref, tree)


def test_build_deterministic():
    pts, nrm, offs = synth.make_points("net_d5", batch=4)
    oc = _gpu()
    p, n = torch.as_tensor(pts).cuda(), torch.as_tensor(nrm).cuda()
    a = oc.oc_build(p, n, offs, 5, 2)
    b = oc.oc_build(p, n, offs, 5, 2)
    for l in range(6):
        assert torch.equal(a.keys(l), b.keys(l)) and torch.equal(a.labels(l), b.labels(l))
        if l:
            assert torch.equal(a.nbr(l), b.nbr(l))
    assert torch.equal(a.signal().view(torch.int32), b.signal().view(torch.int32))


@pytest.mark.parametrize("name", ["sphere_d5", "net_d5", "net_d6", "deep_d8", "wide_d7"])
def test_build_workloads_full_size(name):
    w = synth.WORKLOADS[name]
    pts, nrm, offs = synth.make_points(w)
    ref, tree = _build_both(pts, nrm, offs, w.depth, w.full_depth)
    _compare_tree(ref, tree, nb_depths=[w.depth])
    print(f"[build] {name}: N = {[tree.num(l) for l in range(w.depth + 1)]}, "
          f"M = {[tree.nonempty(l) for l in range(w.depth + 1)]}", flush=True)


def test_build_async_finish_two_streams():
    """oc_build_async on one stream, oc_build_finish on another: the same
    octree as the oracle and as oc_build, also with several jobs in flight
    finished out of order (each with its own count buffer)."""
    oc = _gpu()
    cases = [synth.random_cloud(5, 5, 2000, "union"), synth.random_cloud(7, 17, 300, "union"),
             synth.make_points("net_d5", batch=4)]
    depths = [(6, 2), (5, 2), (5, 2)]
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    jobs = []
    with torch.cuda.stream(sa):
        for (pts, nrm, offs), (d, fd) in zip(cases, depths):
            print(f"[build async] P={len(pts)} B={len(offs) - 1} depth={d}", flush=True)
            p, n = torch.as_tensor(pts).cuda(), torch.as_tensor(nrm).cuda()
            jobs.append(oc.oc_build_async(p, n, offs, d, fd))
            # unrelated work queued behind the job on its stream
            torch.mm(torch.ones(512, 512, device="cuda"), torch.ones(512, 512, device="cuda"))
    trees = [None] * len(jobs)
    for k in reversed(range(len(jobs))):
        trees[k] = jobs[k].finish(sb)
    torch.cuda.synchronize()
    for (pts, nrm, offs), (d, fd), tree in zip(cases, depths, trees):
        ref = oracle.Octree(pts, nrm, offs, d, fd)
        _compare_tree(ref, tree)
        whole = oc.oc_build(torch.as_tensor(pts).cuda(), torch.as_tensor(nrm).cuda(), offs, d, fd)
        torch.cuda.synchronize()
        for l in range(d + 1):
            assert torch.equal(whole.keys(l), tree.keys(l)) and torch.equal(whole.labels(l), tree.labels(l))
            if l:
                assert torch.equal(whole.nbr(l), tree.nbr(l))
        assert torch.equal(whole.signal().view(torch.int32), tree.signal().view(torch.int32))


def test_build_async_errors_and_cancel():
    oc = _gpu()
    bad = torch.tensor([[0.5, 1.5, 0.2]], dtype=torch.float32, device="cuda")
    job = oc.oc_build_async(bad, bad, [0, 1], 3, 2)  # the range check happens on the device
    with pytest.raises(oc.OcError) as e:
        job.finish()
    assert e.value.code == 2
    with pytest.raises(oc.OcError):
        job.finish()  # consumed
    good = torch.tensor([[0.5, 0.25, 0.2], [0.1, 0.9, 0.3]], dtype=torch.float32, device="cuda")
    oc.oc_build_async(good, good, [0, 2], 4, 2).cancel()
    with pytest.raises(oc.OcError) as e:
        oc.oc_build_async(good, good, [0, 2], 9, 2)  # argument errors come back at once
    assert e.value.code == 1
    ref, tree = _build_both(good.cpu().numpy(), good.cpu().numpy(), [0, 2], 4, 2)
    _compare_tree(ref, tree)


def test_allocator_failure_reports_nomem_without_leaks():
    """oc_build with an allocator that fails at its k-th request returns
    OC_ERR_NOMEM, nothing is left allocated, and with enough successes the
    build succeeds and oc_octree_free returns everything."""
    import ctypes as C

    import paper_1712_01537_amd as oc

    L = oc.load()
    pts, nrm, offs = synth.random_cloud(3, 2, 500, "union")
    dp = torch.as_tensor(pts).cuda()
    dn = torch.as_tensor(nrm).cuda()
    offs_h = (C.c_int32 * len(offs))(*[int(v) for v in offs])
    live = {}
    state = {"calls": 0, "fail_at": 0}

    def alloc(ctx, nbytes, stream):
        state["calls"] += 1
        if state["calls"] == state["fail_at"]:
            return None
        t = torch.empty(int(nbytes), dtype=torch.uint8, device="cuda")
        live[t.data_ptr()] = t
        return t.data_ptr()

    def free(ctx, ptr, stream):
        assert live.pop(int(ptr), None) is not None, "freed a pointer it was not given"

    a_cb, f_cb = oc._ALLOC_FN(alloc), oc._FREE_FN(free)
    A = oc._Allocator(a_cb, f_cb, None)
    s = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    for fail_at in (1, 2):  # the scratch, then the octree's arrays
        state.update(calls=0, fail_at=fail_at)
        h = C.c_void_p()
        rc = L.oc_build(C.c_void_p(dp.data_ptr()), C.c_void_p(dn.data_ptr()), offs_h,
                        len(offs) - 1, 4, 2, C.byref(A), s, C.byref(h))
        torch.cuda.synchronize()
        print(f"[nomem] fail at request {fail_at}: status {rc}, "
              f"{L.oc_last_error().decode()}", flush=True)
        assert rc == 3 and not h.value, (fail_at, rc)
        assert live == {}, f"{len(live)} buffers left after a failed build"
    state.update(calls=0, fail_at=0)
    h = C.c_void_p()
    assert L.oc_build(C.c_void_p(dp.data_ptr()), C.c_void_p(dn.data_ptr()), offs_h,
                      len(offs) - 1, 4, 2, C.byref(A), s, C.byref(h)) == 0
    assert state["calls"] == 2 and len(live) == 1  # the scratch went back, the tree stays
    L.oc_octree_free(h)
    torch.cuda.synchronize()
    assert live == {}
