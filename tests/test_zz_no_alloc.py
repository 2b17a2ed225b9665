"""oc_conv_fwd_noalloc, the forward whose workspace is the library's static
device array (for callers that cannot allocate), through the C ABI: bit-for-
bit the output of oc_conv_fwd on two calls in a row, the second smaller, so
the second runs on the first's leftover scratch contents; calls whose
workspace would exceed the array are refused."""
import ctypes as C

import numpy as np
import pytest
import torch

import synth

pytestmark = pytest.mark.gpu


def _raw_noalloc(L, tree, depth, K, x, w, y, relu):
    dt = 1 if x.dtype == torch.bfloat16 else 0
    return L.oc_conv_fwd_noalloc(tree.handle, depth, K, 1, dt, C.c_void_p(x.data_ptr()),
                                 x.shape[1], C.c_void_p(w.data_ptr()), w.shape[2],
                                 C.c_void_p(y.data_ptr()), 1 if relu else 0,
                                 C.c_void_p(torch.cuda.current_stream().cuda_stream))


def test_noalloc_matches_workspace_forward():
    import paper_1712_01537_amd as oc

    L = oc.load()
    wl = synth.WORKLOADS["net_d6"]
    pts, nrm, offs = synth.make_points(wl)
    tree = oc.oc_build(torch.as_tensor(pts).cuda(), torch.as_tensor(nrm).cuda(), offs, wl.depth,
                       wl.full_depth)
    rng = np.random.default_rng(11)
    cap = 32 << 20

    def need(depth, K, cin, cout, dt):
        return L.oc_conv_fwd_workspace(tree.handle, depth, K, 1,
                                       1 if dt == torch.bfloat16 else 0, cin, cout)

    # the network's fp32 layers whose workspace (split reduction partials)
    # fits the static array, most rows first: each later call is smaller and
    # runs on the scratch the previous one left
    layers = [(d, 3, ci, co, torch.float32) for d, ci, co in
              ((5, 16, 32), (4, 32, 64), (3, 64, 128), (2, 128, 256))]
    fit = [c for c in layers if 0 < need(*c) <= cap]
    assert len(fit) >= 2, [need(*c) for c in layers]
    cases = [fit[0] + (True,), fit[1] + (False,),
             (5, 5, 32, 32, torch.bfloat16, False), (4, 5, 16, 32, torch.bfloat16, True)]
    for depth, K, cin, cout, dt, relu in cases:
        n = tree.num(depth)
        x = torch.as_tensor(rng.standard_normal((n, cin)).astype(np.float32)).cuda().to(dt)
        w = torch.as_tensor((rng.standard_normal((K ** 3, cin, cout)) / np.sqrt(27 * cin))
                            .astype(np.float32)).cuda().to(dt)
        print(f"[noalloc] d{depth} K{K} {cin}->{cout} {dt} rows {n} workspace "
              f"{need(depth, K, cin, cout, dt)} bytes", flush=True)
        ref = oc.oc_conv_fwd(tree, depth, K, 1, x, w, relu=relu)
        y = torch.full((n, cout), float("nan"), device="cuda")
        assert _raw_noalloc(L, tree, depth, K, x, w, y, relu) == 0, L.oc_last_error()
        torch.cuda.synchronize()
        assert torch.equal(y.view(torch.int32), ref.view(torch.int32)), (depth, K, cin, cout)
    # a call needing more than the static array is refused, nothing written
    n = tree.num(6)
    x = torch.zeros((n, 24), dtype=torch.bfloat16, device="cuda")  # widened to fp32: 50 MB
    w = torch.zeros((27, 24, 16), dtype=torch.bfloat16, device="cuda")
    y = torch.full((n, 16), 7.0, device="cuda")
    assert need(6, 3, 24, 16, torch.bfloat16) > cap
    assert _raw_noalloc(L, tree, 6, 3, x, w, y, False) == 5  # OC_ERR_UNSUPPORTED
    assert b"static scratch" in L.oc_last_error()
    torch.cuda.synchronize()
    assert bool((y == 7.0).all())
    tree.free()
