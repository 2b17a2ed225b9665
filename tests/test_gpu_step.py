"""The timed step of the bench, end to end at full size: the call sequence
bench.py runs (fused ReLU in the forward, conv + ReLU + pool in one call
where a pooling follows a convolution, the ReLU's backward inside the
pooling's routing, a convolution's input gradient routed through the
pooling below it in one call, no input gradient for the first layer,
separate input- and weight-gradient calls) on the octree the GPU builds, every tensor of the
step against the oracle.

Each op is checked on the GPU's own inputs to that op, so errors do not
compound, and the oracle takes the decisions that floating point makes
(ReLU signs, pooling maxima) from the GPU's values: the ReLU mask of a
backward is [y > 0] of the GPU's forward output, the routing uses the GPU's
switches.  Those decisions are themselves checked: the forward output is
within the fp32 rule of the oracle's ReLU(pre-activation) everywhere (ReLU is
1-Lipschitz), and the switches are bit-exact against the oracle's pooling of
the GPU's convolution output (a max over identical values is exact)."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_dw_close, assert_f32_close

pytestmark = pytest.mark.gpu


def _np(t):
    return None if t is None else t.detach().cpu().numpy()


@pytest.mark.parametrize("name", ["net_d6", "seg_d6"])
def test_bench_step_end_to_end(name):
    import bench
    import paper_1712_01537_amd as oc

    wl = synth.WORKLOADS[name]
    print(f"[step] {name}: building the bench's step", flush=True)
    step = bench.Step(oc, torch, synth, wl)
    pts, nrm, offs = synth.make_points(wl)
    tree = oc.oc_build(step.pts, step.nrm, offs, wl.depth, wl.full_depth)
    ref = oracle.Octree(pts, nrm, offs, wl.depth, wl.full_depth)
    for l in range(wl.depth + 1):
        assert np.array_equal(tree.labels(l).cpu().numpy(), ref.labels(l)), l
    step.record = {}
    step.network(tree)
    torch.cuda.synchronize()
    fwd, bwd = step.record["fwd"], step.record["bwd"]
    print(f"[step] {name}: forward", flush=True)
    unpooled = {}  # depth-l outputs of conv + pool calls, recomputed unpooled
    for li, L in enumerate(wl.layers):
        x, y, sw = (_np(t) for t in fwd[li])
        l = L.depth
        if li == 0 and wl.signal_input:
            assert_f32_close(x, ref.signal, "signal", rtol=1e-6, atol=1e-7)
        if L.op == "conv" and y is None:
            # run with the pooling above it in one call: its output here is
            # the same kernel's unpooled forward on the same inputs (the two
            # agree bit for bit, a test of the operations)
            assert step.pooled(li)
            y = _np(oc.oc_conv_fwd(tree, l, L.ksize, L.stride, fwd[li][0], step.weights[li],
                                   relu=L.relu))
            unpooled[li + 1] = y
        elif L.op == "pool" and x is None:
            x = unpooled[li]
        if L.op == "conv":
            nb = ref.neighbors(l, L.ksize, stride=L.stride)
            pre = oracle.conv_fwd(nb, x, _np(step.weights[li]))
            r = L.stride.bit_length() - 1
            if r:
                pre = oracle.renew(ref.labels(l - r), pre)
            assert_f32_close(y, oracle.relu_fwd(pre) if L.relu else pre, f"{name}/{li} y")
        elif L.op == "deconv":
            w = _np(step.weights[li])
            yr = (oracle.deconv_fwd(ref.neighbors(l, L.ksize), x, w, ref.num(l)) if L.stride == 1
                  else oracle.deconv_s2_fwd(ref, l, x, w))
            assert_f32_close(y, yr, f"{name}/{li} y")
        elif L.op == "pool":
            yr, swr = oracle.pool_fwd(ref.labels(l - 1), x)
            np.testing.assert_array_equal(y, yr)
            np.testing.assert_array_equal(sw, swr)
        elif L.op == "unpool":
            np.testing.assert_array_equal(
                y, oracle.unpool_fwd(ref.labels(l - 1), x, sw, ref.num(l)))
    print(f"[step] {name}: backward", flush=True)
    np.testing.assert_array_equal(_np(bwd[len(wl.layers) - 1][0]), _np(step.dy_last))
    for li in reversed(range(len(wl.layers))):
        L = wl.layers[li]
        l = L.depth
        g_in, g_out, dw = (_np(t) for t in bwd[li])
        x, y, sw = (_np(t) for t in fwd[li])
        if L.op == "pool" and x is None:
            x = unpooled[li]
        if L.op == "conv":
            nb = ref.neighbors(l, L.ksize, stride=L.stride)
            w = _np(step.weights[li])
            # the ReLU's backward is in this call only when no pooling above
            # applied it already (the bench's rule)
            above = wl.layers[li + 1] if li + 1 < len(wl.layers) else None
            masked_above = above is not None and above.op == "pool"
            ge = oracle.relu_bwd(y, g_in) if (L.relu and not masked_above) else g_in
            r = L.stride.bit_length() - 1
            if r:
                ge = oracle.renew_bwd(ref.labels(l - r), ge, nb.shape[0])
            rule = assert_dw_close(dw, oracle.conv_bwd_weight(nb, x, ge, L.ksize ** 3),
                                   f"{name}/{li} dw")
            print(f"[step] {name}/{li} dw rule: {rule}", flush=True)
            if li == 0:
                assert g_out is None  # the signal needs no gradient
            elif g_out is None:
                # the input gradient went on through the pooling below in the
                # same call: check the routed gradient the pooling recorded
                assert step.routed_pool(li) == li - 1
                _, routed_gpu, _ = (_np(t) for t in bwd[li - 1])
                px, _, psw = (_np(t) for t in fwd[li - 1])
                if px is None:
                    px = unpooled[li - 1]
                routed = oracle.pool_bwd(ref.labels(l), oracle.conv_bwd_data(nb, ge, w, x.shape[0]),
                                         psw, ref.num(l + 1))
                if step.pool_mask(li - 1):
                    routed = oracle.relu_bwd(px, routed)  # the ReLU below, on the GPU's values
                assert_f32_close(routed_gpu, routed, f"{name}/{li} dx routed")
            else:
                assert_f32_close(g_out, oracle.conv_bwd_data(nb, ge, w, x.shape[0]),
                                 f"{name}/{li} dx")
        elif L.op == "deconv":
            w = _np(step.weights[li])
            if L.stride == 1:
                dxr, dwr = oracle.deconv_bwd(ref.neighbors(l, L.ksize), x, w, g_in)
            else:
                dxr, dwr = oracle.deconv_s2_bwd(ref, l, x, w, g_in)
            assert_f32_close(g_out, dxr, f"{name}/{li} dx")
            assert_dw_close(dw, dwr, f"{name}/{li} dw")
        elif L.op == "pool" and g_in is None:
            continue  # routed with the input gradient of the conv above (checked there)
        elif L.op == "pool":
            routed = oracle.pool_bwd(ref.labels(l - 1), g_in, sw, ref.num(l))
            below = wl.layers[li - 1] if li > 0 else None
            if below is not None and below.op == "conv" and below.relu:
                routed = oracle.relu_bwd(x, routed)  # the ReLU below, on the GPU's values
            np.testing.assert_array_equal(g_out, routed)
        elif L.op == "unpool":
            np.testing.assert_array_equal(g_out, oracle.unpool_bwd(ref.labels(l - 1), g_in, sw))
    tree.free()
    print(f"[step] {name}: every tensor of the step matches", flush=True)


def _same_tensors(got, want, where):
    if isinstance(got, dict):
        assert got.keys() == want.keys(), where
        for k in got:
            _same_tensors(got[k], want[k], f"{where}/{k}")
    elif isinstance(got, (tuple, list)):
        assert len(got) == len(want), where
        for i, (a, b) in enumerate(zip(got, want)):
            _same_tensors(a, b, f"{where}/{i}")
    elif got is None or want is None:
        assert got is None and want is None, where
    else:
        assert torch.equal(got, want), where


@pytest.mark.parametrize("name", ["net_d6", "wide_d7"])
def test_bench_step_build_stream(name):
    """The timed step with the next batch's build on its own stream, started
    after the forward of the layer the bench names for this network: after
    several steps, every tensor of the network (outputs, switches, input and
    weight gradients) equals bit for bit that of the same network on an
    octree built alone, and the octree built for the next step equals a
    direct build at every depth.  The kernels are deterministic, so any
    difference is an ordering fault between the two streams."""
    import bench
    import paper_1712_01537_amd as oc

    wl = synth.WORKLOADS[name]
    print(f"[step] {name}: two-stream steps", flush=True)
    step = bench.Step(oc, torch, synth, wl)
    assert step.build_after == bench.BUILD_AFTER[name]
    step.bstream = torch.cuda.Stream()
    for _ in range(3):
        step()
    step.record = {}
    step()
    torch.cuda.synchronize()
    got = step.record
    _, _, offs = synth.make_points(wl)
    tree = oc.oc_build(step.pts, step.nrm, offs, wl.depth, wl.full_depth)
    for l in range(wl.depth + 1):
        assert torch.equal(step.cur.labels(l), tree.labels(l)), l
    print(f"[step] {name}: one-stream reference", flush=True)
    step.record = {}
    step.network(tree)
    torch.cuda.synchronize()
    want = step.record
    # the first layer's input may be the freed octree's signal: left out
    got["fwd"][0] = got["fwd"][0][1:]
    want["fwd"][0] = want["fwd"][0][1:]
    _same_tensors(got, want, name)
