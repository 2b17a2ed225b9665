"""GPU parity of the O-CNN(d) training iteration (the rest of Sec. 4 and 5
around the octree operations): batch normalisation, FC layers, dropout,
softmax cross-entropy and SGD against the float64 oracle (oracle/train.py),
and the bench's whole training step at full size, op by op on the GPU's own
inputs (ReLU and pooling decisions taken from the GPU's values, as in
test_gpu_step), plus its loss against an independent oracle iteration."""
import numpy as np
import pytest
import torch

import oracle
import synth
from helpers import assert_dw_close, assert_f32_close
from oracle import train as T

pytestmark = pytest.mark.gpu


def _np(t):
    return None if t is None else t.detach().cpu().numpy()


def _cuda(a, dtype=torch.float32):
    return torch.as_tensor(np.ascontiguousarray(a)).to(dtype).cuda()


@pytest.mark.parametrize("n,c", [(1, 3), (517, 8), (70001, 16), (2048, 300), (123457, 5)])
def test_bn_small(n, c):
    import paper_1712_01537_amd as oc
    rng = np.random.default_rng(n + c)
    x = (rng.standard_normal((n, c)) * 2 + 0.5).astype(np.float32)
    gamma = (1 + 0.2 * rng.standard_normal(c)).astype(np.float32)
    beta = (0.1 * rng.standard_normal(c)).astype(np.float32)
    dy = rng.standard_normal((n, c)).astype(np.float32)
    print(f"[bn] n={n} c={c}", flush=True)
    for relu in (False, True):
        y, mean, invstd = oc.oc_bn_fwd(_cuda(x), _cuda(gamma), _cuda(beta), relu=relu)
        yr, mr, ir = T.bn_fwd(x, gamma, beta)
        assert_f32_close(_np(mean), mr, "mean", rtol=1e-6, atol=1e-7)
        assert_f32_close(_np(invstd), ir, "invstd", rtol=1e-6, atol=1e-7)
        assert_f32_close(_np(y), np.maximum(yr, 0) if relu else yr, "y")
    dx, dg, db = oc.oc_bn_bwd(_cuda(x), _cuda(dy), _cuda(gamma), mean, invstd)
    dxr, dgr, dbr = T.bn_bwd(x, dy, gamma, mr, ir)
    assert_f32_close(_np(dx), dxr, "dx")
    assert_dw_close(_np(dg), dgr, "dgamma")
    assert_dw_close(_np(db), dbr, "dbeta")
    dx2, dg2, _ = oc.oc_bn_bwd(_cuda(x), _cuda(dy), _cuda(gamma), mean, invstd)
    assert torch.equal(dx, dx2) and torch.equal(dg, dg2)  # reproducible


def test_head_ops_small():
    import paper_1712_01537_amd as oc
    rng = np.random.default_rng(3)
    B, cin, cout, nc = 7, 37, 19, 11
    x = rng.standard_normal((B, cin)).astype(np.float32)
    w = rng.standard_normal((cin, cout)).astype(np.float32)
    b = rng.standard_normal(cout).astype(np.float32)
    dy = rng.standard_normal((B, cout)).astype(np.float32)
    assert_f32_close(_np(oc.oc_fc_fwd(_cuda(x), _cuda(w), _cuda(b))), T.fc_fwd(x, w, b), "fc y")
    dx, dw, db = oc.oc_fc_bwd(_cuda(x), _cuda(w), _cuda(dy))
    dxr, dwr, dbr = T.fc_bwd(x, w, dy)
    assert_f32_close(_np(dx), dxr, "fc dx")
    assert_f32_close(_np(dw), dwr, "fc dw")
    assert_f32_close(_np(db), dbr, "fc db")
    keep = (rng.random((B, cin)) < 0.5).astype(np.uint8)
    np.testing.assert_allclose(_np(oc.oc_dropout(_cuda(x), _cuda(keep, torch.uint8), 0.5)),
                               T.dropout(x, keep, 0.5), rtol=0, atol=0)
    z = (3 * rng.standard_normal((B, nc))).astype(np.float32)
    labels = rng.integers(0, nc, B).astype(np.int32)
    loss, dz = oc.oc_softmax_ce(_cuda(z), _cuda(labels, torch.int32))
    lr, dzr = T.softmax_ce(z, labels)
    assert abs(float(loss) - lr) <= 1e-6 + 1e-5 * abs(lr)
    assert_f32_close(_np(dz), dzr, "dz")
    wv = rng.standard_normal(1000).astype(np.float32)
    g = rng.standard_normal(1000).astype(np.float32)
    v = rng.standard_normal(1000).astype(np.float32)
    wt, vt = _cuda(wv), _cuda(v)
    oc.oc_sgd(wt, _cuda(g), vt, 0.1, 0.9, 5e-4)
    wr, vr = T.sgd_step(wv, g, v, 0.1, 0.9, 5e-4)
    assert_f32_close(_np(wt), wr, "sgd w")
    assert_f32_close(_np(vt), vr, "sgd v")


@pytest.mark.parametrize("seed,B,n,depth,c,relu", [(61, 2, 500, 4, 8, True),
                                                    (62, 3, 300, 5, 16, False),
                                                    (63, 1, 200, 3, 3, True)])
def test_bn_pool_fused(seed, B, n, depth, c, relu):
    """Normalisation + ReLU + 2x2x2 max-pool in one call: bit-identical to the
    two calls, and the oracle's normalisation and pooling."""
    import paper_1712_01537_amd as oc
    pts, nrm, offs = synth.random_cloud(seed, B, n, "union")
    ref = oracle.Octree(pts, nrm, offs, depth, 2)
    tree = oc.oc_build(torch.as_tensor(pts).cuda(), torch.as_tensor(nrm).cuda(), offs, depth, 2)
    l = depth
    rng = np.random.default_rng(seed)
    z = (2 * rng.standard_normal((ref.num(l), c)) + 0.3).astype(np.float32)
    g = rng.uniform(0.5, 1.5, c).astype(np.float32)
    b = rng.standard_normal(c).astype(np.float32)
    y, sw, mean, invstd = oc.oc_bn_pool_fwd(tree, l, _cuda(z), _cuda(g), _cuda(b), relu=relu)
    a, mean2, invstd2 = oc.oc_bn_fwd(_cuda(z), _cuda(g), _cuda(b), relu=relu)
    yu, swu = oc.oc_pool_fwd(tree, l, a)
    assert torch.equal(y.view(torch.int32), yu.view(torch.int32)) and torch.equal(sw, swu)
    assert torch.equal(mean, mean2) and torch.equal(invstd, invstd2)
    bn, mr, ir = T.bn_fwd(z, g, b)
    assert_f32_close(_np(mean), mr, "mean", rtol=1e-6, atol=1e-7)
    assert_f32_close(_np(invstd), ir, "invstd", rtol=1e-6, atol=1e-7)
    yr, _ = oracle.pool_fwd(ref.labels(l - 1), np.maximum(bn, 0) if relu else bn)
    assert_f32_close(_np(y), yr, "pooled")
    po, swo = oracle.pool_fwd(ref.labels(l - 1), _np(a))  # the GPU's own values: exact
    np.testing.assert_array_equal(_np(y), po)
    np.testing.assert_array_equal(_np(sw), swo)
    tree.free()


def test_training_step_full_size():
    import bench
    import paper_1712_01537_amd as oc

    wl = synth.WORKLOADS["ocnn_d6"]
    print("[train] building the bench's training step", flush=True)
    step = bench.TrainStep(oc, torch, synth, wl)
    pts, nrm, offs = synth.make_points(wl)
    tree = oc.oc_build(step.pts, step.nrm, offs, wl.depth, wl.full_depth)
    ref = oracle.Octree(pts, nrm, offs, wl.depth, wl.full_depth)
    step.record = {}
    step.network(tree)
    torch.cuda.synchronize()
    rec = step.record
    d = synth.make_train_inputs(wl)
    print("[train] forward", flush=True)
    acts = {}  # the depth-l activations the fused call does not keep, recomputed
    for li, xin, z, a, mean, invstd, p, sw in rec["units"]:
        L = wl.layers[li]
        l = L.depth
        if a is None:
            # the same normalisation on the GPU, unpooled (bit-identical to
            # what the fused call pools: a test of the operations), with the
            # parameters before the update
            gb = d["bn"][li]
            a, mean2, invstd2 = oc.oc_bn_fwd(z, _cuda(gb[0]), _cuda(gb[1]), relu=True)
            assert torch.equal(mean2, mean) and torch.equal(invstd2, invstd)
        acts[li] = a
        x_, z_, a_ = _np(xin), _np(z), _np(a)
        w = _np(rec["before"]["dec"]["w"])  # conv weights are at the head of the buffer
        off = sum(27 * M.cin * M.cout for M in wl.layers[:li])
        w = w[off:off + 27 * L.cin * L.cout].reshape(27, L.cin, L.cout)
        if li == 0:
            assert_f32_close(x_, ref.signal, "signal", rtol=1e-6, atol=1e-7)
        nb = ref.neighbors(l, 3)
        assert_f32_close(z_, oracle.conv_fwd(nb, x_, w), f"unit {l} conv")
        g, b = d["bn"][li]
        bn, mr, ir = T.bn_fwd(z_, g, b)
        assert_f32_close(_np(mean), mr, f"unit {l} mean", rtol=1e-6, atol=1e-7)
        assert_f32_close(a_, np.maximum(bn, 0), f"unit {l} bn+relu")
        pr, swr = oracle.pool_fwd(ref.labels(l - 1), a_)
        np.testing.assert_array_equal(_np(p), pr)
        np.testing.assert_array_equal(_np(sw), swr)
    feat = _np(rec["feat"])
    h0 = T.dropout(feat, d["keep1"], 0.5)
    assert_f32_close(_np(rec["h0"]), h0, "h0")
    assert_f32_close(_np(rec["h1"]), T.fc_fwd(_np(rec["h0"]), d["fc1_w"], d["fc1_b"]), "h1")
    assert_f32_close(_np(rec["logits"]), T.fc_fwd(_np(rec["h2"]), d["fc2_w"], d["fc2_b"]),
                     "logits")
    lr_, dzr = T.softmax_ce(_np(rec["logits"]), d["labels"])
    assert abs(float(rec["loss"]) - lr_) <= 1e-5 * abs(lr_)
    assert_f32_close(_np(rec["dlogits"]), dzr, "dlogits")
    print("[train] backward", flush=True)
    for li, xin, z, a, mean, invstd, p, sw in reversed(rec["units"]):
        L = wl.layers[li]
        l = L.depth
        g_in, da, dz_, _ = (_np(t) for t in rec["bwd"][li])
        if g_in is not None:  # the head's gradient, routed by its own call
            da_r = oracle.relu_bwd(_np(acts[li]), oracle.pool_bwd(ref.labels(l - 1), g_in,
                                                          _np(sw), ref.num(l)))
            np.testing.assert_array_equal(da, da_r)
        else:
            # routed by the unit above in the same call as its input gradient
            U = wl.layers[li + 1]
            off_u = sum(27 * M.cin * M.cout for M in wl.layers[:li + 1])
            w_u = _np(rec["before"]["dec"]["w"])[off_u:off_u + 27 * U.cin * U.cout].reshape(
                27, U.cin, U.cout)
            dx_u = oracle.conv_bwd_data(ref.neighbors(l - 1, 3), _np(rec["bwd"][li + 1][2]), w_u,
                                        ref.num(l - 1))
            da_r = oracle.relu_bwd(_np(acts[li]), oracle.pool_bwd(ref.labels(l - 1), dx_u,
                                                          _np(sw), ref.num(l)))
            assert_f32_close(da, da_r, f"unit {l} routed dx")
        g, b = d["bn"][li]
        dzr, dgr, dbr = T.bn_bwd(_np(z), da, g, *T.bn_fwd(_np(z), g, b)[1:])
        assert_f32_close(dz_, dzr, f"unit {l} bn dx")
        nb = ref.neighbors(l, 3)
        off = sum(27 * M.cin * M.cout for M in wl.layers[:li])
        w = _np(rec["before"]["dec"]["w"])[off:off + 27 * L.cin * L.cout].reshape(27, L.cin, L.cout)
        gw = _np(step.conv_p[li]["g"])
        rule = assert_dw_close(gw, oracle.conv_bwd_weight(nb, _np(xin), dz_, 27), f"unit {l} dW")
        print(f"[train] unit {l} dW rule: {rule}", flush=True)
        # (the input gradient of units above the first is checked, routed, with the unit below)
    # the update, on the GPU's gradients
    for key, dec in (("dec", step.DECAY), ("pla", 0.0)):
        b = step.flat[key]
        wr, vr = T.sgd_step(_np(rec["before"][key]["w"]), _np(b["g"]),
                            _np(rec["before"][key]["v"]), step.LR, step.MOMENTUM, dec)
        assert_f32_close(_np(b["w"]), wr, f"sgd {key} w")
        assert_f32_close(_np(b["v"]), vr, f"sgd {key} v")
    # the loss of an independent float64 iteration of the oracle
    params = []
    for li, L in enumerate(wl.layers):
        params += [synth.make_weights(wl, li, 3, L.cin, L.cout).astype(np.float64),
                   d["bn"][li][0].astype(np.float64), d["bn"][li][1].astype(np.float64)]
    params += [d["fc1_w"], d["fc1_b"], d["fc2_w"], d["fc2_b"]]
    params = [np.asarray(q, np.float64) for q in params]
    loss64 = T.ocnn_step(ref, params, [np.zeros_like(q) for q in params], d["labels"],
                         d["keep1"], d["keep2"])[0]
    print(f"[train] loss GPU {float(rec['loss']):.7f} oracle {loss64:.7f}", flush=True)
    assert abs(float(rec["loss"]) - loss64) <= 1e-4 * abs(loss64)
    tree.free()
