"""Pins of the training-iteration oracle (oracle/train.py) against float64
torch on the CPU: batch normalisation (training mode) and its autograd,
linear layers, softmax cross-entropy, SGD with momentum and weight decay, and
central differences of the whole O-CNN(d) loss with respect to parameters of
every kind."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth
from oracle import train as T


def test_bn_matches_torch_batch_norm():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((37, 5)) * 3 + 1
    gamma, beta = rng.standard_normal(5), rng.standard_normal(5)
    dy = rng.standard_normal((37, 5))
    y, mean, invstd = T.bn_fwd(x, gamma, beta)
    xt = torch.tensor(x, requires_grad=True)
    gt = torch.tensor(gamma, requires_grad=True)
    bt = torch.tensor(beta, requires_grad=True)
    yt = F.batch_norm(xt, None, None, gt, bt, training=True, eps=T.BN_EPS)
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-12, atol=1e-12)
    yt.backward(torch.tensor(dy))
    dx, dg, db = T.bn_bwd(x, dy, gamma, mean, invstd)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)


def test_fc_and_softmax_ce_match_torch():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((6, 11))
    w, b = rng.standard_normal((11, 4)), rng.standard_normal(4)
    labels = np.array([0, 3, 1, 1, 2, 3])
    xt = torch.tensor(x, requires_grad=True)
    wt = torch.tensor(w, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    zt = F.linear(xt, wt.T, bt)
    z = T.fc_fwd(x, w, b)
    np.testing.assert_allclose(z, zt.detach().numpy(), rtol=1e-12, atol=1e-12)
    loss_t = F.cross_entropy(zt, torch.tensor(labels))
    loss, dz = T.softmax_ce(z, labels)
    assert abs(loss - loss_t.item()) < 1e-12
    loss_t.backward()
    dx, dw, db = T.fc_bwd(x, w, dz)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-12)
    # large logits: the shift keeps the softmax finite
    l2, _ = T.softmax_ce(z + 1000.0, labels)
    assert abs(l2 - loss) < 1e-9


def test_dropout_special_cases_and_adjoint():
    rng = np.random.default_rng(3)
    x, v = rng.standard_normal((5, 7)), rng.standard_normal((5, 7))
    keep = rng.random((5, 7)) < 0.5
    np.testing.assert_array_equal(T.dropout(x, np.ones_like(x), 0.0), x)
    np.testing.assert_array_equal(T.dropout(x, np.ones_like(x), 0.5), 2 * x)
    assert not T.dropout(x, np.zeros_like(x), 0.5).any()
    # a diagonal operator: <dropout(x), v> = <x, dropout(v)>
    assert np.isclose(np.sum(T.dropout(x, keep, 0.5) * v), np.sum(x * T.dropout(v, keep, 0.5)))


def test_sgd_matches_torch_optimizer():
    rng = np.random.default_rng(4)
    w0 = rng.standard_normal(9)
    grads = [rng.standard_normal(9) for _ in range(4)]
    wt = torch.tensor(w0, requires_grad=True)
    opt = torch.optim.SGD([wt], lr=0.1, momentum=0.9, weight_decay=5e-4)
    w, v = w0.copy(), np.zeros(9)
    for g in grads:
        wt.grad = torch.tensor(g)
        opt.step()
        w, v = T.sgd_step(w, g, v, 0.1, 0.9, 5e-4)
        np.testing.assert_allclose(w, wt.detach().numpy(), rtol=1e-12, atol=1e-14)


def _setup(depth=4, B=2, n=300, seed=5, classes=5):
    pts, nrm, offs = synth.random_cloud(seed, B, n, "union")
    tree = oracle.Octree(pts, nrm, offs, depth, 2)
    rng = np.random.default_rng(seed)
    params = []
    for kind, _, shape in T.ocnn_params(depth, classes):
        if kind == "gamma":
            params.append(1 + 0.1 * rng.standard_normal(shape))
        elif kind in ("beta", "fc1_b", "fc2_b"):
            params.append(0.1 * rng.standard_normal(shape))
        else:
            params.append(rng.standard_normal(shape) / np.sqrt(np.prod(shape[:-1])))
    c2 = T.unit_channels(2)
    keep1 = rng.random((B, 8 * c2)) < 0.5
    keep2 = rng.random((B, 128)) < 0.5
    labels = rng.integers(0, classes, B)
    return tree, params, keep1, keep2, labels


def test_ocnn_step_gradients_by_central_differences():
    tree, params, keep1, keep2, labels = _setup()
    vel = [np.zeros_like(p) for p in params]
    loss, new_p, new_v, grads, _ = T.ocnn_step(tree, params, vel, labels, keep1, keep2)
    kinds = T.ocnn_params(tree.depth, 5)
    rng = np.random.default_rng(9)
    h = 1e-6
    for i, (kind, l, shape) in enumerate(kinds):
        for _ in range(2):
            j = tuple(int(rng.integers(0, s)) for s in shape)
            pp = [p.copy() for p in params]
            pp[i][j] += h
            lp = T.ocnn_step(tree, pp, vel, labels, keep1, keep2)[0]
            pp[i][j] -= 2 * h
            lm = T.ocnn_step(tree, pp, vel, labels, keep1, keep2)[0]
            fd = (lp - lm) / (2 * h)
            assert abs(fd - grads[i][j]) <= 1e-5 * max(1.0, abs(fd)), (kind, l, j, fd, grads[i][j])
    # the update: v = lr (g + decay w) from zero velocity, w' = w - v
    for (kind, _, _), p, g, pn, vn in zip(kinds, params, grads, new_p, new_v):
        dec = 5e-4 if kind in T.DECAYED else 0.0
        np.testing.assert_allclose(vn, 0.1 * (g + dec * p), rtol=1e-12, atol=1e-15)
        np.testing.assert_allclose(pn, p - vn, rtol=1e-12, atol=1e-15)
    assert np.isfinite(loss) and loss > 0
