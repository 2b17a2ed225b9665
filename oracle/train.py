"""Plain float64 oracle of the O-CNN(d) training iteration (Sec. 4 "Network
structure", Sec. 5 "Training details"): the basic unit U_l (octree
convolution, batch normalisation, ReLU, 2x2x2 max-pooling), the
classification head (dropout, fully connected layers, softmax with the
cross-entropy loss) and the SGD update with momentum and weight decay.

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: numpy in float64, the
octree operations from the C++ oracle, nothing shared with the HIP library.
Random numbers the method draws (dropout masks, labels, initial weights) are
inputs, drawn by ``synth``.

Readings taken where the paper is brief (stated once, used everywhere):
  * Batch normalisation (the method the paper cites for it, Ioffe and
    Szegedy 2015, in training mode): per channel, the mean and the biased
    variance over every row of the depth's feature map (all N_l octants of
    the batch, empty children included, as every octant carries a feature),
    x_hat = (x - mean) / sqrt(var + eps), y = gamma x_hat + beta, eps = 1e-5.
  * The unit U_l is conv (no bias) -> BN -> ReLU -> 2x2x2 max-pool to depth
    l-1; O-CNN(d) is U_d .. U_2, so the last pooling leaves the eight depth-1
    octants of each shape, all present because the octree is full to depth
    2; their features, in key order, are the shape's input to the head
    (8 C_2 values).  C_l = 2^max(1, 9 - l); the input signal has 3 channels.
  * Dropout with ratio p scales kept values by 1 / (1 - p) during training;
    the keep masks are inputs.
  * FC layers have a bias; weights are [in][out].
  * The loss is the mean over the batch of the cross-entropy of the softmax.
  * SGD as in the paper's framework: v <- mu v + lr (g + lambda w),
    w <- w - v; weight decay applies to the convolution and FC weights, not
    to BN's gamma/beta or the FC biases.
"""
from __future__ import annotations

import numpy as np

from . import (Octree, conv_bwd_data, conv_bwd_weight, conv_fwd, pool_bwd, pool_fwd,
               relu_bwd, relu_fwd)

BN_EPS = 1e-5


def bn_fwd(x, gamma, beta, eps=BN_EPS):
    """Batch normalisation over the rows of x [n][C] (training mode).
    Returns y, and (mean, invstd) for the backward."""
    x = np.asarray(x, np.float64)
    n = x.shape[0]
    mean = x.sum(axis=0) / n
    var = ((x - mean) ** 2).sum(axis=0) / n
    invstd = 1.0 / np.sqrt(var + eps)
    xhat = (x - mean) * invstd
    return xhat * gamma + beta, mean, invstd


def bn_bwd(x, dy, gamma, mean, invstd):
    """Gradients of bn_fwd: dx, dgamma, dbeta (the chain rule through the
    batch statistics)."""
    x = np.asarray(x, np.float64)
    dy = np.asarray(dy, np.float64)
    n = x.shape[0]
    xhat = (x - mean) * invstd
    dbeta = dy.sum(axis=0)
    dgamma = (dy * xhat).sum(axis=0)
    dx = gamma * invstd * (dy - dbeta / n - xhat * dgamma / n)
    return dx, dgamma, dbeta


def fc_fwd(x, w, b):
    """y = x w + b; x [B][in], w [in][out], b [out]."""
    return np.asarray(x, np.float64) @ np.asarray(w, np.float64) + b


def fc_bwd(x, w, dy):
    """dx = dy w^T, dw = x^T dy, db = sum of dy over the batch."""
    x = np.asarray(x, np.float64)
    dy = np.asarray(dy, np.float64)
    return dy @ np.asarray(w, np.float64).T, x.T @ dy, dy.sum(axis=0)


def dropout(x, keep, p):
    """x * keep / (1 - p); keep in {0, 1}, the same shape as x (also the
    backward, applied to dy)."""
    return np.asarray(x, np.float64) * np.asarray(keep, np.float64) / (1.0 - p)


def softmax_ce(z, labels):
    """Mean over the batch of -log softmax(z)[label] and its gradient
    (softmax(z) - onehot(label)) / B; z [B][N_c]."""
    z = np.asarray(z, np.float64)
    B = z.shape[0]
    e = np.exp(z - z.max(axis=1, keepdims=True))
    p = e / e.sum(axis=1, keepdims=True)
    idx = np.arange(B)
    loss = -np.log(p[idx, labels]).sum() / B
    dz = p.copy()
    dz[idx, labels] -= 1.0
    return loss, dz / B


def sgd_step(w, g, v, lr, momentum, decay):
    """One SGD step with momentum and weight decay: returns (w', v')."""
    v = momentum * np.asarray(v, np.float64) + lr * (np.asarray(g, np.float64) + decay * w)
    return w - v, v


def unit_channels(l):
    """C_l = 2^max(1, 9 - l)."""
    return 2 ** max(1, 9 - l)


def ocnn_params(depth, n_classes):
    """Shapes of the parameters of O-CNN(depth) + head, in a fixed order:
    per unit l = depth .. 2: conv weight [27][cin][C_l], gamma [C_l], beta
    [C_l]; then fc1 w [8 C_2][128], b [128]; fc2 w [128][n_classes], b."""
    shapes = []
    cin = 3
    for l in range(depth, 1, -1):
        c = unit_channels(l)
        shapes += [("conv", l, (27, cin, c)), ("gamma", l, (c,)), ("beta", l, (c,))]
        cin = c
    shapes += [("fc1_w", 0, (8 * cin, 128)), ("fc1_b", 0, (128,)),
               ("fc2_w", 0, (128, n_classes)), ("fc2_b", 0, (n_classes,))]
    return shapes


DECAYED = ("conv", "fc1_w", "fc2_w")


def ocnn_step(tree: Octree, params, vel, labels, keep1, keep2, p_drop=0.5, lr=0.1,
              momentum=0.9, decay=5e-4):
    """One training iteration of O-CNN(d) (Sec. 4 and 5) on a built octree.
    params / vel: lists in the order of ocnn_params (float64 arrays);
    labels [B] int; keep1 [B][8 C_2], keep2 [B][128] dropout masks.
    Returns (loss, new params, new velocities, grads, record) where record
    holds the intermediate tensors (for op-by-op comparisons)."""
    d = tree.depth
    B = tree.batch
    x = tree.signal.astype(np.float64)
    rec = {"units": []}
    pi = 0
    for l in range(d, 1, -1):
        w, gamma, beta = params[pi], params[pi + 1], params[pi + 2]
        nb = tree.neighbors(l, 3)
        z = conv_fwd(nb, x, w)
        bn, mean, invstd = bn_fwd(z, gamma, beta)
        a = relu_fwd(bn)
        pooled, sw = pool_fwd(tree.labels(l - 1), a)
        rec["units"].append(dict(l=l, x=x, nb=nb, z=z, bn=bn, mean=mean, invstd=invstd, a=a,
                                 sw=sw, pooled=pooled))
        x = pooled
        pi += 3
    feat = x.reshape(B, -1)  # depth 1: eight rows per shape, in key order
    h0 = dropout(feat, keep1, p_drop)
    h1 = fc_fwd(h0, params[pi], params[pi + 1])
    h2 = dropout(h1, keep2, p_drop)
    z = fc_fwd(h2, params[pi + 2], params[pi + 3])
    loss, dz = softmax_ce(z, labels)
    rec.update(feat=feat, h0=h0, h1=h1, h2=h2, logits=z, dlogits=dz)
    # backward
    grads = [None] * len(params)
    dh2, grads[pi + 2], grads[pi + 3] = fc_bwd(h2, params[pi + 2], dz)
    dh1 = dropout(dh2, keep2, p_drop)
    dh0, grads[pi], grads[pi + 1] = fc_bwd(h0, params[pi], dh1)
    dfeat = dropout(dh0, keep1, p_drop)
    g = dfeat.reshape(x.shape)
    rec["dfeat"] = dfeat
    for u in reversed(rec["units"]):
        pi -= 3
        l = u["l"]
        da = pool_bwd(tree.labels(l - 1), g, u["sw"], tree.num(l))
        dbn = relu_bwd(u["bn"], da)
        dz_, grads[pi + 1], grads[pi + 2] = bn_bwd(u["z"], dbn, params[pi + 1], u["mean"],
                                                   u["invstd"])
        grads[pi] = conv_bwd_weight(u["nb"], u["x"], dz_, 27)
        u.update(da=da, dbn=dbn, dz=dz_)
        g = conv_bwd_data(u["nb"], dz_, params[pi], u["x"].shape[0]) if l < d else None
    # SGD
    kinds = [k for k, _, _ in ocnn_params(d, params[-1].shape[0])]
    new_p, new_v = [], []
    for kind, w, gr, v in zip(kinds, params, grads, vel):
        wn, vn = sgd_step(w, gr, v, lr, momentum, decay if kind in DECAYED else 0.0)
        new_p.append(wn)
        new_v.append(vn)
    return loss, new_p, new_v, grads, rec
