"""The LeNet-style SGD-momentum training step composed from oracle calls.

conv(1->32, 5x5, p2)+relu -> maxpool 2x2/2 -> conv(32->64, 5x5, p2)+relu ->
maxpool 2x2/2 -> affine 3136->512 + relu -> affine 512->10 -> softmax +
cross-entropy; backward in reverse; then v <- mu v - lr g, theta <- theta + v
for the eight parameter tensors (the paper's Section 2 training loop for its
example network, with the momentum update of Section 3 "Optimizers").
Test infrastructure like the rest of the oracle: composes only the oracle's
functions.
"""
import numpy as np

from . import (affine_bwd, affine_fwd, conv2d_backward_data, conv2d_backward_filter,
               conv2d_forward, max_pool2d_bwd, max_pool2d_fwd, sgd_momentum_update,
               softmax_forward, softmax_xent)

PARAM_ORDER = ("W1", "b1", "W2", "b2", "W3", "b3", "W4", "b4")


def forward_backward(X, Y, p):
    """Returns (loss, grads dict, activations dict)."""
    a = {}
    a["c1"], _, _ = conv2d_forward(X, p["W1"], p["b1"], 1, 28, 28, 5, 5, 1, 2, relu=True)
    a["p1"], a["i1"], _, _ = max_pool2d_fwd(a["c1"], 32, 28, 28, 2, 2, 2, 0)
    a["c2"], _, _ = conv2d_forward(a["p1"], p["W2"], p["b2"], 32, 14, 14, 5, 5, 1, 2,
                                          relu=True)
    a["p2"], a["i2"], _, _ = max_pool2d_fwd(a["c2"], 64, 14, 14, 2, 2, 2, 0)
    a["h"] = affine_fwd(a["p2"], p["W3"], p["b3"], relu=True)
    a["s"] = affine_fwd(a["h"], p["W4"], p["b4"], relu=False)
    loss, ds, _ = softmax_xent(a["s"], Y, want_probs=False)
    g = {}
    dh, g["W4"], g["b4"] = affine_bwd(ds, a["h"], p["W4"], None)
    dp2, g["W3"], g["b3"] = affine_bwd(dh, a["p2"], p["W3"], a["h"])
    dc2 = max_pool2d_bwd(dp2, a["i2"], 64, 14, 14, 2, 2, 2, 0)
    g["W2"], g["b2"] = conv2d_backward_filter(a["p1"], dc2, a["c2"], 32, 14, 14, 5, 5,
                                                     1, 2, 64)
    dp1 = conv2d_backward_data(p["W2"], dc2, a["c2"], 32, 14, 14, 5, 5, 1, 2)
    dc1 = max_pool2d_bwd(dp1, a["i1"], 32, 28, 28, 2, 2, 2, 0)
    g["W1"], g["b1"] = conv2d_backward_filter(X, dc1, a["c1"], 1, 28, 28, 5, 5, 1, 2, 32)
    return loss, g, a


def train_step(X, Y, params, vel, lr=0.01, mu=0.9):
    """One step; returns (loss, new params, new velocities, grads, activations)."""
    loss, g, a = forward_backward(X, Y, params)
    newp, newv = {}, {}
    for k in PARAM_ORDER:
        th, v = sgd_momentum_update(params[k], g[k], vel[k], lr, mu)
        newp[k] = th.reshape(params[k].shape)
        newv[k] = v.reshape(params[k].shape)
    return loss, newp, newv, g, a


def zero_velocities(params):
    return {k: np.zeros_like(v) for k, v in params.items()}


def forward_probs(X, p):
    """Forward-only scoring: class probabilities of each row of X."""
    c1, _, _ = conv2d_forward(X, p["W1"], p["b1"], 1, 28, 28, 5, 5, 1, 2, relu=True)
    p1, _, _, _ = max_pool2d_fwd(c1, 32, 28, 28, 2, 2, 2, 0)
    c2, _, _ = conv2d_forward(p1, p["W2"], p["b2"], 32, 14, 14, 5, 5, 1, 2, relu=True)
    p2, _, _, _ = max_pool2d_fwd(c2, 64, 14, 14, 2, 2, 2, 0)
    h = affine_fwd(p2, p["W3"], p["b3"], relu=True)
    s = affine_fwd(h, p["W4"], p["b4"], relu=False)
    return softmax_forward(s)
