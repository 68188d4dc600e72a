"""Pins for the oracle's max-pool, bias_add_relu, affine, softmax/cross-entropy,
SGD-momentum and count_nonzero (CPU only).

References: torch CPU routines (max_pool2d with indices, autograd, softmax,
cross_entropy), numpy matmul/sum, closed forms (uniform scores give ln K, the
two-step momentum recurrence), invariants (row sums, shift invariance, gradient
routing) and the unfused chain in the order the paper's listing composes it.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as tF

import oracle
from paper_1802_04647_amd.inputs import rng


def _rel(a, b):
    den = np.max(np.abs(b))
    return np.max(np.abs(a - b)) / (den if den > 0 else 1.0)


# ----------------------------------------------------------------------------- pool
POOLS = [  # (N, C, H, W, Hf, Wf, s, p)
    (2, 3, 8, 8, 2, 2, 2, 0),
    (2, 2, 7, 9, 3, 3, 2, 1),
    (1, 2, 6, 5, 2, 3, 1, 1),
    (2, 1, 9, 9, 3, 2, 3, 0),
]


@pytest.mark.parametrize("cfg", POOLS, ids=str)
def test_pool_matches_torch_including_ties(cfg):
    N, C, H, W, Hf, Wf, s, p = cfg
    g = rng(21)
    # quantised values produce many ties; relu-like zeros too
    X = np.maximum(np.round(g.standard_normal((N, C * H * W)) * 2) / 2, 0.0)
    out, idx, Ho, Wo = oracle.max_pool2d_fwd(X, C, H, W, Hf, Wf, s, p)
    x = torch.from_numpy(X.reshape(N, C, H, W)).requires_grad_()
    y, ti = tF.max_pool2d(x, (Hf, Wf), s, p, return_indices=True)
    assert y.shape[2:] == (Ho, Wo)
    assert np.array_equal(out, y.detach().reshape(N, -1).numpy())
    # torch's index is within one channel plane; ours is the in-row column index
    plane = (np.arange(C) * H * W)[None, :, None]
    assert np.array_equal(idx, (ti.reshape(N, C, -1).numpy() + plane).reshape(N, -1))
    dout = g.standard_normal(out.shape)
    y.backward(torch.from_numpy(dout.reshape(y.shape)))
    dX = oracle.max_pool2d_bwd(dout, idx, C, H, W, Hf, Wf, s, p)
    assert _rel(dX, x.grad.reshape(N, -1).numpy()) < 1e-15


def test_pool_argmax_position_rules():
    H = W = 4
    inc = np.arange(16, dtype=np.float64)[None, :]
    _, idx, _, _ = oracle.max_pool2d_fwd(inc, 1, H, W, 2, 2, 2, 0)
    assert list(idx[0]) == [5, 7, 13, 15]          # bottom-right of each window
    _, idx, _, _ = oracle.max_pool2d_fwd(-inc, 1, H, W, 2, 2, 2, 0)
    assert list(idx[0]) == [0, 2, 8, 10]           # top-left
    _, idx, _, _ = oracle.max_pool2d_fwd(np.zeros((1, 16)), 1, H, W, 2, 2, 2, 0)
    assert list(idx[0]) == [0, 2, 8, 10]           # ties: first in row-major order
    sz = np.zeros((1, 16))
    sz[0, [0, 2, 8, 10]] = -0.0
    _, idx2, _, _ = oracle.max_pool2d_fwd(sz, 1, H, W, 2, 2, 2, 0)
    assert list(idx2[0]) == [0, 2, 8, 10]          # signed zeros compare equal


def test_pool_padding_never_selected():
    X = -np.ones((1, 9)) * 5.0                     # all inputs below the pad's "0"
    out, idx, Ho, Wo = oracle.max_pool2d_fwd(X, 1, 3, 3, 2, 2, 1, 1)
    assert (Ho, Wo) == (4, 4)
    assert (out == -5.0).all() and (idx >= 0).all() and (idx < 9).all()


def test_pool_backward_routes_and_conserves():
    g = rng(22)
    N, C, H, W = 2, 3, 6, 6
    X = g.standard_normal((N, C * H * W))
    out, idx, Ho, Wo = oracle.max_pool2d_fwd(X, C, H, W, 3, 3, 1, 1)   # overlapping windows
    dout = g.standard_normal(out.shape)
    dX = oracle.max_pool2d_bwd(dout, idx, C, H, W, 3, 3, 1, 1)
    assert abs(dX.sum() - dout.sum()) < 1e-12 * np.abs(dout).sum()
    chosen = np.zeros(dX.shape, bool)
    for n in range(N):
        chosen[n, idx[n]] = True
    assert not dX[~chosen].any()


def test_pool_finite_differences_distinct_values():
    g = rng(23)
    X = g.permutation(np.arange(2 * 36, dtype=np.float64)).reshape(1, -1) * 0.1
    out, idx, _, _ = oracle.max_pool2d_fwd(X, 2, 6, 6, 2, 2, 2, 0)
    R = g.standard_normal(out.shape)
    dX = oracle.max_pool2d_bwd(R, idx, 2, 6, 6, 2, 2, 2, 0)
    h = 1e-4
    for e in range(0, 72, 5):
        p, m = X.copy(), X.copy()
        p[0, e] += h
        m[0, e] -= h
        fd = (np.sum(oracle.max_pool2d_fwd(p, 2, 6, 6, 2, 2, 2, 0)[0] * R)
              - np.sum(oracle.max_pool2d_fwd(m, 2, 6, 6, 2, 2, 2, 0)[0] * R)) / (2 * h)
        assert abs(fd - dX[0, e]) < 1e-9


# ------------------------------------------------------------------------ bias_add_relu
def test_bias_add_relu_against_numpy_broadcast():
    g = rng(24)
    X = g.standard_normal((3, 4 * 10))
    b = g.standard_normal(4)
    got = oracle.bias_add_relu(X, b, 4, 10, relu=True)
    ref = torch.relu(torch.from_numpy(X.reshape(3, 4, 10)) + torch.from_numpy(b)[:, None])
    assert np.array_equal(got, ref.reshape(3, -1).numpy())
    assert np.array_equal(oracle.bias_add_relu(X, None, 4, 10, relu=False), X)
    assert np.array_equal(oracle.bias_add_relu(X, b, 4, 10, relu=False),
                          (X.reshape(3, 4, 10) + b[:, None]).reshape(3, -1))


# ----------------------------------------------------------------------------- affine
@pytest.mark.parametrize("relu", [False, True])
def test_affine_matches_torch(relu):
    g = rng(25)
    N, D, M = 5, 7, 4
    X, W, b = g.standard_normal((N, D)), g.standard_normal((D, M)), g.standard_normal(M)
    out = oracle.affine_fwd(X, W, b, relu=relu)
    x = torch.from_numpy(X).requires_grad_()
    w = torch.from_numpy(W).requires_grad_()
    bb = torch.from_numpy(b).requires_grad_()
    y = x @ w + bb
    if relu:
        y = torch.relu(y)
    assert _rel(out, y.detach().numpy()) < 1e-14
    dout = g.standard_normal((N, M))
    y.backward(torch.from_numpy(dout))
    dX, dW, db = oracle.affine_bwd(dout, X, W, out if relu else None)
    assert _rel(dX, x.grad.numpy()) < 1e-14
    assert _rel(dW, w.grad.numpy()) < 1e-14
    assert _rel(db, bb.grad.numpy()) < 1e-14
    _, dW2, db2 = oracle.affine_bwd(dout, X, W, out if relu else None, want_dX=False)
    assert np.array_equal(dW, dW2) and np.array_equal(db, db2)


def test_affine_matmul_and_finite_differences():
    g = rng(26)
    N, D, M = 4, 6, 3
    X, W, b = g.standard_normal((N, D)), g.standard_normal((D, M)), g.standard_normal(M)
    assert _rel(oracle.affine_fwd(X, W, b), X @ W + b) < 1e-14
    R = g.standard_normal((N, M))
    dX, dW, db = oracle.affine_bwd(R, X, W)
    h = 1e-6
    for (arr, grad) in ((X, dX), (W, dW), (b, db)):
        flat = arr.reshape(-1)
        for e in range(flat.size):
            old = flat[e]
            flat[e] = old + h
            lp = np.sum(oracle.affine_fwd(X, W, b) * R)
            flat[e] = old - h
            lm = np.sum(oracle.affine_fwd(X, W, b) * R)
            flat[e] = old
            assert abs((lp - lm) / (2 * h) - grad.reshape(-1)[e]) < 1e-7


# ---------------------------------------------------------------------------- softmax
def test_softmax_xent_matches_torch():
    g = rng(27)
    N, K = 6, 10
    S = g.standard_normal((N, K)) * 3
    lab = g.integers(0, K, N)
    Y = np.eye(K)[lab]
    loss, dS, P = oracle.softmax_xent(S, Y)
    s = torch.from_numpy(S).requires_grad_()
    tl = tF.cross_entropy(s, torch.from_numpy(lab))
    tl.backward()
    assert abs(loss - tl.item()) < 1e-14 * abs(tl.item())
    assert _rel(dS, s.grad.numpy()) < 1e-14
    assert _rel(P, torch.softmax(torch.from_numpy(S), 1).numpy()) < 1e-15


def test_softmax_closed_forms_and_invariants():
    K = 10
    loss, dS, P = oracle.softmax_xent(np.zeros((3, K)), np.eye(K)[[1, 4, 9]])
    assert abs(loss - math.log(K)) < 1e-15 and abs(loss - 2.302585092994046) < 1e-15
    g = rng(28)
    S = g.standard_normal((5, K)) * 4
    Y = np.eye(K)[g.integers(0, K, 5)]
    loss, dS, P = oracle.softmax_xent(S, Y)
    assert np.all(np.abs(P.sum(1) - 1) < 1e-15 * K)
    assert np.all(np.abs(dS.sum(1)) < 1e-16 * K)
    loss2, dS2, P2 = oracle.softmax_xent(S + 123.0, Y)   # shift invariance
    assert abs(loss2 - loss) < 1e-12 and _rel(dS2, dS) < 1e-12
    big = np.zeros((2, K))
    big[0, 3] = 1000.0
    big[1, 7] = 1000.0
    l3, d3, p3 = oracle.softmax_xent(big, np.eye(K)[[3, 7]])
    assert np.isfinite(l3) and abs(l3) < 1e-300 and np.isfinite(d3).all()


def test_softmax_fused_equals_paper_chain():
    # the unfused chain of Section 2's example: softmax forward, then the
    # cross-entropy backward, then the softmax backward
    g = rng(29)
    N, K = 8, 10
    S = g.standard_normal((N, K)) * 2
    Y = np.eye(K)[g.integers(0, K, N)]
    loss, dS, P = oracle.softmax_xent(S, Y)
    P2 = oracle.softmax_forward(S)
    assert _rel(P, P2) < 1e-15
    assert abs(oracle.xent_forward(P2, Y) - loss) < 1e-14 * abs(loss)
    dS2 = oracle.softmax_backward(oracle.xent_backward(P2, Y), P2)
    assert _rel(dS, dS2) < 1e-13


# -------------------------------------------------------------------------------- sgd
def test_sgd_momentum_two_step_closed_form():
    g = rng(30)
    th0 = g.standard_normal(11)
    g1, g2 = g.standard_normal(11), g.standard_normal(11)
    lr, mu = 0.01, 0.9
    th1, v1 = oracle.sgd_momentum_update(th0, g1, np.zeros(11), lr, mu)
    th2, v2 = oracle.sgd_momentum_update(th1, g2, v1, lr, mu)
    assert np.allclose(v1, -lr * g1, rtol=0, atol=1e-17)
    assert np.allclose(v2, mu * (-lr * g1) - lr * g2, rtol=1e-15, atol=1e-17)
    assert np.allclose(th2, th0 - lr * g1 + mu * (-lr * g1) - lr * g2, rtol=1e-14, atol=1e-15)
    th, v = oracle.sgd_momentum_update(th0, g1, np.zeros(11), 0.0, mu)
    assert np.array_equal(th, th0)
    # mu = 0 is the plain gradient step of Section 2's example
    th, _ = oracle.sgd_momentum_update(th0, g1, np.zeros(11), lr, 0.0)
    assert np.array_equal(th, th0 - lr * g1)


def test_sgd_matches_torch_optimizer():
    g = rng(31)
    th0 = g.standard_normal(9)
    grads = [g.standard_normal(9) for _ in range(3)]
    p = torch.nn.Parameter(torch.from_numpy(th0.copy()))
    opt = torch.optim.SGD([p], lr=0.01, momentum=0.9)
    th, v = th0, np.zeros(9)
    for gr in grads:
        p.grad = torch.from_numpy(gr.copy())
        opt.step()
        th, v = oracle.sgd_momentum_update(th, gr, v, 0.01, 0.9)
    assert _rel(th, p.detach().numpy()) < 1e-14


def test_count_nonzero():
    X = np.array([[0.0, -0.0, 1.0, 2.5], [np.inf, 0.0, -3.0, 0.0]])
    assert oracle.count_nonzero(X) == 4
