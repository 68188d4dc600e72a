"""Pins for the oracle's conv2d forward/backward (CPU only).

None of these re-types the oracle's formula: the references are torch's CPU
conv2d and autograd (a library routine), numpy matmul in the cases where the
convolution degenerates into a GEMM, bit-exact structural identities (delta,
identity and shifted filters, stride subsampling, explicit zero padding), the
adjoint (dot-product) identities that tie the two backward passes to the
forward pass, and central finite differences.
"""
import itertools

import numpy as np
import pytest
import torch
import torch.nn.functional as tF

import oracle
from paper_1802_04647_amd.inputs import ConvShape, random_conv_case, rng

pytestmark = pytest.mark.filterwarnings("ignore::UserWarning")


def _torch_conv(X, W, b, s: ConvShape, relu):
    x = torch.from_numpy(X.reshape(s.N, s.C, s.Hin, s.Win))
    w = torch.from_numpy(W.reshape(s.F, s.C, s.Hf, s.Wf))
    y = tF.conv2d(x, w, torch.from_numpy(b), stride=s.stride, padding=s.pad)
    if relu:
        y = torch.relu(y)
    return y.reshape(s.N, -1).numpy()


def _rel(a, b):
    den = np.max(np.abs(b))
    return np.max(np.abs(a - b)) / (den if den > 0 else 1.0)


SHAPES = [
    ConvShape(2, 3, 7, 6, 3, 3, 3, 1, 1),
    ConvShape(2, 2, 7, 7, 3, 3, 2, 2, 0),
    ConvShape(1, 3, 9, 8, 2, 3, 3, 3, 2),
    ConvShape(2, 1, 5, 7, 2, 2, 3, 2, 1),
    ConvShape(1, 2, 6, 6, 3, 1, 1, 1, 0),
    ConvShape(2, 3, 7, 7, 2, 5, 5, 1, 2),
    ConvShape(1, 2, 8, 5, 2, 3, 1, 3, 1),
]


@pytest.mark.parametrize("s", SHAPES, ids=str)
def test_forward_matches_torch_conv2d(s):
    X, W, b, _ = random_conv_case(1, s, zero_frac=0.3)
    for relu in (False, True):
        got, Ho, Wo = oracle.conv2d_forward(X, W, b, s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride,
                                            s.pad, relu=relu)
        assert (Ho, Wo) == (s.Hout, s.Wout)
        ref = _torch_conv(X, W, b, s, relu)
        assert _rel(got, ref) < 1e-14


@pytest.mark.parametrize("s", SHAPES, ids=str)
def test_backward_matches_torch_autograd(s):
    X, W, b, dout = random_conv_case(2, s, zero_frac=0.3)
    for relu in (False, True):
        out, _, _ = oracle.conv2d_forward(X, W, b, s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride,
                                          s.pad, relu=relu)
        mask_src = out if relu else None
        dW, db = oracle.conv2d_backward_filter(X, dout, mask_src, s.C, s.Hin, s.Win, s.Hf, s.Wf,
                                               s.stride, s.pad, s.F)
        dX = oracle.conv2d_backward_data(W, dout, mask_src, s.C, s.Hin, s.Win, s.Hf, s.Wf,
                                         s.stride, s.pad)
        x = torch.from_numpy(X.reshape(s.N, s.C, s.Hin, s.Win)).requires_grad_()
        w = torch.from_numpy(W.reshape(s.F, s.C, s.Hf, s.Wf)).requires_grad_()
        bb = torch.from_numpy(b).requires_grad_()
        y = tF.conv2d(x, w, bb, stride=s.stride, padding=s.pad)
        if relu:
            y = torch.relu(y)
        y.backward(torch.from_numpy(dout.reshape(y.shape)))
        assert _rel(dW, w.grad.reshape(s.F, -1).numpy()) < 1e-13
        assert _rel(db, bb.grad.numpy()) < 1e-13
        assert _rel(dX, x.grad.reshape(s.N, -1).numpy()) < 1e-13


def test_delta_filter_shifts_bit_exact():
    # A single 1 at tap (0,0) of a 3x3 filter with pad 1: out[h,w] = x[h-1,w-1], zero-filled.
    s = ConvShape(2, 1, 6, 5, 1, 3, 3, 1, 1)
    X = rng(3).standard_normal((2, 30))
    W = np.zeros((1, 9))
    W[0, 0] = 1.0
    out, _, _ = oracle.conv2d_forward(X, W, np.zeros(1), 1, 6, 5, 3, 3, 1, 1, relu=False)
    img = X.reshape(2, 6, 5)
    exp = np.zeros_like(img)
    exp[:, 1:, 1:] = img[:, :-1, :-1]
    assert np.array_equal(out.reshape(2, 6, 5), exp)


def test_delta_filter_each_tap():
    s = ConvShape(1, 2, 5, 6, 2, 3, 3, 1, 1)
    X = rng(4).standard_normal((1, 60))
    img = np.pad(X.reshape(2, 5, 6), ((0, 0), (1, 1), (1, 1)))
    for c, i, j in itertools.product(range(2), range(3), range(3)):
        W = np.zeros((2, 18))
        W[1, c * 9 + i * 3 + j] = 1.0
        out, _, _ = oracle.conv2d_forward(X, W, None, 2, 5, 6, 3, 3, 1, 1, relu=False)
        o = out.reshape(2, 5, 6)
        assert np.array_equal(o[1], img[c, i:i + 5, j:j + 6])
        assert not o[0].any()


def test_identity_filters_bit_exact():
    C = 3
    X = rng(5).standard_normal((2, C * 36))
    b = np.array([0.5, -0.25, 0.0])
    exp = np.maximum(X.reshape(2, C, 36) + b[None, :, None], 0.0).reshape(2, -1)
    W1 = np.eye(C)                                   # 1x1 identity, p=0
    o1, _, _ = oracle.conv2d_forward(X, W1, b, C, 6, 6, 1, 1, 1, 0, relu=True)
    assert np.array_equal(o1, exp)
    W3 = np.zeros((C, C * 9))                        # 3x3 centre tap, p=1
    for c in range(C):
        W3[c, c * 9 + 4] = 1.0
    o3, _, _ = oracle.conv2d_forward(X, W3, b, C, 6, 6, 3, 3, 1, 1, relu=True)
    assert np.array_equal(o3, exp)


def test_padding_equals_explicit_zero_pad_bit_exact():
    s = ConvShape(2, 2, 5, 7, 3, 3, 3, 1, 2)
    X, W, b, _ = random_conv_case(6, s)
    o, Ho, Wo = oracle.conv2d_forward(X, W, b, 2, 5, 7, 3, 3, 1, 2, relu=False)
    Xp = np.pad(X.reshape(2, 2, 5, 7), ((0, 0), (0, 0), (2, 2), (2, 2))).reshape(2, -1)
    o2, Ho2, Wo2 = oracle.conv2d_forward(Xp, W, b, 2, 9, 11, 3, 3, 1, 0, relu=False)
    assert (Ho, Wo) == (Ho2, Wo2)
    assert np.array_equal(o, o2)


@pytest.mark.parametrize("stride", [2, 3])
def test_stride_is_subsampling_bit_exact(stride):
    X, W, b, _ = random_conv_case(7, ConvShape(2, 2, 9, 8, 2, 3, 3, 1, 1))
    o1, H1, W1_ = oracle.conv2d_forward(X, W, b, 2, 9, 8, 3, 3, 1, 1, relu=True)
    os_, Hs, Ws = oracle.conv2d_forward(X, W, b, 2, 9, 8, 3, 3, stride, 1, relu=True)
    full = o1.reshape(2, 2, H1, W1_)[:, :, ::stride, ::stride]
    assert full.shape[2:] == (Hs, Ws)
    assert np.array_equal(os_.reshape(full.shape), full)


def test_full_window_is_a_matmul():
    # Hf = Hin, Wf = Win, p = 0: pre = X W^T + b (textbook GEMM).
    N, C, H, Wd, F = 3, 2, 4, 5, 4
    g = rng(8)
    X = g.standard_normal((N, C * H * Wd))
    W = g.standard_normal((F, C * H * Wd))
    b = g.standard_normal(F)
    o, Ho, Wo = oracle.conv2d_forward(X, W, b, C, H, Wd, H, Wd, 1, 0, relu=False)
    assert (Ho, Wo) == (1, 1)
    assert _rel(o, X @ W.T + b) < 1e-14


def test_one_by_one_is_a_per_image_matmul():
    N, C, H, Wd, F = 2, 3, 4, 6, 5
    g = rng(9)
    X = g.standard_normal((N, C * H * Wd))
    W = g.standard_normal((F, C))
    o, _, _ = oracle.conv2d_forward(X, W, None, C, H, Wd, 1, 1, 1, 0, relu=False)
    for n in range(N):
        assert _rel(o[n].reshape(F, -1), W @ X[n].reshape(C, -1)) < 1e-14


@pytest.mark.parametrize("s", SHAPES, ids=str)
def test_adjoint_identities(s):
    # <conv(X,W), R> = <X, bwd_data(W,R)> = <W, bwd_filter(X,R)>, relu off, b = 0.
    X, W, _, R = random_conv_case(10, s)
    o, _, _ = oracle.conv2d_forward(X, W, None, s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad,
                                    relu=False)
    dX = oracle.conv2d_backward_data(W, R, None, s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)
    dW, db = oracle.conv2d_backward_filter(X, R, None, s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride,
                                           s.pad, s.F)
    lhs = np.sum(o * R)
    scale = np.sum(np.abs(o * R))
    assert abs(np.sum(X * dX) - lhs) <= 1e-13 * scale
    assert abs(np.sum(W * dW) - lhs) <= 1e-13 * scale
    # db is the derivative of <conv + b, R> with respect to b: per-filter sums of R.
    assert np.allclose(db, R.reshape(s.N, s.F, -1).sum(axis=(0, 2)), rtol=1e-13, atol=1e-13)


def test_uncovered_border_gets_zero_gradient():
    # stride 3, 8 wide, 2-wide filter, p=0: windows start at 0, 3, 6, so 2 and 5 are never covered.
    s = ConvShape(1, 1, 8, 8, 1, 2, 2, 3, 0)
    X, W, _, R = random_conv_case(11, s)
    dX = oracle.conv2d_backward_data(W, R, None, 1, 8, 8, 2, 2, 3, 0).reshape(8, 8)
    for k in (2, 5):
        assert not dX[k, :].any() and not dX[:, k].any()
    for k in (0, 1, 3, 4, 6, 7):
        assert dX[k, 0] != 0.0 and dX[0, k] != 0.0


def test_finite_differences_away_from_kink():
    # b = +10 keeps every pre-activation positive, so relu is the identity locally.
    s = ConvShape(1, 2, 5, 5, 2, 3, 3, 2, 1)
    X, W, _, R = random_conv_case(12, s, bias=10.0)
    b = np.full(s.F, 10.0)
    args = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)

    def L(Xv, Wv, bv):
        o, _, _ = oracle.conv2d_forward(Xv, Wv, bv, *args, relu=True)
        return np.sum(o * R)

    out, _, _ = oracle.conv2d_forward(X, W, b, *args, relu=True)
    assert (out > 0).all()
    dW, db = oracle.conv2d_backward_filter(X, R, out, *args, s.F)
    dX = oracle.conv2d_backward_data(W, R, out, *args)
    h = 1e-6
    for arr, grad, which in ((X, dX, 0), (W, dW, 1), (b, db, 2)):
        flat = arr.reshape(-1)
        for e in range(0, flat.size, max(1, flat.size // 12)):
            p, m = flat.copy(), flat.copy()
            p[e] += h
            m[e] -= h
            vp = [X, W, b]
            vm = [X, W, b]
            vp[which] = p.reshape(arr.shape)
            vm[which] = m.reshape(arr.shape)
            fd = (L(*vp) - L(*vm)) / (2 * h)
            assert abs(fd - grad.reshape(-1)[e]) <= 1e-6 * max(1.0, abs(fd))


def test_relu_mask_zeroes_gradient_where_output_is_zero():
    s = ConvShape(2, 2, 6, 6, 3, 3, 3, 1, 1)
    X, W, b, R = random_conv_case(13, s)
    out, _, _ = oracle.conv2d_forward(X, W, b, *(s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad))
    assert (out == 0).any() and (out > 0).any()
    Rm = np.where(out > 0, R, 0.0)
    a = oracle.conv2d_backward_filter(X, R, out, s.C, s.Hin, s.Win, s.Hf, s.Wf, 1, 1, s.F)
    bref = oracle.conv2d_backward_filter(X, Rm, None, s.C, s.Hin, s.Win, s.Hf, s.Wf, 1, 1, s.F)
    assert np.array_equal(a[0], bref[0]) and np.array_equal(a[1], bref[1])
    c = oracle.conv2d_backward_data(W, R, out, s.C, s.Hin, s.Win, s.Hf, s.Wf, 1, 1)
    d = oracle.conv2d_backward_data(W, Rm, None, s.C, s.Hin, s.Win, s.Hf, s.Wf, 1, 1)
    assert np.array_equal(c, d)


def test_element_functions_agree_with_full_tensors():
    s = ConvShape(2, 3, 7, 6, 4, 3, 3, 2, 1)
    X, W, b, R = random_conv_case(14, s)
    a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)
    out, Ho, Wo = oracle.conv2d_forward(X, W, b, *a, relu=False)
    dW, db = oracle.conv2d_backward_filter(X, R, out, *a, s.F)
    dX = oracle.conv2d_backward_data(W, R, out, *a)
    X, W, b, R = (np.ascontiguousarray(v) for v in (X, W, b, R))
    o4 = out.reshape(s.N, s.F, Ho, Wo)
    assert oracle.conv2d_forward_pre_elem(X, W, b, *a, 1, 2, 1, 2) == o4[1, 2, 1, 2]
    assert oracle.conv2d_backward_filter_elem(X, R, out, s.N, s.C, s.Hin, s.Win, s.F, s.Hf,
                                              s.Wf, s.stride, s.pad, 3, 1, 2, 0) == \
        dW.reshape(s.F, s.C, 3, 3)[3, 1, 2, 0]
    assert oracle.conv2d_backward_bias_elem(R, out, s.N, s.F, Ho, Wo, 2) == db[2]
    assert oracle.conv2d_backward_data_elem(W, R, out, s.C, s.Hin, s.Win, s.F, s.Hf, s.Wf,
                                            s.stride, s.pad, 1, 2, 4, 5) == \
        dX.reshape(s.N, s.C, 7, 6)[1, 2, 4, 5]


def test_out_dim():
    assert oracle.out_dim(28, 5, 1, 2) == 28
    assert oracle.out_dim(56, 3, 1, 1) == 56
    assert oracle.out_dim(7, 3, 2, 0) == 3
    assert oracle.out_dim(2, 3, 1, 0) <= 0
    assert oracle.out_dim(8, 2, 3, 0) == 3


def test_results_do_not_depend_on_thread_count():
    s = ConvShape(2, 3, 9, 9, 4, 3, 3, 1, 1)
    X, W, b, R = random_conv_case(15, s)
    a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)
    n0 = oracle.get_threads()
    try:
        res = []
        for t in (1, 3):
            oracle.set_threads(t)
            out, _, _ = oracle.conv2d_forward(X, W, b, *a)
            res.append((out, *oracle.conv2d_backward_filter(X, R, out, *a, s.F),
                        oracle.conv2d_backward_data(W, R, out, *a)))
    finally:
        oracle.set_threads(n0)
    for u, v in zip(*res):
        assert np.array_equal(u, v)
