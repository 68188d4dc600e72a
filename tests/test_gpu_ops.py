"""GPU parity of the ops around the conv layer (through the C ABI) against the
oracle: max-pool (argmax bit-exact), bias_add_relu, affine, softmax +
cross-entropy, SGD-momentum and count_nonzero, in fp64 and fp32."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import TORCH_DT, assert_close, dev, host, rounded
from paper_1802_04647_amd import dmlnn
from paper_1802_04647_amd.inputs import rng

pytestmark = pytest.mark.gpu

POOLS = [  # (N, C, H, W, Hf, Wf, s, p)
    (64, 64, 14, 14, 2, 2, 2, 0),     # LeNet pool2
    (64, 32, 28, 28, 2, 2, 2, 0),     # LeNet pool1
    (2, 3, 7, 9, 3, 3, 2, 1),
    (2, 2, 6, 5, 2, 3, 1, 1),         # overlapping windows
    (1, 2, 9, 9, 3, 2, 3, 0),
    (1, 2, 10, 11, 3, 3, 3, 0),       # trailing rows/columns no window covers
    (2, 3, 8, 8, 2, 2, 3, 0),         # gaps between windows
    (2, 3, 9, 9, 2, 2, 2, 0),         # odd width: scalar region stores, trailing row/col
    (2, 2, 7, 8, 2, 2, 2, 0),         # even width, odd height: vector stores, trailing row
    (1, 3, 4, 5, 1, 1, 1, 0),         # 1x1 windows at stride 1
]


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_max_pool_bwd_into_misaligned_output(dt):
    # an output one element past an aligned address: the 2-element vector
    # stores of 2x2/2 windows must not be used there
    N, C, H, W = 2, 3, 6, 8
    g = rng(41)
    X = rounded(g.standard_normal((N, C * H * W)), dt)
    _, ref_idx, Ho, Wo = oracle.max_pool2d_fwd(X, C, H, W, 2, 2, 2, 0)
    dout = rounded(g.standard_normal((N, C * Ho * Wo)), dt)
    buf = torch.full((N * C * H * W + 1,), 7.0, dtype=dev(dout, dt).dtype, device="cuda")
    dX = buf[1:]
    assert dX.data_ptr() % 16 != 0
    dmlnn.max_pool2d_bwd(dev(dout, dt), torch.from_numpy(ref_idx).cuda(), C, H, W, 2, 2, 2, 0,
                         dX=dX)
    torch.cuda.synchronize()
    ref = oracle.max_pool2d_bwd(dout, ref_idx, C, H, W, 2, 2, 2, 0)
    assert np.array_equal(host(dX).reshape(ref.shape), ref)
    assert float(buf[0]) == 7.0


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("cfg", POOLS, ids=str)
def test_max_pool_parity(cfg, dt):
    N, C, H, W, Hf, Wf, s, p = cfg
    print(f"\n[gpu] pool {cfg} {dt}", flush=True)
    g = rng(40)
    # relu-like input with many exact-zero ties, plus quantised values
    X = rounded(np.maximum(np.round(g.standard_normal((N, C * H * W)) * 4) / 4, 0.0), dt)
    ref_out, ref_idx, Ho, Wo = oracle.max_pool2d_fwd(X, C, H, W, Hf, Wf, s, p)
    out, idx, Ho2, Wo2 = dmlnn.max_pool2d_fwd(dev(X, dt), C, H, W, Hf, Wf, s, p)
    dout = rounded(g.standard_normal(ref_out.shape), dt)
    dX = dmlnn.max_pool2d_bwd(dev(dout, dt), idx, C, H, W, Hf, Wf, s, p)
    torch.cuda.synchronize()
    assert (Ho, Wo) == (Ho2, Wo2)
    assert np.array_equal(idx.cpu().numpy(), ref_idx)            # bit-exact argmax
    assert np.array_equal(host(out), ref_out)                     # a max is exact
    ref_dX = oracle.max_pool2d_bwd(dout, ref_idx, C, H, W, Hf, Wf, s, p)
    assert_close(host(dX), ref_dX, dt, "pool dX")


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_bias_add_relu_parity(dt):
    g = rng(41)
    N, C, HW = 5, 7, 33
    X = rounded(g.standard_normal((N, C * HW)), dt)
    b = rounded(g.standard_normal(C), dt)
    for relu in (True, False):
        for bias in (b, None):
            ref = oracle.bias_add_relu(X, bias, C, HW, relu=relu)
            got = dmlnn.bias_add_relu(dev(X, dt), dev(bias, dt), C, HW, relu=relu)
            assert_close(host(got), ref, dt, "bias_add_relu")
    Xd = dev(X, dt)                                                # in place
    dmlnn.bias_add_relu(Xd, dev(b, dt), C, HW, relu=True, out=Xd)
    assert_close(host(Xd), oracle.bias_add_relu(X, b, C, HW, relu=True), dt, "in place")


AFFINE = [(64, 3136, 512), (64, 512, 10), (5, 7, 3), (33, 70, 65), (1, 1, 1), (70, 1000, 33),
          (17, 4099, 20), (3, 130, 600), (48, 300, 3000), (130, 1000, 1100),
          (33, 700, 1300),   # dW with K = 33 over many tiles, ragged edges
          (1000, 101, 900)]  # forward with K = 101 (a partial 16-group) over many tiles


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("shape", AFFINE, ids=str)
def test_affine_parity(shape, dt):
    N, D, M = shape
    print(f"\n[gpu] affine {shape} {dt}", flush=True)
    g = rng(42)
    X = rounded(np.maximum(g.standard_normal((N, D)), 0.0), dt)
    W = rounded(g.standard_normal((D, M)) * np.sqrt(2.0 / D), dt)
    b = rounded(g.standard_normal(M) * 0.1, dt)
    dout = rounded(g.standard_normal((N, M)), dt)
    for relu in (True, False):
        ref_out = oracle.affine_fwd(X, W, b, relu=relu)
        out = dmlnn.affine_fwd(dev(X, dt), dev(W, dt), dev(b, dt), relu=relu)
        assert_close(host(out), ref_out, dt, "affine out")
        mask = rounded(ref_out, dt) if relu else None
        rdX, rdW, rdb = oracle.affine_bwd(dout, X, W, mask)
        dX, dW, db = dmlnn.affine_bwd(dev(dout, dt), dev(X, dt), dev(W, dt), dev(mask, dt))
        assert_close(host(dX), rdX, dt, "affine dX")
        assert_close(host(dW), rdW, dt, "affine dW")
        assert_close(host(db), rdb, dt, "affine db")
    _, dW2, _ = dmlnn.affine_bwd(dev(dout, dt), dev(X, dt), dev(W, dt), None, want_dX=False,
                                 want_db=False)
    assert_close(host(dW2), oracle.affine_bwd(dout, X, W, None)[1], dt, "affine dW only")
    # each output computed alone (separate calls) equals the joint call
    mask = rounded(oracle.affine_fwd(X, W, b, relu=True), dt)
    args = (dev(dout, dt), dev(X, dt), dev(W, dt), dev(mask, dt))
    dXj, dWj, dbj = dmlnn.affine_bwd(*args)
    dXs, _, _ = dmlnn.affine_bwd(*args, want_dW=False, want_db=False)
    _, _, dbs = dmlnn.affine_bwd(*args, want_dX=False, want_dW=False)
    assert dWj is not None and torch.equal(dXs, dXj) and torch.equal(dbs, dbj)


# products whose reduction splits over blocks: the batch-64 3136 -> 512 forward
# (32 x 32 tiles, seven splits), a dX from K = 3000 and a 17 x 20 forward from
# K = 4099 (16 x 16 tiles, nine splits, a partial last 16-group)
SPLIT = [(64, 3136, 512), (48, 300, 3000), (17, 4099, 20)]


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("shape", SPLIT, ids=str)
def test_affine_split_workspace(shape, dt):
    """The full workspace, a workspace for two splits and none all match the
    oracle; each is bitwise reproducible run to run (the split count, and so
    the order of the additions, depends only on the sizes and the workspace
    size)."""
    N, D, M = shape
    print(f"\n[gpu] affine split {shape} {dt}", flush=True)
    g = rng(45)
    X = rounded(np.maximum(g.standard_normal((N, D)), 0.0), dt)
    W = rounded(g.standard_normal((D, M)) * np.sqrt(2.0 / D), dt)
    b = rounded(g.standard_normal(M) * 0.1, dt)
    dout = rounded(g.standard_normal((N, M)), dt)
    tdt = torch.float64 if dt == "f64" else torch.float32
    full = dmlnn.affine_workspace_size(tdt, N, D, M)
    assert full > 0
    ref_out = oracle.affine_fwd(X, W, b, relu=True)
    mask = rounded(ref_out, dt)
    rdX, rdW, rdb = oracle.affine_bwd(dout, X, W, mask)
    esz = 8 if dt == "f64" else 4
    for nb in (full, 2 * max(N * M, N * D) * esz, 0):
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
        runs = []
        for _ in range(2):
            out = dmlnn.affine_fwd(dev(X, dt), dev(W, dt), dev(b, dt), relu=True, workspace=ws)
            dX, dW, db = dmlnn.affine_bwd(dev(dout, dt), dev(X, dt), dev(W, dt), dev(mask, dt),
                                          workspace=ws)
            runs.append((out, dX, dW, db))
        assert_close(host(runs[0][0]), ref_out, dt, f"affine out ws={nb}")
        assert_close(host(runs[0][1]), rdX, dt, f"affine dX ws={nb}")
        assert_close(host(runs[0][2]), rdW, dt, f"affine dW ws={nb}")
        assert_close(host(runs[0][3]), rdb, dt, f"affine db ws={nb}")
        for a, c in zip(*runs):
            assert torch.equal(a, c)


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("shape", [(64, 512, 10), (64, 3136, 512), (33, 70, 65), (5, 7, 3)],
                         ids=str)
def test_affine_relu_input(shape, dt):
    """relu_input folds the relu backward of the layer below into dX: dX times
    (X > 0), X a relu output with exact zeros; dW and db are unchanged."""
    N, D, M = shape
    print(f"\n[gpu] affine relu_input {shape} {dt}", flush=True)
    g = rng(46)
    X = rounded(np.maximum(g.standard_normal((N, D)), 0.0), dt)
    W = rounded(g.standard_normal((D, M)) * np.sqrt(2.0 / D), dt)
    dout = rounded(g.standard_normal((N, M)), dt)
    rdX, rdW, rdb = oracle.affine_bwd(dout, X, W, None)
    dX, dW, db = dmlnn.affine_bwd(dev(dout, dt), dev(X, dt), dev(W, dt), None, relu_input=True)
    assert_close(host(dX), rdX * (X > 0), dt, "affine dX relu_input")
    assert_close(host(dW), rdW, dt, "affine dW")
    assert_close(host(db), rdb, dt, "affine db")
    assert np.all(host(dX)[X == 0] == 0)


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_affine_misaligned_operands_bitwise(dt):
    # Operands whose rows are not 16-byte aligned take per-element loads instead
    # of vector loads; both read k in the same order, so the results are equal.
    N, D, M = 20, 96, 40
    g = rng(44)
    X = rounded(g.standard_normal((N, D)), dt)
    W = rounded(g.standard_normal((D, M)), dt)
    dout = rounded(g.standard_normal((N, M)), dt)
    tdt = torch.float64 if dt == "f64" else torch.float32

    def shifted(a):  # a copy of a that starts one element past an aligned allocation
        buf = torch.zeros(a.size + 1, dtype=tdt, device="cuda")
        v = buf[1:].view(a.shape)
        v.copy_(torch.from_numpy(a).to(tdt))
        return v

    zb = dev(np.zeros(M), dt)
    out_a = dmlnn.affine_fwd(dev(X, dt), dev(W, dt), zb, relu=False)
    out_m = dmlnn.affine_fwd(shifted(X), shifted(W), zb, relu=False)
    assert torch.equal(out_a, out_m)
    assert_close(host(out_a), oracle.affine_fwd(X, W, np.zeros(M), relu=False), dt, "affine out")
    dX_a, dW_a, _ = dmlnn.affine_bwd(dev(dout, dt), dev(X, dt), dev(W, dt), None)
    dX_m, dW_m, _ = dmlnn.affine_bwd(shifted(dout), shifted(X), shifted(W), None)
    assert torch.equal(dX_a, dX_m) and torch.equal(dW_a, dW_m)


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("NK", [(64, 10), (7, 3), (5, 130), (1, 1)], ids=str)
def test_softmax_xent_parity(NK, dt):
    N, K = NK
    g = rng(43)
    S = rounded(g.standard_normal((N, K)) * 3, dt)
    Y = np.eye(K)[g.integers(0, K, N)]
    rl, rdS, rP = oracle.softmax_xent(S, Y)
    loss, dS, P = dmlnn.softmax_xent(dev(S, dt), dev(Y, dt))
    torch.cuda.synchronize()
    assert abs(host(loss)[0] - rl) <= {"f64": 1e-10, "f32": 1e-4}[dt] * max(abs(rl), 1e-300)
    assert_close(host(dS), rdS, dt, "dscores")
    assert_close(host(P), rP, dt, "probs")


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("NK", [(100003, 10), (3001, 130), (5000, 1)], ids=str)
def test_softmax_xent_many_blocks(NK, dt):
    """Batches past one block: with the workspace the rows spread over many
    blocks and the loss shares are added in block order.  Against the oracle,
    bitwise the same on a second call, and dscores / probs bitwise equal to the
    one-block form (only the loss's summation order differs between forms)."""
    N, K = NK
    g = rng(45)
    S = rounded(g.standard_normal((N, K)) * 3, dt)
    Y = np.eye(K)[g.integers(0, K, N)]
    nb = dmlnn.softmax_xent_workspace_size(TORCH_DT[dt], N, K)
    assert nb > 8
    print(f"\n[gpu] softmax_xent N={N} K={K} {dt} workspace {nb} B", flush=True)
    Sd, Yd = dev(S, dt), dev(Y, dt)
    loss, dS, P = dmlnn.softmax_xent(Sd, Yd)
    loss2, dS2, P2 = dmlnn.softmax_xent(Sd, Yd)
    loss1, dS1, P1 = dmlnn.softmax_xent(Sd, Yd, workspace=torch.empty(0, dtype=torch.uint8,
                                                                         device=Sd.device))
    torch.cuda.synchronize()
    rl, rdS, rP = oracle.softmax_xent(S, Y)
    tol = {"f64": 1e-10, "f32": 1e-4}[dt]
    for got in (loss, loss1):
        assert abs(host(got)[0] - rl) <= tol * max(abs(rl), 1e-300)
    assert_close(host(dS), rdS, dt, "dscores")
    assert_close(host(P), rP, dt, "probs")
    assert torch.equal(loss, loss2) and torch.equal(dS, dS2) and torch.equal(P, P2)
    assert torch.equal(dS, dS1) and torch.equal(P, P1)


def test_softmax_uniform_scores_closed_form():
    K = 10
    loss, dS, P = dmlnn.softmax_xent(dev(np.zeros((3, K)), "f64"), dev(np.eye(K)[[1, 4, 9]], "f64"))
    assert abs(host(loss)[0] - np.log(10.0)) < 1e-14
    assert np.allclose(host(P), 0.1, rtol=0, atol=1e-16)


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_sgd_momentum_parity(dt):
    g = rng(44)
    n = 1663370
    th = rounded(g.standard_normal(n), dt)
    v = np.zeros(n)
    tth, tv = dev(th, dt), dev(v, dt)
    for step in range(3):
        gr = rounded(g.standard_normal(n), dt)
        th, v = oracle.sgd_momentum_update(th, gr, v, 0.01, 0.9)
        dmlnn.sgd_momentum_update(tth, dev(gr, dt), tv, 0.01, 0.9)
        th, v = rounded(th, dt), rounded(v, dt)     # the GPU keeps state in the mode's type
    assert_close(host(tth), th, dt, "theta")
    assert_close(host(tv), v, dt, "velocity")


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_count_nonzero_exact(dt):
    g = rng(45)
    for n in (1, 63, 64, 65, 1000003):
        X = rounded(np.where(g.random(n) < 0.2, g.random(n), 0.0), dt)
        X[:: max(1, n // 7)] = -0.0
        got = dmlnn.count_nonzero(dev(X, dt))
        assert int(got.item()) == oracle.count_nonzero(X)
