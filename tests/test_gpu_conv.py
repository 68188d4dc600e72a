"""GPU parity of the conv2d passes (through the C ABI) against the oracle.

Element-by-element on small shapes that span several tiles, ragged tails,
strides 1-3, pads 0-3 (including pad >= filter size), non-square filters, more
than 64 filters and channel counts that leave a ragged channel chunk; the
LeNet/ResNet-shaped workloads at full size where the oracle finishes in
seconds; and the 256-image ResNet-shaped workload at full size on sampled
outputs that the oracle computes one by one.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import TOL, assert_close, dev, host, rounded
from paper_1802_04647_amd import dmlnn
from paper_1802_04647_amd.inputs import SHAPES, ConvShape, conv_layer_inputs, random_conv_case

pytestmark = pytest.mark.gpu

CASES = [
    ConvShape(2, 3, 7, 6, 5, 3, 3, 1, 1),
    ConvShape(2, 5, 9, 9, 70, 3, 3, 1, 1),      # two filter tiles
    ConvShape(1, 9, 13, 11, 8, 5, 5, 2, 2),     # stride 2
    ConvShape(2, 37, 10, 10, 16, 3, 3, 1, 0),   # ragged channel chunk
    ConvShape(1, 2, 8, 5, 3, 3, 1, 3, 1),       # non-square filter, stride 3
    ConvShape(2, 4, 6, 6, 3, 1, 1, 1, 0),       # 1x1
    ConvShape(1, 3, 5, 6, 2, 3, 3, 1, 3),       # pad >= filter size
    ConvShape(3, 2, 1, 1, 4, 3, 3, 1, 1),       # 1x1 image
    ConvShape(2, 2, 9, 7, 3, 2, 3, 2, 0),       # uncovered border cells
    ConvShape(1, 6, 30, 30, 33, 3, 3, 1, 1),    # many pixel tiles per image
    ConvShape(1, 2, 5, 500, 3, 3, 3, 1, 1),     # rows too wide for LDS-DMA staging
    ConvShape(1, 3, 4, 700, 2, 3, 3, 2, 1),     # wide rows, stride 2
    # backward_filter row-ring kernel (whole k range per block)
    ConvShape(2, 64, 7, 12, 3, 3, 3, 1, 1),     # k range 576, image boundary inside a split
    ConvShape(2, 64, 6, 24, 5, 3, 3, 2, 1),     # stride 2: two new rows per tile
    ConvShape(1, 42, 12, 13, 4, 3, 3, 1, 0),    # k range 384, no padding
    ConvShape(3, 7, 10, 20, 3, 5, 5, 1, 2),     # 5x5 filter, five-slot ring
    ConvShape(1, 21, 9, 40, 2, 3, 3, 3, 1),     # stride equal to the filter height
    ConvShape(1, 21, 13, 48, 2, 3, 3, 4, 1),    # stride above the filter height
    ConvShape(2, 192, 4, 12, 2, 1, 1, 1, 0),    # 1x1 filter, one-slot ring
    ConvShape(1, 128, 3, 12, 2, 3, 3, 1, 1),    # two k ranges
    ConvShape(3, 23, 11, 18, 3, 5, 5, 2, 2),    # 5x5 stride 2: splits start mid-image, ring slots wrap
    ConvShape(2, 23, 60, 60, 80, 5, 5, 1, 2),   # row-mapped staging at its limits: 64-element
                                                # window rows, 60-pixel tiles; two filter tiles
    ConvShape(1, 64, 60, 60, 8, 3, 3, 1, 1),    # 60-wide rows over 64 channels: past the row
                                                # ring's staging, the tiled backward_filter
    # at most four output rows (forward F <= 4, backward_data C <= 4): direct kernel
    ConvShape(2, 3, 9, 11, 1, 7, 7, 1, 3),      # F = 1, 7x7 (any-width tap loop)
    ConvShape(1, 1, 16, 16, 6, 3, 3, 2, 1),     # backward_data C = 1, stride 2
    ConvShape(1, 4, 70, 3, 2, 5, 3, 1, 2),      # narrow tall image: tiles span many rows
    ConvShape(1, 2, 12, 12, 100, 3, 3, 1, 1),   # backward_data over 100 channels in chunks
    ConvShape(1, 2, 9, 9, 4, 8, 8, 1, 3),       # filter wider than 7: matrix-core path
    ConvShape(32, 5, 9, 9, 64, 3, 3, 1, 1),     # forward: filter-resident kernel (ragged chunk)
    ConvShape(16, 7, 10, 10, 130, 3, 3, 1, 1),  # forward: filter-resident, ragged filter group
]


def _args(s):
    return (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)


def _run_all(s, X, W, b, dout, mask, dt, relu=True):
    """GPU fwd, bwd_filter, bwd_data on identical inputs; returns host arrays."""
    a = _args(s)
    print(f"\n[gpu] conv {s} {dt} relu={relu}", flush=True)
    out, Ho, Wo = dmlnn.conv2d_forward(dev(X, dt), dev(W, dt), dev(b, dt), *a, relu=relu)
    dW, db = dmlnn.conv2d_backward_filter(dev(X, dt), dev(dout, dt), dev(mask, dt), *a, s.F)
    dX = dmlnn.conv2d_backward_data(dev(W, dt), dev(dout, dt), dev(mask, dt), *a)
    torch.cuda.synchronize()
    return host(out), host(dW), host(db), host(dX), (Ho, Wo)


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("s", CASES, ids=str)
def test_conv_parity_small(s, dt):
    X0, W0, b0, dout0 = random_conv_case(100, s, zero_frac=0.3)
    X, W, b, dout = (rounded(v, dt) for v in (X0, W0, b0, dout0))
    a = _args(s)
    for relu in (True, False):
        ref_out, Ho, Wo = oracle.conv2d_forward(X, W, b, *a, relu=relu)
        # the backward mask source is the oracle's forward output in the mode's type
        mask = rounded(ref_out, dt) if relu else None
        out, dW, db, dX, hw = _run_all(s, X, W, b, dout, mask, dt, relu=relu)
        assert hw == (Ho, Wo)
        ref_dW, ref_db = oracle.conv2d_backward_filter(X, dout, mask, *a, s.F)
        ref_dX = oracle.conv2d_backward_data(W, dout, mask, *a)
        assert_close(out, ref_out, dt, "forward")
        assert_close(dW, ref_dW, dt, "dW")
        assert_close(db, ref_db, dt, "db")
        assert_close(dX, ref_dX, dt, "dX")
        if relu:
            assert (out >= 0).all()


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("s", [ConvShape(64, 32, 14, 14, 64, 5, 5, 1, 2),
                               ConvShape(128, 20, 6, 6, 16, 3, 3, 1, 1),
                               ConvShape(64, 40, 8, 8, 24, 5, 5, 1, 2)], ids=str)
def test_backward_data_without_mask(s, dt):
    """backward_data with no relu mask (as in the LeNet step, whose pool backward
    folds the mask in): LeNet conv2 at batch 64, a ragged 32-row tile, and a
    ragged last channel chunk."""
    X0, W0, b0, dout0 = random_conv_case(101, s, zero_frac=0.3)
    W, dout = (rounded(v, dt) for v in (W0, dout0))
    a = _args(s)
    print(f"\n[gpu] backward_data {s} {dt}", flush=True)
    dX = dmlnn.conv2d_backward_data(dev(W, dt), dev(dout, dt), None, *a)
    torch.cuda.synchronize()
    assert_close(host(dX), oracle.conv2d_backward_data(W, dout, None, *a), dt, "dX")


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("name", ["conv_small", "lenet_conv1", "lenet_conv2"])
def test_conv_parity_workloads(name, dt):
    s = SHAPES[name]
    X0, W0, b0, dout0 = conv_layer_inputs(name)
    X, W, b = (rounded(v, dt) for v in (X0, W0, b0))
    a = _args(s)
    ref_out, _, _ = oracle.conv2d_forward(X, W, b, *a, relu=True)
    mask = rounded(ref_out, dt)
    if name == "lenet_conv2":
        # the conv's upstream gradient comes through the 2x2/2 max-pool backward
        _, idx, _, _ = oracle.max_pool2d_fwd(mask, s.F, s.Hout, s.Wout, 2, 2, 2, 0)
        dout = rounded(oracle.max_pool2d_bwd(rounded(dout0, dt), idx, s.F, s.Hout, s.Wout,
                                             2, 2, 2, 0), dt)
        assert np.mean(dout == 0) >= 0.75
    else:
        dout = rounded(dout0, dt)
    out, dW, db, dX, _ = _run_all(s, X, W, b, dout, mask, dt)
    ref_dW, ref_db = oracle.conv2d_backward_filter(X, dout, mask, *a, s.F)
    ref_dX = oracle.conv2d_backward_data(W, dout, mask, *a)
    assert_close(out, ref_out, dt, "forward")
    assert_close(dW, ref_dW, dt, "dW")
    assert_close(db, ref_db, dt, "db")
    assert_close(dX, ref_dX, dt, "dX")


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_conv_parity_resnet_two_images_elementwise(dt):
    # ResNet-shaped layer (64 -> 64, 56x56, 3x3 p1) on 2 images: every element.
    s = ConvShape(2, 64, 56, 56, 64, 3, 3, 1, 1)
    X0, W0, b0, dout0 = conv_layer_inputs("resnet_conv", N=2)
    X, W, b, dout = (rounded(v, dt) for v in (X0, W0, b0, dout0))
    a = _args(s)
    ref_out, _, _ = oracle.conv2d_forward(X, W, b, *a, relu=True)
    mask = rounded(ref_out, dt)
    out, dW, db, dX, _ = _run_all(s, X, W, b, dout, mask, dt)
    assert_close(out, ref_out, dt, "forward")
    ref_dW, ref_db = oracle.conv2d_backward_filter(X, dout, mask, *a, s.F)
    assert_close(dW, ref_dW, dt, "dW")
    assert_close(db, ref_db, dt, "db")
    assert_close(dX, oracle.conv2d_backward_data(W, dout, mask, *a), dt, "dX")


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_conv_parity_resnet_full_batch(dt):
    """All 256 images of the benchmark layer, in the launch configuration the
    benchmark times: every element of out, dW, db and dX against the oracle
    (whose full run takes about 20 s per dtype on 16 host cores).  The relu mask
    source of both backward passes is the oracle's forward output in the mode's
    type, so both sides read the same bytes."""
    s = SHAPES["resnet_conv"]
    X0, W0, b0, dout0 = conv_layer_inputs("resnet_conv")
    X, W, b, dout = (rounded(v, dt) for v in (X0, W0, b0, dout0))
    del X0, dout0
    a = _args(s)
    ref_out, _, _ = oracle.conv2d_forward(X, W, b, *a, relu=True)
    mask = rounded(ref_out, dt)
    out, dW, db, dX, _ = _run_all(s, X, W, b, dout, mask, dt)
    assert_close(out, ref_out, dt, "forward")
    del out, ref_out
    ref_dW, ref_db = oracle.conv2d_backward_filter(X, dout, mask, *a, s.F)
    assert_close(dW, ref_dW, dt, "dW")
    assert_close(db, ref_db, dt, "db")
    assert_close(dX, oracle.conv2d_backward_data(W, dout, mask, *a), dt, "dX")


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_adjoint_identities_resnet_full_batch(dt):
    """On the GPU, at the benchmark layer's full size (no bias, relu or mask):
    <conv(X, W), R> = <X, backward_data(W, R)> = <W, backward_filter(X, R)>,
    the identities that make the backward passes the adjoints of the forward
    pass.  Each side is a sum of about 10^10 products; they agree to a few
    units of the dtype's rounding."""
    s = SHAPES["resnet_conv"]
    X0, W0, _, R0 = conv_layer_inputs("resnet_conv")
    X, W, R = dev(X0, dt), dev(W0, dt), dev(R0, dt)
    del X0, R0
    a = _args(s)
    Y, _, _ = dmlnn.conv2d_forward(X, W, None, *a, relu=False)
    dX = dmlnn.conv2d_backward_data(W, R, None, *a)
    dW, _ = dmlnn.conv2d_backward_filter(X, R, None, *a, s.F, want_db=False)
    torch.cuda.synchronize()
    f64 = lambda t: t.to(torch.float64)  # noqa: E731
    lhs = float((f64(Y) * f64(R)).sum())
    via_data = float((f64(X) * f64(dX)).sum())
    via_filter = float((f64(W) * f64(dW)).sum())
    scale = float((f64(Y).abs() * f64(R).abs()).sum())
    tol = 1e-12 if dt == "f64" else 1e-5
    assert abs(lhs - via_data) <= tol * scale
    assert abs(lhs - via_filter) <= tol * scale


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_resnet_full_batch_is_deterministic(dt):
    """Two runs of every pass on the benchmark layer give bitwise equal results:
    the backward_filter split count is fixed by the plan and the occupancy HIP
    reports, and its partials are added in a fixed order (no float atomics)."""
    s = SHAPES["resnet_conv"]
    X0, W0, b0, dout0 = conv_layer_inputs("resnet_conv")
    X, W, b, dout = dev(X0, dt), dev(W0, dt), dev(b0, dt), dev(dout0, dt)
    del X0, dout0
    a = _args(s)
    runs = []
    for _ in range(2):
        out, _, _ = dmlnn.conv2d_forward(X, W, b, *a, relu=True)
        dW, db = dmlnn.conv2d_backward_filter(X, dout, out, *a, s.F)
        dX = dmlnn.conv2d_backward_data(W, dout, out, *a)
        torch.cuda.synchronize()
        runs.append((out, dW, db, dX))
    for u, v in zip(*runs):
        assert torch.equal(u, v)


def test_conv_parity_over_4gib_fp64():
    """A batch whose input, output and gradients each exceed 4 GiB (2700 images of
    the ResNet-shaped layer, fp64): the images past the 4 GiB mark take the same
    kernels, so every offset there must be computed in 64 bits.  Only the last
    four images are non-zero; sampled outputs of those images, and sampled
    filter-gradient entries (sums over all 2700 images), against the oracle."""
    s0 = SHAPES["resnet_conv"]
    N = 2700
    s = ConvShape(N, s0.C, s0.Hin, s0.Win, s0.F, s0.Hf, s0.Wf, s0.stride, s0.pad)
    a = _args(s)
    Ho, Wo = s.Hout, s.Wout
    assert N * s.C * s.Hin * s.Win * 8 > 2 ** 32
    g = np.random.Generator(np.random.PCG64(4096))
    tail = 4
    X = np.zeros((N, s.C * s.Hin * s.Win))
    X[-tail:] = np.maximum(g.standard_normal((tail, X.shape[1])), 0.0)
    W = g.standard_normal((s.F, s.C * s.Hf * s.Wf)) * np.sqrt(2.0 / (s.C * s.Hf * s.Wf))
    b = g.standard_normal(s.F) * 0.1
    dout = np.zeros((N, s.F * Ho * Wo))
    dout[-tail:] = g.standard_normal((tail, dout.shape[1]))
    mask = np.zeros_like(dout)
    mask[-tail:] = np.maximum(g.standard_normal((tail, dout.shape[1])), 0.0)
    print(f"\n[gpu] conv over 4 GiB: {s} f64", flush=True)
    Xd, Wd, bd = dev(X, "f64"), dev(W, "f64"), dev(b, "f64")
    outd, _, _ = dmlnn.conv2d_forward(Xd, Wd, bd, *a, relu=True)
    doutd, maskd = dev(dout, "f64"), dev(mask, "f64")
    dW, db = dmlnn.conv2d_backward_filter(Xd, doutd, maskd, *a, s.F)
    dXd = dmlnn.conv2d_backward_data(Wd, doutd, maskd, *a)
    torch.cuda.synchronize()
    tol = TOL["f64"]
    n_lo = N - tail
    idx = g.integers(0, [tail, s.F, Ho, Wo], size=(200, 4))
    idx[:, 0] += n_lo
    ref = np.array([max(oracle.conv2d_forward_pre_elem(X, W, b, *a, *e), 0.0) for e in idx])
    got = torch.stack([outd[e[0], (e[1] * Ho + e[2]) * Wo + e[3]] for e in idx]).cpu().numpy()
    assert np.max(np.abs(got - ref)) <= tol * np.max(np.abs(ref))
    # an image before the non-zero tail: relu(b) exactly
    assert torch.equal(outd[n_lo - 1].view(s.F, -1),
                       torch.relu(bd).view(s.F, 1).expand(s.F, Ho * Wo))
    idx = g.integers(0, [tail, s.C, s.Hin, s.Win], size=(200, 4))
    idx[:, 0] += n_lo
    refx = np.array([oracle.conv2d_backward_data_elem(W, dout, mask, s.C, s.Hin, s.Win, s.F,
                                                      s.Hf, s.Wf, s.stride, s.pad, *e)
                     for e in idx])
    gotx = torch.stack([dXd[e[0], (e[1] * s.Hin + e[2]) * s.Win + e[3]] for e in idx]).cpu().numpy()
    assert np.max(np.abs(gotx - refx)) <= tol * np.max(np.abs(refx))
    sel = g.integers(0, [s.F, s.C, s.Hf, s.Wf], size=(8, 4))
    refw = np.array([oracle.conv2d_backward_filter_elem(X, dout, mask, s.N, s.C, s.Hin, s.Win,
                                                        s.F, s.Hf, s.Wf, s.stride, s.pad, *e)
                     for e in sel])
    dWh = host(dW).reshape(s.F, s.C, s.Hf, s.Wf)
    gotw = dWh[sel[:, 0], sel[:, 1], sel[:, 2], sel[:, 3]]
    assert np.max(np.abs(gotw - refw)) <= tol * np.max(np.abs(refw))
    refb = np.array([oracle.conv2d_backward_bias_elem(dout, mask, s.N, s.F, Ho, Wo, f)
                     for f in range(s.F)])
    assert_close(host(db), refb, "f64", "db")


def test_zero_skip_matches_dense_bitwise():
    s = SHAPES["lenet_conv1"]
    X0, W0, b0, dout0 = conv_layer_inputs("lenet_conv1")
    # structured zeros: blank out whole rows so entire MFMA fragments are zero
    X0 = X0.reshape(s.N, 28, 28).copy()
    X0[:, :10, :] = 0.0
    X0 = X0.reshape(s.N, -1)
    a = _args(s)
    res = []
    prev = dmlnn.set_zero_skip(0)
    try:
        mask = None
        for mode in (0, 1):
            dmlnn.set_zero_skip(mode)
            out, _, _ = dmlnn.conv2d_forward(dev(X0, "f64"), dev(W0, "f64"), dev(b0, "f64"), *a)
            mask = out if mask is None else mask   # both modes' backward passes: one mask
            dW, db = dmlnn.conv2d_backward_filter(dev(X0, "f64"), dev(dout0, "f64"), mask, *a,
                                                  s.F)
            dX = dmlnn.conv2d_backward_data(dev(W0, "f64"), dev(dout0, "f64"), mask, *a)
            torch.cuda.synchronize()
            res.append([t + 0.0 for t in (out, dW, db, dX)])   # +0.0 folds -0 into +0
    finally:
        dmlnn.set_zero_skip(prev)
    # bitwise where both modes run one kernel form (where the dense mode's
    # kernel has no skip form the two agree to rounding only)
    kern = {p: [dmlnn.conv2d_plan(torch.float64, p, *s.args(), zero_skip=z)["kernel"]
                for z in (0, 1)]
            for p in ("forward", "backward_filter", "backward_data")}
    for (u, v), p in zip(zip(*res), ("forward", "backward_filter", "backward_filter",
                                      "backward_data")):
        if kern[p][0] == kern[p][1]:
            assert torch.equal(u, v), p
        else:
            assert_close(host(v), host(u), "f64", p)


def test_backward_filter_is_deterministic():
    s = SHAPES["lenet_conv2"]
    X0, W0, b0, dout0 = conv_layer_inputs("lenet_conv2")
    a = _args(s)
    X = dev(X0, "f32")
    out, _, _ = dmlnn.conv2d_forward(X, dev(W0, "f32"), dev(b0, "f32"), *a)
    g = torch.randn(out.shape, generator=torch.Generator().manual_seed(3)).to("cuda", torch.float32)
    r1 = dmlnn.conv2d_backward_filter(X, g, out, *a, s.F)
    r2 = dmlnn.conv2d_backward_filter(X, g, out, *a, s.F)
    torch.cuda.synchronize()
    assert torch.equal(r1[0], r2[0]) and torch.equal(r1[1], r2[1])


def test_identity_filter_is_exact():
    # 3x3 centre-tap identity with p=1: out = relu(X + b) bit-exactly (one non-zero product).
    C = 8
    X = np.random.Generator(np.random.PCG64(11)).standard_normal((3, C * 100))
    W = np.zeros((C, C * 9))
    for c in range(C):
        W[c, c * 9 + 4] = 1.0
    b = np.linspace(-0.5, 0.5, C)
    out, _, _ = dmlnn.conv2d_forward(dev(X, "f64"), dev(W, "f64"), dev(b, "f64"), C, 10, 10, 3, 3,
                                     1, 1)
    exp = np.maximum(X.reshape(3, C, 100) + b[None, :, None], 0.0).reshape(3, -1)
    assert np.array_equal(host(out), exp)


# backward_filter that also writes the masked gradient it stages, which
# backward_data then takes with no mask: the row-ring kernel (one and two k
# ranges), the tiled kernel (register and direct staging, several k ranges,
# rows cut into slices), both dtypes
EMIT_CASES = [
    ConvShape(2, 40, 12, 12, 48, 3, 3, 1, 1),
    ConvShape(1, 128, 3, 12, 2, 3, 3, 1, 1),
    ConvShape(3, 20, 9, 9, 70, 5, 5, 2, 2),
    ConvShape(4, 16, 16, 16, 40, 3, 3, 2, 1),
    ConvShape(1, 6, 5, 500, 8, 3, 3, 1, 1),
]


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("s", EMIT_CASES, ids=str)
def test_backward_filter_emits_masked_gradient(s, dt):
    X0, W0, b0, dout0 = random_conv_case(71, s, zero_frac=0.3)
    X, W, b, dout = (rounded(v, dt) for v in (X0, W0, b0, dout0))
    a = _args(s)
    print(f"\n[gpu] backward_filter emit {s} {dt}", flush=True)
    out, _, _ = dmlnn.conv2d_forward(dev(X, dt), dev(W, dt), dev(b, dt), *a, relu=True)
    Xd, dd = dev(X, dt), dev(dout, dt)
    dW0, db0 = dmlnn.conv2d_backward_filter(Xd, dd, out, *a, s.F)
    dX0 = dmlnn.conv2d_backward_data(dev(W, dt), dd, out, *a)
    g = torch.full_like(dd, float("nan"))
    dW1, db1 = dmlnn.conv2d_backward_filter(Xd, dd, out, *a, s.F, g_out=g)
    dX1 = dmlnn.conv2d_backward_data(dev(W, dt), g, None, *a)
    # in place: dout itself receives the masked gradient
    dd2 = dd.clone()
    dW2, db2 = dmlnn.conv2d_backward_filter(Xd, dd2, out, *a, s.F, g_out=dd2)
    torch.cuda.synchronize()
    want_g = torch.where(out > 0, dd, torch.zeros_like(dd))
    assert torch.equal(g, want_g) and torch.equal(dd2, want_g)
    for x0, x1 in ((dW0, dW1), (db0, db1), (dX0, dX1), (dW0, dW2), (db0, db2)):
        assert torch.equal(x0, x1)
    ref_dW, ref_db = oracle.conv2d_backward_filter(X, dout, host(out), *a, s.F)
    assert_close(host(dW1), ref_dW, dt, "dW")
    assert_close(host(db1), ref_db, dt, "db")


def test_images_of_2gib_register_path():
    """The largest image class: a per-image X of 2.1 GB (fp64), beyond the 32-bit
    byte offsets of the LDS-DMA kernels, takes the register-staged forward and
    a row-sliced backward_filter; checked at sampled outputs against the
    oracle's element functions (the full oracle would take hours)."""
    s = ConvShape(1, 4096, 256, 256, 16, 3, 3, 1, 1)
    assert s.C * s.Hin * s.Win * 8 >= 2 ** 31
    assert dmlnn.conv2d_plan(torch.float64, "forward", *s.args())["kernel"] == "igemm_reg"
    r = np.random.default_rng(2 ** 31)
    X = np.maximum(r.standard_normal((1, s.C * s.Hin * s.Win)), 0.0)
    W = r.standard_normal((s.F, s.K)) * np.sqrt(2.0 / s.K)
    b = r.standard_normal(s.F) * 0.1
    dout = r.standard_normal((1, s.F * s.Hout * s.Wout))
    a = _args(s)
    print(f"\n[gpu] 2 GiB image {s} f64", flush=True)
    Xd = torch.from_numpy(X).cuda()
    out, _, _ = dmlnn.conv2d_forward(Xd, dev(W, "f64"), dev(b, "f64"), *a, relu=True)
    dW, db = dmlnn.conv2d_backward_filter(Xd, dev(dout, "f64"), out, *a, s.F)
    dX = dmlnn.conv2d_backward_data(dev(W, "f64"), dev(dout, "f64"), out, *a)
    torch.cuda.synchronize()
    out_h, dW_h, db_h = host(out), host(dW), host(db)
    pick = np.random.default_rng(7)
    got, ref = [], []
    for _ in range(96):
        f, oh, ow = (int(pick.integers(v)) for v in (s.F, s.Hout, s.Wout))
        got.append(out_h[0, (f * s.Hout + oh) * s.Wout + ow])
        ref.append(max(oracle.conv2d_forward_pre_elem(X, W, b, *a, 0, f, oh, ow), 0.0))
    assert_close(np.array(got), np.array(ref), "f64", "out (sampled)")
    got, ref = [], []
    for _ in range(24):
        f, c, i, j = (int(pick.integers(v)) for v in (s.F, s.C, s.Hf, s.Wf))
        got.append(dW_h[f, (c * s.Hf + i) * s.Wf + j])
        ref.append(oracle.conv2d_backward_filter_elem(X, dout, out_h, 1, s.C, s.Hin, s.Win, s.F,
                                                      s.Hf, s.Wf, s.stride, s.pad, f, c, i, j))
    assert_close(np.array(got), np.array(ref), "f64", "dW (sampled)")
    ref_db = [oracle.conv2d_backward_bias_elem(dout, out_h, 1, s.F, s.Hout, s.Wout, f)
              for f in range(s.F)]
    assert_close(db_h, np.array(ref_db), "f64", "db")
    idx = [tuple(int(pick.integers(v)) for v in (s.C, s.Hin, s.Win)) for _ in range(96)]
    flat = torch.tensor([(c * s.Hin + h) * s.Win + w for c, h, w in idx], device="cuda")
    got = dX[0, flat].cpu().numpy()
    ref = [oracle.conv2d_backward_data_elem(W, dout, out_h, s.C, s.Hin, s.Win, s.F, s.Hf, s.Wf,
                                            s.stride, s.pad, 0, c, h, w) for c, h, w in idx]
    assert_close(got, np.array(ref), "f64", "dX (sampled)")
