"""The zero-skip path (the paper's sparse-input / dense-filter operator, Section 3
"Sparse Operations") against the oracle, on every kernel form that has a skip
instantiation.

With the zero-skip mode on, each conv2d pass must match the oracle within the
mode's tolerance and be bitwise equal to the dense path up to the sign of zero
results.  The plan query checks, for every case, which kernel form runs (LDS-DMA
implicit GEMM in its plain, two-way and four-way k-split forms, forward and
backward; the register-staged implicit GEMM; the fused pool epilogue; the
row-ring and the tiled backward_filter), so each skip instantiation is
executed.  Inputs carry structured zeros (zero bands and channels in X, dout and
the relu-mask source), so whole fragments are skipped, besides the workloads of
configs 1-3 with their own zeros.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_close, dev, host, rounded
from paper_1802_04647_amd import dmlnn
from paper_1802_04647_amd.inputs import (SHAPES, ConvShape, conv_layer_inputs,
                                         structured_zero_conv_case)

pytestmark = pytest.mark.gpu

TORCH = {"f64": torch.float64, "f32": torch.float32}

# Between them these take every kernel form with a skip instantiation, in both
# dtypes (checked on the CPU by tests/test_plan.py through the plan query).
CASES = [
    ConvShape(2, 40, 12, 12, 48, 3, 3, 1, 1),    # fwd/bwd plain (f64), row-ring wgrad
    ConvShape(2, 8, 28, 28, 12, 5, 5, 1, 2),     # fwd/bwd two-way k split
    ConvShape(2, 24, 10, 10, 20, 3, 3, 1, 1),    # fwd/bwd four-way k split, tiled wgrad
    ConvShape(4, 16, 16, 16, 40, 3, 3, 2, 1),    # stride 2: up-sampled backward source
    ConvShape(1, 6, 5, 500, 8, 3, 3, 1, 1),      # rows too wide for LDS-DMA (f64): register path
    ConvShape(40, 40, 56, 56, 48, 3, 3, 1, 1),   # 224-pixel tiles (NB = 7)
]


def _args(s):
    return (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)


def _plans(s, dt):
    return {p: dmlnn.conv2d_plan(TORCH[dt], p, *s.args(), zero_skip=1)
            for p in ("forward", "backward_filter", "backward_data")}


def _plan_key(s, dt, pname, zs):
    p = dmlnn.conv2d_plan(TORCH[dt], pname, *s.args(), zero_skip=zs)
    return (p["kernel"], p["k_split"], p["tile_pixels"], p["chunk"], p["splits"])


def _passes(s, X, W, b, dout, mask, dt):
    a = _args(s)
    out, _, _ = dmlnn.conv2d_forward(dev(X, dt), dev(W, dt), dev(b, dt), *a, relu=True)
    dW, db = dmlnn.conv2d_backward_filter(dev(X, dt), dev(dout, dt), dev(mask, dt), *a, s.F)
    dX = dmlnn.conv2d_backward_data(dev(W, dt), dev(dout, dt), dev(mask, dt), *a)
    torch.cuda.synchronize()
    return [t + 0.0 for t in (out, dW, db, dX)]   # + 0.0 folds -0 into +0


def _skip_on_vs_oracle(s, X, W, b, dout, mask, dt):
    a = _args(s)
    print(f"\n[gpu] zero skip {s} {dt}", flush=True)
    prev = dmlnn.set_zero_skip(1)
    try:
        on = _passes(s, X, W, b, dout, mask, dt)
        dmlnn.set_zero_skip(0)
        off = _passes(s, X, W, b, dout, mask, dt)
    finally:
        dmlnn.set_zero_skip(prev)
    # bitwise equal to the dense path of the same kernel form (the filter-resident
    # forward has no skip form: with the skip on, that pass takes the LDS-DMA
    # kernel, whose summation order differs; the oracle bound holds for both)
    same = {p: _plan_key(s, dt, p, 1) == _plan_key(s, dt, p, 0)
            for p in ("forward", "backward_filter", "backward_data")}
    for u, v, what, pname in zip(on, off, ("forward", "dW", "db", "dX"),
                                 ("forward", "backward_filter", "backward_filter",
                                  "backward_data")):
        if same[pname]:
            assert torch.equal(u, v), f"{what}: skip path differs from the dense path"
    ref_out, _, _ = oracle.conv2d_forward(X, W, b, *a, relu=True)
    ref_dW, ref_db = oracle.conv2d_backward_filter(X, dout, mask, *a, s.F)
    ref_dX = oracle.conv2d_backward_data(W, dout, mask, *a)
    for got, ref, what in zip(on, (ref_out, ref_dW, ref_db, ref_dX), ("forward", "dW", "db", "dX")):
        assert_close(host(got), ref, dt, what)


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("s", CASES, ids=str)
def test_structured_zeros_skip_matches_oracle(s, dt):
    X, W, b, dout, mask = (rounded(v, dt) for v in structured_zero_conv_case(61, s))
    _skip_on_vs_oracle(s, X, W, b, dout, mask, dt)


@pytest.mark.parametrize("dt", ["f64", "f32"])
@pytest.mark.parametrize("name", ["conv_small", "lenet_conv1", "lenet_conv2"])
def test_workloads_skip_matches_oracle(name, dt):
    """Configs 1-3 with the skip on.  LeNet conv2's backward passes take the
    pooled gradient (at least 75% zeros) as dout, as in the training step."""
    s = SHAPES[name]
    X0, W0, b0, dout0 = conv_layer_inputs(name)
    X, W, b = (rounded(v, dt) for v in (X0, W0, b0))
    a = _args(s)
    ref_out, _, _ = oracle.conv2d_forward(X, W, b, *a, relu=True)
    mask = rounded(ref_out, dt)
    if name == "lenet_conv2":
        _, idx, _, _ = oracle.max_pool2d_fwd(mask, s.F, s.Hout, s.Wout, 2, 2, 2, 0)
        dout = rounded(oracle.max_pool2d_bwd(rounded(dout0, dt), idx, s.F, s.Hout, s.Wout,
                                             2, 2, 2, 0), dt)
    else:
        dout = rounded(dout0, dt)
    _skip_on_vs_oracle(s, X, W, b, dout, mask, dt)


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_fused_pool_skip_matches_oracle(dt):
    """conv + bias + relu + 2x2/2 max-pool in one kernel with the skip on: the conv
    output against the oracle, and the pooled values and argmax exactly equal to
    the oracle's pooling of the call's own conv output (so a rounding difference
    in the convolution cannot move an argmax)."""
    s = ConvShape(8, 8, 28, 28, 24, 5, 5, 1, 2)
    X, W, b, _, _ = (rounded(v, dt) for v in structured_zero_conv_case(62, s))
    a = _args(s)
    assert dmlnn.conv2d_plan(TORCH[dt], "forward", *s.args(), zero_skip=1)["zero_skip"] == 1
    prev = dmlnn.set_zero_skip(1)
    try:
        out, pooled, argmax, _, _ = dmlnn.conv2d_forward_pool(
            dev(X, dt), dev(W, dt), dev(b, dt), *a, 2, 2, 2, 0, keep_out=True)
        torch.cuda.synchronize()
    finally:
        dmlnn.set_zero_skip(prev)
    ref, _, _ = oracle.conv2d_forward(X, W, b, *a, relu=True)
    assert_close(host(out), ref, dt, "conv out")
    rp, ri, _, _ = oracle.max_pool2d_fwd(host(out), s.F, s.Hout, s.Wout, 2, 2, 2, 0)
    assert np.array_equal(host(pooled), rp)
    assert np.array_equal(argmax.cpu().numpy(), ri)


def test_mode_chosen_from_count_nonzero():
    """The nnz-driven choice end to end: count the non-zeros of a 1%-dense
    LeNet-shaped input on the GPU, let the library's rule pick the mode from
    that count, and run backward_filter (which stages X) in it against the
    oracle; the forward (the LDS-DMA kernel here) takes the skip as well, and
    a layer whose dense forward has no skip form (the filter-resident kernel of
    LeNet conv2) stays dense."""
    from paper_1802_04647_amd.inputs import rng, sparse_uniform
    s = SHAPES["lenet_conv1"]
    _, W, b, dout = conv_layer_inputs("lenet_conv1")
    X = sparse_uniform(rng(71), rng(72), (s.N, s.C * s.Hin * s.Win), keep=0.01)
    Xd = dev(X, "f64")
    nnz = int(dmlnn.count_nonzero(Xd).item())
    assert nnz == np.count_nonzero(X)
    assert dmlnn.conv2d_zero_skip_choice(torch.float64, "forward", nnz, *s.args()) == 1
    assert dmlnn.conv2d_zero_skip_choice(torch.float64, "forward", 0,
                                         *SHAPES["lenet_conv2"].args()) == 0
    mode = dmlnn.conv2d_zero_skip_choice(torch.float64, "backward_filter", nnz, *s.args())
    assert mode == 1
    dense = dmlnn.conv2d_zero_skip_choice(torch.float64, "backward_filter", int(0.2 * X.size),
                                          *s.args())
    assert dense == 0
    prev = dmlnn.set_zero_skip(mode)
    try:
        dW, db = dmlnn.conv2d_backward_filter(Xd, dev(dout, "f64"), None, *_args(s), s.F)
        torch.cuda.synchronize()
    finally:
        dmlnn.set_zero_skip(prev)
    ref_dW, ref_db = oracle.conv2d_backward_filter(X, dout, None, *_args(s), s.F)
    assert_close(host(dW), ref_dW, "f64", "dW")
    assert_close(host(db), ref_db, "f64", "db")
