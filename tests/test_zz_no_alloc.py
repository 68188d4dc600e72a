"""conv2d_backward_filter_noalloc, the backward_filter entry point for callers
that cannot allocate, against conv2d_backward_filter (the entry point with a
caller workspace): two calls in a row on one GPU, the second with a smaller
input, each bitwise equal to the workspace entry point's result (same plan, same
split order) and within the oracle bound on the small case.  The no-alloc calls
get preallocated outputs and must not allocate device memory."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_close, dev, host
from paper_1802_04647_amd import dmlnn
from paper_1802_04647_amd.inputs import SHAPES, ConvShape, conv_layer_inputs, random_conv_case

pytestmark = pytest.mark.gpu


def _args(s):
    return (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)


def _inputs(s, dt, seed):
    if s == SHAPES["resnet_conv"]:
        X, _, _, dout = conv_layer_inputs("resnet_conv")
        g = np.random.Generator(np.random.PCG64(seed))
        mask = np.maximum(g.standard_normal(dout.shape), 0.0)
    else:
        X, _, _, dout = random_conv_case(seed, s, zero_frac=0.3)
        mask = np.maximum(random_conv_case(seed + 1, s)[3], 0.0)
    return dev(X, dt), dev(dout, dt), dev(mask, dt)


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_noalloc_matches_workspace_entry_point(dt):
    # the benchmark layer (its workspace, 75.6 MB, fits the scratch), then a
    # smaller layer with fewer splits, so stale partials of the first call sit
    # in the scratch during the second
    shapes = [SHAPES["resnet_conv"], ConvShape(3, 20, 13, 11, 24, 5, 5, 1, 2)]
    for k, s in enumerate(shapes):
        print(f"\n[gpu] backward_filter_noalloc call {k + 1}: {s} {dt}", flush=True)
        X, dout, mask = _inputs(s, dt, 90 + k)
        a = _args(s)
        ref_dW, ref_db = dmlnn.conv2d_backward_filter(X, dout, mask, *a, s.F)
        dW = torch.empty_like(ref_dW)
        db = torch.empty_like(ref_db)
        torch.cuda.synchronize()
        before = torch.cuda.memory_allocated()
        dmlnn.conv2d_backward_filter_noalloc(X, dout, mask, *a, s.F, dW, db)
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() == before
        assert torch.equal(dW, ref_dW) and torch.equal(db, ref_db)
        if k == 1:   # the small case against the oracle as well
            Xh, douth, maskh = host(X), host(dout), host(mask)
            rW, rb = oracle.conv2d_backward_filter(Xh, douth, maskh, *a, s.F)
            assert_close(host(dW), rW, dt, "dW")
            assert_close(host(db), rb, dt, "db")


def test_noalloc_without_bias_gradient():
    s = ConvShape(2, 7, 9, 9, 5, 3, 3, 2, 1)
    X, dout, mask = _inputs(s, "f64", 95)
    ref_dW, _ = dmlnn.conv2d_backward_filter(X, dout, mask, *_args(s), s.F, want_db=False)
    dW = torch.empty_like(ref_dW)
    dmlnn.conv2d_backward_filter_noalloc(X, dout, mask, *_args(s), s.F, dW, None)
    torch.cuda.synchronize()
    assert torch.equal(dW, ref_dW)
