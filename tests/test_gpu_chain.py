"""Chained parity in fp64: the LeNet training step (1 and 3 steps, so momentum is
non-zero) and the conv -> relu -> pool -> pool-backward -> conv-backward chain of
the second LeNet conv layer, against the oracle composition.  Relu masks and
pool argmaxes flip only if a pre-activation lies within rounding distance of
zero, which fp64 makes astronomically unlikely; the tests report the counts."""
import numpy as np
import pytest
import torch

from oracle import lenet as lenet_oracle
import oracle
from gpu_util import assert_close, dev, host
from paper_1802_04647_amd import dmlnn
from paper_1802_04647_amd.inputs import SHAPES, conv_layer_inputs, lenet_train_inputs
from paper_1802_04647_amd.lenet import PARAM_ORDER, LeNetTrainer

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("fused", [True, False], ids=["pool-backward-fused", "unfused"])
@pytest.mark.parametrize("steps", [1, 3])
def test_lenet_training_steps(steps, fused):
    """fused: the conv backward passes read the pool gradients directly;
    unfused: the pool backward kernel stores the conv-output gradients first."""
    print(f"\n[gpu] lenet training {steps} step(s), fused pool backward {fused}", flush=True)
    X, Y, params = lenet_train_inputs()
    tr = LeNetTrainer(params, fused_pool_backward=fused)
    Xd, Yd = dev(X, "f64"), dev(Y, "f64")
    p, v = params, lenet_oracle.zero_velocities(params)
    for _ in range(steps):
        loss = tr.step(Xd, Yd)
        torch.cuda.synchronize()
        gl = host(loss)[0]
        ref_loss, p, v, g, a = lenet_oracle.train_step(X, Y, p, v)
        assert abs(gl - ref_loss) <= 1e-10 * abs(ref_loss)
    # the last step's activations (the trainer keeps only the pooled ones): values
    # close, relu masks and argmaxes exactly equal
    assert_close(host(tr.p1), a["p1"], "f64", "pool1")
    assert_close(host(tr.p2), a["p2"], "f64", "pool2")
    assert np.array_equal(host(tr.p1) > 0, a["p1"] > 0)
    assert np.array_equal(host(tr.p2) > 0, a["p2"] > 0)
    assert np.array_equal(tr.i1.cpu().numpy(), a["i1"])
    assert np.array_equal(tr.i2.cpu().numpy(), a["i2"])
    for k in PARAM_ORDER:
        assert_close(host(tr.g[k]).reshape(g[k].shape), g[k], "f64", "grad " + k)
        assert_close(host(tr.p[k]).reshape(p[k].shape), p[k], "f64", "param " + k)
        assert_close(host(tr.v[k]).reshape(v[k].shape), v[k], "f64", "velocity " + k)


def test_lenet_training_step_batch_100():
    """A batch past one softmax block (100 rows of 10 classes: two blocks and
    their loss shares in the trainer's workspace), and past the 64-image tiles
    of the conv and affine kernels, against the oracle step."""
    print("\n[gpu] lenet training step, batch 100", flush=True)
    X, Y, params = lenet_train_inputs(100)
    assert dmlnn.softmax_xent_workspace_size(torch.float64, 100, 10) == 2 * 8
    tr = LeNetTrainer(params, N=100)
    loss = tr.step(dev(X, "f64"), dev(Y, "f64"))
    torch.cuda.synchronize()
    ref_loss, p, v, g, a = lenet_oracle.train_step(X, Y, params,
                                                   lenet_oracle.zero_velocities(params))
    assert abs(host(loss)[0] - ref_loss) <= 1e-10 * abs(ref_loss)
    assert np.array_equal(tr.i2.cpu().numpy(), a["i2"])
    for k in PARAM_ORDER:
        assert_close(host(tr.g[k]).reshape(g[k].shape), g[k], "f64", "grad " + k)
        assert_close(host(tr.p[k]).reshape(p[k].shape), p[k], "f64", "param " + k)


def test_lenet_conv2_pool_chain():
    s = SHAPES["lenet_conv2"]
    X, W, b, dP = conv_layer_inputs("lenet_conv2")
    a = (s.C, s.Hin, s.Win, s.Hf, s.Wf, s.stride, s.pad)
    # oracle chain
    r_out, _, _ = oracle.conv2d_forward(X, W, b, *a)
    r_pool, r_idx, Hp, Wp = oracle.max_pool2d_fwd(r_out, s.F, s.Hout, s.Wout, 2, 2, 2, 0)
    r_dY = oracle.max_pool2d_bwd(dP, r_idx, s.F, s.Hout, s.Wout, 2, 2, 2, 0)
    r_dW, r_db = oracle.conv2d_backward_filter(X, r_dY, r_out, *a, s.F)
    r_dX = oracle.conv2d_backward_data(W, r_dY, r_out, *a)
    # GPU chain, each step fed by the previous GPU step
    out, _, _ = dmlnn.conv2d_forward(dev(X, "f64"), dev(W, "f64"), dev(b, "f64"), *a)
    pool, idx, _, _ = dmlnn.max_pool2d_fwd(out, s.F, s.Hout, s.Wout, 2, 2, 2, 0)
    dY = dmlnn.max_pool2d_bwd(dev(dP, "f64"), idx, s.F, s.Hout, s.Wout, 2, 2, 2, 0)
    dW, db = dmlnn.conv2d_backward_filter(dev(X, "f64"), dY, out, *a, s.F)
    dX = dmlnn.conv2d_backward_data(dev(W, "f64"), dY, out, *a)
    torch.cuda.synchronize()
    mask_flips = int(np.sum((host(out) > 0) != (r_out > 0)))
    argmax_flips = int(np.sum(idx.cpu().numpy() != r_idx))
    print(f"mask flips {mask_flips}, argmax flips {argmax_flips}")
    assert mask_flips == 0 and argmax_flips == 0
    assert_close(host(out), r_out, "f64", "out")
    assert_close(host(pool), r_pool, "f64", "pool")
    assert_close(host(dY), r_dY, "f64", "dY")
    assert_close(host(dW), r_dW, "f64", "dW")
    assert_close(host(db), r_db, "f64", "db")
    assert_close(host(dX), r_dX, "f64", "dX")
