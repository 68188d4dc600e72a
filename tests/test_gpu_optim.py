"""GPU parity of the optimizer updates against the oracle: three consecutive
steps with fresh gradients on a ragged length (not a multiple of the block or
grid stride), fp64 and fp32.  The state buffers persist between steps on both
sides.  In fp32 mode the GPU computes in fp32 from the same fp32-rounded
inputs; the oracle computes in fp64."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_close, dev, host, rounded
from paper_1802_04647_amd import dmlnn

pytestmark = pytest.mark.gpu

N = 100_003


def _draws(k, dt):
    r = np.random.default_rng(4242 + k)
    th = rounded(r.standard_normal(N), dt)
    gs = [rounded(r.standard_normal(N), dt) for _ in range(3)]
    return th, gs


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_sgd(dt):
    th, gs = _draws(0, dt)
    t_d = dev(th, dt)
    ref = th
    for g in gs:
        dmlnn.sgd_update(t_d, dev(g, dt), 0.05)
        ref = oracle.sgd_update(ref, g, 0.05)
    torch.cuda.synchronize()
    assert_close(host(t_d), ref, dt, "theta")


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_sgd_nesterov(dt):
    th, gs = _draws(1, dt)
    t_d, v_d = dev(th, dt), dev(np.zeros(N), dt)
    ref, v = th, np.zeros(N)
    for g in gs:
        dmlnn.sgd_nesterov_update(t_d, dev(g, dt), v_d, 0.05, 0.9)
        ref, v = oracle.sgd_nesterov_update(ref, g, v, 0.05, 0.9)
    torch.cuda.synchronize()
    assert_close(host(t_d), ref, dt, "theta")
    assert_close(host(v_d), v, dt, "v")


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_adagrad(dt):
    th, gs = _draws(2, dt)
    t_d, c_d = dev(th, dt), dev(np.zeros(N), dt)
    ref, c = th, np.zeros(N)
    for g in gs:
        dmlnn.adagrad_update(t_d, dev(g, dt), c_d, 0.01, 1e-6)
        ref, c = oracle.adagrad_update(ref, g, c, 0.01, 1e-6)
    torch.cuda.synchronize()
    assert_close(host(t_d), ref, dt, "theta")
    assert_close(host(c_d), c, dt, "cache")


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_rmsprop(dt):
    th, gs = _draws(3, dt)
    t_d, c_d = dev(th, dt), dev(np.zeros(N), dt)
    ref, c = th, np.zeros(N)
    for g in gs:
        dmlnn.rmsprop_update(t_d, dev(g, dt), c_d, 0.01, 0.99, 1e-6)
        ref, c = oracle.rmsprop_update(ref, g, c, 0.01, 0.99, 1e-6)
    torch.cuda.synchronize()
    assert_close(host(t_d), ref, dt, "theta")
    assert_close(host(c_d), c, dt, "cache")


@pytest.mark.parametrize("dt", ["f64", "f32"])
def test_adam(dt):
    th, gs = _draws(4, dt)
    t_d, m_d, v_d = dev(th, dt), dev(np.zeros(N), dt), dev(np.zeros(N), dt)
    ref, m, v = th, np.zeros(N), np.zeros(N)
    for t, g in enumerate(gs, start=1):
        dmlnn.adam_update(t_d, dev(g, dt), m_d, v_d, 1e-3, 0.9, 0.999, 1e-8, t)
        ref, m, v = oracle.adam_update(ref, g, m, v, 1e-3, 0.9, 0.999, 1e-8, t)
    torch.cuda.synchronize()
    assert_close(host(t_d), ref, dt, "theta")
    assert_close(host(m_d), m, dt, "m")
    assert_close(host(v_d), v, dt, "v")
