"""Pins for the oracle's optimizer updates (Section 2 names Adagrad, Adam,
RMSprop, SGD and SGD with Nesterov momentum; the readings are the published
methods' usual statements).  Each pin is a fact fixed by the mathematics, not a
retyped update: exact small cases, special cases that reduce to another
optimizer, closed forms for a constant gradient over many steps, and Adam's
equivalence with its bias-corrected statement."""
import numpy as np

import oracle


def _rng(k):
    return np.random.default_rng(1802 + k)


def test_sgd_exact():
    th = np.array([1.0, 2.0, 3.0])
    g = np.array([4.0, -8.0, 0.5])
    assert np.array_equal(oracle.sgd_update(th, g, 0.25), np.array([0.0, 4.0, 2.875]))


def test_nesterov_without_momentum_is_sgd():
    r = _rng(1)
    th, g = r.standard_normal(1000), r.standard_normal(1000)
    t1, v1 = oracle.sgd_nesterov_update(th, g, np.zeros(1000), 0.01, 0.0)
    assert np.array_equal(t1, oracle.sgd_update(th, g, 0.01))
    assert np.array_equal(v1, -0.01 * g)


def test_nesterov_constant_gradient_closed_form():
    # v_t = -lr g (1 - mu^t)/(1 - mu); theta_T = theta_0 + sum_t v_t + mu v_T
    lr, mu, T = 0.05, 0.9, 25
    g = np.array([1.5, -0.25, 3.0])
    th, v = np.array([0.5, -1.0, 2.0]), np.zeros(3)
    th0 = th.copy()
    for _ in range(T):
        th, v = oracle.sgd_nesterov_update(th, g, v, lr, mu)
    vt = lambda t: -lr * g * (1 - mu ** t) / (1 - mu)  # noqa: E731
    expect = th0 + sum(vt(t) for t in range(1, T + 1)) + mu * vt(T)
    np.testing.assert_allclose(th, expect, rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(v, vt(T), rtol=1e-13)


def test_adagrad_constant_gradient_closed_form():
    # cache_t = t g^2, so theta_T = theta_0 - lr g sum_t 1/(sqrt(t)|g| + eps)
    lr, eps, T = 0.1, 1e-6, 40
    g = np.array([2.0, -0.5, 1e-3])
    th, c = np.array([1.0, 1.0, 1.0]), np.zeros(3)
    for _ in range(T):
        th, c = oracle.adagrad_update(th, g, c, lr, eps)
    s = sum(1.0 / (np.sqrt(t) * np.abs(g) + eps) for t in range(1, T + 1))
    np.testing.assert_allclose(th, 1.0 - lr * g * s, rtol=1e-13)
    np.testing.assert_allclose(c, T * g * g, rtol=1e-14)


def test_rmsprop_constant_gradient_closed_form():
    # cache_t = g^2 (1 - rho^t)
    lr, rho, eps, T = 0.01, 0.9, 1e-8, 30
    g = np.array([0.3, -4.0])
    th, c = np.array([0.0, 0.0]), np.zeros(2)
    for _ in range(T):
        th, c = oracle.rmsprop_update(th, g, c, lr, rho, eps)
    s = sum(1.0 / (np.abs(g) * np.sqrt(1 - rho ** t) + eps) for t in range(1, T + 1))
    np.testing.assert_allclose(th, -lr * g * s, rtol=1e-12)
    np.testing.assert_allclose(c, g * g * (1 - rho ** T), rtol=1e-13)


def test_rmsprop_without_decay_is_normalised_sgd():
    r = _rng(2)
    th, g, c = r.standard_normal(500), r.standard_normal(500), r.random(500)
    t1, c1 = oracle.rmsprop_update(th, g, c, 0.01, 0.0, 1e-8)
    np.testing.assert_allclose(t1, th - 0.01 * g / (np.abs(g) + 1e-8), rtol=1e-14)
    np.testing.assert_allclose(c1, g * g, rtol=1e-15)


def test_adam_constant_gradient_moves_lr_per_step():
    # with eps = 0 and a constant gradient, m_t = g (1 - b1^t) and v_t = g^2 (1 - b2^t),
    # so the folded bias corrections cancel: every step moves theta by lr against sign(g)
    lr, T = 0.003, 50
    g = np.array([5.0, -0.01, 123.0])
    th, m, v = np.zeros(3), np.zeros(3), np.zeros(3)
    for t in range(1, T + 1):
        th, m, v = oracle.adam_update(th, g, m, v, lr, 0.9, 0.999, 0.0, t)
    np.testing.assert_allclose(th, -T * lr * np.sign(g), rtol=1e-12)


def test_adam_matches_bias_corrected_statement():
    # Kingma and Ba's Algorithm 1: theta -= lr mhat / (sqrt(vhat) + eps'), with
    # mhat = m/(1-b1^t), vhat = v/(1-b2^t); it equals the folded step size form when
    # eps' = eps / sqrt(1 - b2^t).
    r = _rng(3)
    lr, b1, b2, eps = 1e-3, 0.9, 0.999, 1e-8
    th = r.standard_normal(200)
    m, v = np.zeros(200), np.zeros(200)
    th_ref, m_ref, v_ref = th.copy(), np.zeros(200), np.zeros(200)
    for t in range(1, 8):
        g = r.standard_normal(200)
        th, m, v = oracle.adam_update(th, g, m, v, lr, b1, b2, eps, t)
        m_ref = b1 * m_ref + (1 - b1) * g
        v_ref = b2 * v_ref + (1 - b2) * g * g
        mhat, vhat = m_ref / (1 - b1 ** t), v_ref / (1 - b2 ** t)
        th_ref = th_ref - lr * mhat / (np.sqrt(vhat) + eps / np.sqrt(1 - b2 ** t))
    np.testing.assert_allclose(th, th_ref, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(m, m_ref, rtol=1e-14)
