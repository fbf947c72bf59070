"""Pins of the optimiser oracle and the learning-rate schedules (CPU only):
closed forms of Adam for constant and sign-flipping gradients, its scale
invariance, SGD and the delay clamp, and the schedules' closed forms."""
import math

import numpy as np
import pytest

from oracle.optim import Optimiser, adam, adam_init, clamp_delays, sgd
from paper_2501_07331_amd import schedules


def test_adam_constant_gradient_moves_by_lr_every_step():
    # with g constant, m_k = (1 - b1^k) g and v_k = (1 - b2^k) g^2, so the
    # bias-corrected step is lr g / (|g| + eps) at every k
    g = np.array([2.5, -0.01, 3e-6, -7.0])
    x = np.zeros(4)
    st = adam_init(4)
    lr, eps = 0.05, 1e-8
    for k in range(1, 7):
        x_new = adam(x, g, lr, st, eps=eps)
        assert np.allclose(x - x_new, lr * g / (np.abs(g) + eps), rtol=1e-12, atol=0)
        x = x_new
    assert st.k == 6


def test_adam_sign_flip_two_steps():
    # g = +1 then -1 with b1 = 0.9, b2 = 0.999: m2 = 0.9*0.1 - 0.1 = -0.01,
    # 1 - b1^2 = 0.19, so m_hat = -1/19; v2 = 0.999*0.001 + 0.001 = 0.001999
    # = 1 - b2^2, so v_hat = 1: the second step is +lr/19 / (1 + eps)
    st = adam_init(1)
    lr, eps = 1.0, 1e-8
    x1 = adam(np.zeros(1), np.ones(1), lr, st, eps=eps)
    assert x1[0] == pytest.approx(-1.0 / (1.0 + eps), rel=1e-14)
    x2 = adam(x1, -np.ones(1), lr, st, eps=eps)
    assert x2[0] - x1[0] == pytest.approx((1.0 / 19.0) / (1.0 + eps), rel=1e-12)


def test_adam_is_invariant_to_gradient_scale():
    rng = np.random.default_rng(5)
    gs = rng.normal(size=(5, 10))
    a, b = adam_init(10), adam_init(10)
    xa = xb = np.zeros(10)
    for g in gs:
        xa = adam(xa, g, 0.1, a, eps=0.0)
        xb = adam(xb, 1e4 * g, 0.1, b, eps=0.0)
    assert np.allclose(xa, xb, rtol=1e-12, atol=1e-15)


def test_sgd_and_clamp():
    assert np.array_equal(sgd([1.0, 2.0], [0.5, -1.0], 2.0), [0.0, 4.0])
    assert np.array_equal(clamp_delays([-1.0, 3.0, 300.0], 0.0, 255.0), [0.0, 3.0, 255.0])


def test_optimiser_per_projection_factors_and_freeze():
    W = [np.ones((2, 2)), np.ones((2, 3))]
    D = [np.full((2, 2), 5.0), np.full((2, 3), 5.0)]
    g = [np.ones((2, 2)), np.ones((2, 3))]
    o = Optimiser("sgd")
    W1, D1 = o.step(W, D, g, g, 0.5, 10.0, 0.0, 4.0, scale_w=[1.0, 0.0], scale_d=[0.0, 1.0])
    assert np.all(W1[0] == 0.5) and np.all(W1[1] == 1.0)
    assert np.all(D1[0] == 4.0)            # unchanged 5.0, clamped to d_max
    assert np.all(D1[1] == 0.0)            # 5 - 10, clamped to d_min


def test_schedules():
    assert schedules.epoch_decay(0.01, 0) == 0.01
    assert schedules.epoch_decay(0.01, 3) == pytest.approx(0.01 * 0.998 ** 3, rel=1e-15)
    # 1e-3 * 1.05^k reaches 1 at k = ceil(ln 1000 / ln 1.05) = 142
    k = math.ceil(math.log(1000.0) / math.log(1.05))
    assert k == 142
    assert schedules.ease_in(2.0, 0) == pytest.approx(2e-3)
    assert schedules.ease_in(2.0, k - 1) < 2.0
    assert schedules.ease_in(2.0, k) == 2.0 and schedules.ease_in(2.0, 10 * k) == 2.0
    with pytest.raises(ValueError):
        schedules.ease_in(1.0, -1)
