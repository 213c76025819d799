"""Pins of the training-step reference (L1 gradient, Adam) against closed
forms that a mistake in the reference (a dropped bias correction, swapped
decay rates, a wrong sign) would break."""
import numpy as np

from oracle.train_ref import adam_step, l1_loss_grad


def test_l1_sign_and_sum():
    img = np.array([0.5, 0.25, 1.0, 0.0], np.float32)
    tgt = np.array([0.25, 0.25, 2.0, -1.0], np.float32)
    g, loss = l1_loss_grad(img, tgt)
    assert np.array_equal(g, [1.0, 0.0, -1.0, 1.0])
    assert loss == 0.25 + 0.0 + 1.0 + 1.0


def test_adam_first_step_closed_form():
    # t = 1 from zero moments: m_hat = g, v_hat = g^2 exactly, so the step is
    # lr g / (|g| + eps) whatever the decay rates are
    rng = np.random.default_rng(0)
    p, g = rng.standard_normal(100), rng.standard_normal(100)
    for b1, b2 in ((0.9, 0.999), (0.5, 0.25), (0.0, 0.0)):
        p1, m1, v1 = adam_step(p, g, np.zeros(100), np.zeros(100), 1, 1e-2, b1, b2, 1e-8)
        np.testing.assert_allclose(p1, p - 1e-2 * g / (np.abs(g) + 1e-8), rtol=0, atol=1e-15)
        np.testing.assert_allclose(m1, (1 - b1) * g, rtol=1e-15)
        np.testing.assert_allclose(v1, (1 - b2) * g * g, rtol=1e-15)


def test_adam_constant_gradient():
    # with a constant gradient the bias-corrected moments stay g and g^2, so
    # every step moves by lr g / (|g| + eps)
    g = np.array([3.0, -0.5, 1e-3])
    p, m, v = np.zeros(3), np.zeros(3), np.zeros(3)
    for t in range(1, 8):
        p, m, v = adam_step(p, g, m, v, t, 0.1, 0.9, 0.99, 0.0)
        np.testing.assert_allclose(p, -0.1 * t * np.sign(g), rtol=1e-12)


def test_adam_zero_gradient_and_decay():
    # a zero gradient after a first step: the first moment decays by b1 per
    # step, the second by b2, and the parameter keeps moving by the
    # bias-corrected ratio
    g0 = np.array([2.0])
    p, m, v = adam_step(np.zeros(1), g0, np.zeros(1), np.zeros(1), 1, 1.0, 0.5, 0.75, 0.0)
    p2, m2, v2 = adam_step(p, np.zeros(1), m, v, 2, 1.0, 0.5, 0.75, 0.0)
    assert m2[0] == 0.5 * m[0] and v2[0] == 0.75 * v[0]
    m_hat, v_hat = m2[0] / (1 - 0.25), v2[0] / (1 - 0.5625)
    np.testing.assert_allclose(p2, p - m_hat / np.sqrt(v_hat), rtol=1e-15)
