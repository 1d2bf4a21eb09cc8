"""Pins of the optimizer oracle (AdamW, the reading of the unnamed optimizer of Sec. 4.1)
against closed forms of its published definition: the first step, a zero gradient (pure
decoupled decay) and a constant gradient (exact bias correction)."""
import numpy as np

import oracle as O


def _rng(seed=0):
    return np.random.default_rng(seed)


def test_first_step_is_normalised_gradient_plus_decay():
    # t = 1: m_hat = g and v_hat = g^2 exactly, so the step is lr (g / (|g| + eps) + wd w)
    r = _rng(1)
    w, g = r.standard_normal(1000), r.standard_normal(1000) * 1e-3
    lr, wd, eps = 1e-2, 0.1, 1e-8
    w1, m1, v1 = O.adamw_step(w, g, np.zeros_like(w), np.zeros_like(w), 1, lr, 0.9, 0.999, eps, wd)
    np.testing.assert_allclose(w1, w - lr * (g / (np.abs(g) + eps) + wd * w), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(m1, 0.1 * g, rtol=1e-12)
    np.testing.assert_allclose(v1, 0.001 * g * g, rtol=1e-12)


def test_zero_gradient_is_pure_decoupled_decay():
    # g = 0: moments stay 0, the update is the decay alone, w_t = w_0 (1 - lr wd)^t
    r = _rng(2)
    w0 = r.standard_normal(257)
    w, m, v = w0.copy(), np.zeros(257), np.zeros(257)
    for t in range(1, 6):
        w, m, v = O.adamw_step(w, np.zeros(257), m, v, t, 3e-2, 0.9, 0.999, 1e-8, 0.5)
    np.testing.assert_allclose(w, w0 * (1 - 3e-2 * 0.5) ** 5, rtol=1e-12)
    assert not m.any() and not v.any()


def test_constant_gradient_has_exact_bias_correction():
    # g_t = g: m_t = (1 - b1^t) g and v_t = (1 - b2^t) g^2, so every step moves by
    # lr g / (|g| + eps) and after t steps w = w_0 - t lr g / (|g| + eps)
    r = _rng(3)
    w0, g = r.standard_normal(64), r.standard_normal(64)
    w, m, v = w0.copy(), np.zeros(64), np.zeros(64)
    for t in range(1, 11):
        w, m, v = O.adamw_step(w, g, m, v, t, 1e-3, 0.9, 0.999, 1e-8, 0.0)
    np.testing.assert_allclose(w, w0 - 10 * 1e-3 * g / (np.abs(g) + 1e-8), rtol=1e-10)
    np.testing.assert_allclose(m, (1 - 0.9 ** 10) * g, rtol=1e-12)
    np.testing.assert_allclose(v, (1 - 0.999 ** 10) * g * g, rtol=1e-12)
