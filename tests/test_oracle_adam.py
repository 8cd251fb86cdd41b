"""Pins of the Adam oracle (oracle/adam.py) to closed forms of Algorithm 1 of
Kingma and Ba: from zero moments the bias-corrected moments of a constant
gradient are exactly g and g^2, so every step moves a parameter by
lr * g / (|g| + eps); with a zero gradient the moments decay geometrically;
each row takes its own learning rate; the half copy rounds to nearest even."""
import numpy as np

from oracle import adam

B1, B2, EPS = 0.9, 0.999, 1e-8


def test_first_step_is_lr_times_normalised_gradient():
    rng = np.random.default_rng(0)
    g = rng.normal(size=(3, 50)) * np.logspace(-6, 2, 50)
    g[1, 7] = 0.0
    theta0 = rng.normal(size=g.shape)
    lr = np.array([1e-3, 5e-2, 2.0])
    th, m, v = adam.adam_step(theta0, g, np.zeros_like(g), np.zeros_like(g), lr, B1, B2, EPS, 1)
    expect = theta0 - lr[:, None] * g / (np.abs(g) + EPS)
    assert np.allclose(th, expect, rtol=1e-13, atol=1e-15)
    assert np.allclose(m, (1 - B1) * g, rtol=1e-15, atol=0) and np.allclose(v, (1 - B2) * g * g, rtol=1e-15, atol=0)
    assert th[1, 7] == theta0[1, 7]


def test_constant_gradient_moves_linearly_with_bias_correction():
    # without the 1 - b^t corrections the first steps would be 10x and ~30x too short
    g = np.array([[0.3, -2.0, 1e-4, 50.0]])
    theta = np.zeros_like(g)
    m = np.zeros_like(g)
    v = np.zeros_like(g)
    for t in range(1, 26):
        theta, m, v = adam.adam_step(theta, g, m, v, [0.01], B1, B2, EPS, t)
        expect = -t * 0.01 * g / (np.abs(g) + EPS)
        assert np.allclose(theta, expect, rtol=1e-11, atol=1e-15), t


def test_zero_gradient_decays_moments_geometrically():
    rng = np.random.default_rng(1)
    m0 = rng.normal(size=(2, 9))
    v0 = rng.random((2, 9))
    theta, m, v = rng.normal(size=(2, 9)), m0.copy(), v0.copy()
    b1, b2 = 0.8, 0.95
    for t in range(1, 7):
        theta, m, v = adam.adam_step(theta, np.zeros_like(m0), m, v, [1e-3, 1e-3], b1, b2, EPS, t)
        assert np.allclose(m, b1 ** t * m0, rtol=1e-14, atol=0)
        assert np.allclose(v, b2 ** t * v0, rtol=1e-14, atol=0)


def test_one_learning_rate_per_row():
    rng = np.random.default_rng(2)
    g = rng.normal(size=(4, 30))
    theta0 = rng.normal(size=g.shape)
    lr = np.array([0.0, 1e-3, 3e-2, 1.0])
    th, _, _ = adam.adam_step(theta0, g, np.zeros_like(g), np.zeros_like(g), lr, B1, B2, EPS, 1)
    assert np.array_equal(th[0], theta0[0])
    for r in range(1, 4):
        step = (theta0[r] - th[r]) / (g[r] / (np.abs(g[r]) + EPS))
        assert np.allclose(step, lr[r], rtol=1e-10)


def test_half_copy_rounds_to_nearest_even():
    x = np.array([1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11, -(2.0 + 2.0 ** -10), 65519.0, 65520.0, 1e-8],
                 np.float32)
    h = adam.half_copy(x).view(np.float16).astype(np.float64)
    assert h[0] == 1.0                        # tie -> even mantissa
    assert h[1] == 1.0 + 2.0 ** -9            # tie -> even mantissa (upwards)
    assert h[2] == -2.0                       # tie at exponent 1 -> even
    assert h[3] == 65504.0                    # largest finite binary16
    assert np.isinf(h[4])                     # rounds past the largest finite value
    assert h[5] == 0.0                        # below half the smallest subnormal
