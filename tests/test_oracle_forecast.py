"""Pins for the finite-difference forecast (Eq. 2): exact on linear trajectories, the
closed-form bias on quadratics, order 0 is reuse, the warm-up cap, and the closed-form
coefficient form of the same recursion."""
import numpy as np
import pytest

import oracle as O


def traj(fn, R, n_ref):
    """Feed refreshes at tau = 0, R, 2R, ... of the trajectory fn(tau) into a cache."""
    def run(K):
        c = O.TaylorCache(K)
        for j in range(n_ref):
            c.refresh(fn(j * R), j * R)
        return c
    return run


@pytest.mark.parametrize("K", [1, 2, 3])
@pytest.mark.parametrize("R", [1, 3, 5])
def test_first_order_is_exact_on_linear_trajectories(K, R):
    a = np.array([0.3, -1.2, 2.5])
    b = np.array([0.7, 0.01, -0.4])
    fn = lambda tau: a + b * tau
    for n_ref in (2, 3, 5):
        c = traj(fn, R, n_ref)(K)
        tau_j = (n_ref - 1) * R
        for m in range(1, R):
            np.testing.assert_allclose(c.forecast(tau_j + m), fn(tau_j + m), rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("R", [2, 5, 6])
def test_quadratic_bias_closed_forms(R):
    a, b, cc = 0.5, -0.25, 0.125
    fn = lambda tau: np.array([a + b * tau + cc * tau * tau])
    for n_ref in (2, 3, 4):
        tau_j = (n_ref - 1) * R
        for m in range(1, R):
            true = fn(tau_j + m)[0]
            f1 = traj(fn, R, n_ref)(1).forecast(tau_j + m)[0]
            assert abs((f1 - true) - (-cc * m * (m + R))) < 1e-10
            f2 = traj(fn, R, n_ref)(2).forecast(tau_j + m)[0]
            expect2 = -cc * R * m if n_ref >= 3 else -cc * m * (m + R)   # warm-up: j=1 caps at order 1
            assert abs((f2 - true) - expect2) < 1e-10


def test_order_zero_is_reuse_and_first_refresh_caps_order():
    rng = np.random.default_rng(0)
    hist = [rng.standard_normal(7) for _ in range(3)]
    c0 = O.TaylorCache(0)
    c2 = O.TaylorCache(2)
    for j, h in enumerate(hist[:1]):
        c0.refresh(h, j * 4)
        c2.refresh(h, j * 4)
    # only one refresh: every order reduces to reuse of that feature
    np.testing.assert_array_equal(c2.forecast(3), hist[0])
    for j, h in enumerate(hist[1:], start=1):
        c0.refresh(h, j * 4)
    np.testing.assert_array_equal(c0.forecast(9), hist[-1])
    with pytest.raises(RuntimeError):
        O.TaylorCache(1).forecast(1)


def coeffs_closed_form(K, R, m):
    a = m / R
    b = m * m / (2.0 * R * R)
    if K == 0:
        return [1.0]
    if K == 1:
        return [1 + a, -a]
    return [1 + a + b, -a - 2 * b, b]


@pytest.mark.parametrize("K", [0, 1, 2])
def test_recursion_equals_coefficient_form(K):
    rng = np.random.default_rng(K)
    R = 5
    hist = [rng.standard_normal(11) for _ in range(6)]
    c = O.TaylorCache(K)
    for j, h in enumerate(hist):
        c.refresh(h, j * R)
    tau_j = 5 * R
    for m in range(1, R):
        cf = coeffs_closed_form(K, R, m)
        expect = sum(cf[q] * hist[-1 - q] for q in range(K + 1))
        np.testing.assert_allclose(c.forecast(tau_j + m), expect, rtol=1e-12, atol=1e-12)
