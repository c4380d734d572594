"""Pins of the oracle's UniPC update (the Wan sampler of Sec. 4.1): reductions
to the Euler step, exactness on constant velocity, and its convergence order
on a linear ODE with a closed-form solution."""
import math

import numpy as np
import pytest

from oracle import sigma_schedule
from oracle.unipc import integrate, orders, predict, step_terms


def euler(velocity, x0, sigmas):
    x = np.asarray(x0, np.float64)
    for i in range(len(sigmas) - 1):
        x = x + (sigmas[i + 1] - sigmas[i]) * velocity(x, sigmas[i])
    return x


def nonlinear(x, s):
    return np.sin(3 * x) + 0.5 * s * x


X0 = np.linspace(-2.0, 2.0, 17)


@pytest.mark.parametrize("shift", [1.0, 3.0, 5.0])
def test_order1_without_corrector_is_euler(shift):
    """sigma_t/sigma_s x - alpha_t (e^{-h}-1)(x - sigma_s v) = x + (sigma_t - sigma_s) v."""
    sig = sigma_schedule(12, shift)
    a = integrate(nonlinear, X0, sig, corrector=False, max_order=1)
    np.testing.assert_allclose(a, euler(nonlinear, X0, sig), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("corrector", [False, True])
def test_constant_velocity_is_exact(corrector):
    """x(sigma) = m + sigma c has a constant data prediction m: every order and
    the corrector reproduce it, x_T = x_0 - c."""
    c = np.cos(X0)
    for T in (1, 2, 5, 13):
        sig = sigma_schedule(T, 3.0)
        x = integrate(lambda x, s: c, X0, sig, corrector=corrector)
        np.testing.assert_allclose(x, X0 - c, rtol=1e-12, atol=1e-12)


def test_single_step_is_euler():
    sig = sigma_schedule(1, 1.0)
    np.testing.assert_allclose(integrate(nonlinear, X0, sig), euler(nonlinear, X0, sig), rtol=1e-14)


def test_order_schedule():
    assert orders(1) == [1]
    assert orders(2) == [1, 1]
    assert orders(5) == [1, 2, 2, 2, 1]


def test_step_terms_limits_and_small_h():
    # sigma_s = 1 (alpha = 0) or sigma_t = 0: h = inf, e^{-h} - 1 = -1, b = (1, 1)
    assert step_terms(1.0, 0.5)[1:] == (-1.0, 1.0, 1.0)
    assert step_terms(0.5, 0.0)[1:] == (-1.0, 1.0, 1.0)
    # h -> 0: b_1 -> 1/2, b_2 -> 1/3 (series of phi_1, phi_2)
    _, B, b1, b2 = step_terms(0.5, 0.5 - 1e-4)
    assert abs(b1 - 0.5) < 1e-3 and abs(b2 - 1.0 / 3.0) < 1e-3


def test_linear_ode_convergence_order():
    """dx/dsigma = k x from sigma = 1 to 0: x(0) = x(1) e^{-k}.  Once T is past
    the pre-asymptotic range, doubling T cuts the UniPC error by at least 2^1.8
    (second order: its first and last steps are order 1 with O(h^2) local
    error); Euler's error halves."""
    k = 1.3
    vel = lambda x, s: k * x
    exact = X0 * math.exp(-k)
    errs, errs_e = [], []
    for T in (40, 80, 160, 320):
        sig = sigma_schedule(T, 1.0)
        errs.append(np.max(np.abs(integrate(vel, X0, sig) - exact)))
        errs_e.append(np.max(np.abs(euler(vel, X0, sig) - exact)))
    for a, b in zip(errs, errs[1:]):
        assert a / b > 2 ** 1.8, errs
    assert errs[-1] < errs_e[-1] / 100
    for a, b in zip(errs_e, errs_e[1:]):
        assert 1.8 < a / b < 2.2


def test_predictor_second_order_uses_history():
    """Order 2 differs from order 1 by -alpha_t B (m_p - m_s) / (2 r)."""
    x, ms, mp = np.array([0.3]), np.array([0.1]), np.array([-0.2])
    p1 = predict(x, ms, mp, 0.6, 0.8, 0.4, 1)
    p2 = predict(x, ms, mp, 0.6, 0.8, 0.4, 2)
    lam = lambda s: math.log((1 - s) / s)
    h = lam(0.4) - lam(0.6)
    r = (lam(0.8) - lam(0.6)) / h
    B = math.exp(-h) - 1.0
    np.testing.assert_allclose(p2 - p1, -(1 - 0.4) * B * 0.5 * (mp - ms) / r, rtol=1e-12)
