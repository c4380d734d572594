"""UniPC multistep update for the flow-matching sampler (oracle; test
infrastructure only).

The paper runs its Wan experiments on a 50-step UniPC sampler (Sec. 4.1,
citing Zhao et al., "UniPC: A Unified Predictor-Corrector Framework for Fast
Sampling of Diffusion Models", 2023).  This module restates that method for
the rectified-flow parametrisation used here:

  x_sigma = alpha_sigma x_data + sigma n,  alpha = 1 - sigma,
  data prediction m = x - sigma v  (v = the network's velocity),
  lambda = log(alpha / sigma),  h = lambda_t - lambda_s  (step s -> t).

UniPC-2 with B(h) = e^h - 1 in data-prediction form ("bh2"):

  predictor (order k), from the corrected sample x_s with history m_s, m_p:
    x_t = (sigma_t / sigma_s) x_s - alpha_t (e^{-h} - 1) m_s
          - [k = 2] alpha_t B 0.5 (m_p - m_s) / r,   r = (lambda_p - lambda_s) / h
  corrector (order k), after the network has seen x_t and returned m_t:
    x_t^c = (sigma_t / sigma_s) x_s - alpha_t (e^{-h} - 1) m_s
            - alpha_t B (rho_1 (m_p - m_s) / r + rho_t (m_t - m_s))
    k = 1: rho_t = 1/2, no rho_1 term;  k = 2: (rho_1, rho_t) solve
    [[1, 1], [r, 1]] rho = (b_1, b_2)
  with B = e^{-h} - 1, phi_1 = B / (-h) - 1, phi_2 = phi_1 / (-h) - 1/2,
  b_1 = phi_1 / B, b_2 = 2 phi_2 / B.

Orders (UniPC's warm-up and lower-order final steps): the predictor of
step i has order min(2, i + 1, T - i); the corrector of step i >= 1 uses the
order of step i - 1's predictor.  At sigma = 1 (alpha = 0) lambda = -inf and
at sigma = 0 lambda = +inf: h is then +inf, e^{-h} = 0, phi_1 = -1,
phi_2 = -1/2, and any history ratio r through such a point is -inf (its
term vanishes).  These are the limits of the formulas, taken exactly.

Pinned by: order-1 prediction without correction equals the Euler step; a
constant velocity field is integrated exactly; the global error on a smooth
linear ODE falls at second order or faster as T doubles (tests).
"""
import math

import numpy as np


def _lam(sig):
    a = 1.0 - sig
    if a <= 0.0:
        return -math.inf
    if sig <= 0.0:
        return math.inf
    return math.log(a) - math.log(sig)


def step_terms(sig_s, sig_t):
    """(h, e^{-h} - 1, b_1, b_2) of the step sigma_s -> sigma_t."""
    h = _lam(sig_t) - _lam(sig_s)
    if math.isinf(h):
        return math.inf, -1.0, 1.0, 1.0
    hh = -h
    B = math.expm1(hh)
    phi1 = B / hh - 1.0
    phi2 = phi1 / hh - 0.5
    return h, B, phi1 / B, 2.0 * phi2 / B


def ratio(sig_p, sig_s, h):
    """r = (lambda_p - lambda_s) / h; -inf when lambda_p is (an exact limit)."""
    lp = _lam(sig_p)
    if math.isinf(lp) or math.isinf(h):
        return -math.inf
    return (lp - _lam(sig_s)) / h


def predict(x_s, m_s, m_p, sig_s, sig_p, sig_t, order):
    """UniP step s -> t of the given order (m_p, sig_p: the step before s)."""
    h, B, _, _ = step_terms(sig_s, sig_t)
    a_t = 1.0 - sig_t
    x = (sig_t / sig_s) * x_s - a_t * B * m_s
    if order == 2:
        r = ratio(sig_p, sig_s, h)
        if not math.isinf(r):
            x = x - a_t * B * 0.5 * (m_p - m_s) / r
    return x


def correct(x_s, m_s, m_p, m_t, sig_s, sig_p, sig_t, order):
    """UniC correction of x_t after the network returned m_t at x_t."""
    h, B, b1, b2 = step_terms(sig_s, sig_t)
    a_t = 1.0 - sig_t
    x = (sig_t / sig_s) * x_s - a_t * B * m_s
    if order == 1:
        return x - a_t * B * 0.5 * (m_t - m_s)
    r = ratio(sig_p, sig_s, h)
    if math.isinf(r):
        return x - a_t * B * b1 * (m_t - m_s)
    rho1 = (b1 - b2) / (1.0 - r)
    rho_t = b1 - rho1
    return x - a_t * B * (rho1 * (m_p - m_s) / r + rho_t * (m_t - m_s))


def orders(T, max_order=2):
    """Predictor order of every step: min(max_order, i + 1, T - i)."""
    return [min(max_order, i + 1, T - i) for i in range(T)]


def integrate(velocity, x0, sigmas, corrector=True, max_order=2, rnd=lambda a: a):
    """Plain UniPC loop over a velocity callable v(x, sigma) (used by the pins;
    the sampler inlines the same two updates around its network call).
    ``rnd`` is applied at the storage points (f32 rounding in the sampler)."""
    T = len(sigmas) - 1
    ords = orders(T, max_order)
    x = rnd(np.asarray(x0, np.float64))
    hist = []       # data predictions m_0 .. m_{i-1}
    x_last = None   # corrected sample that fed the previous predictor
    for i in range(T):
        v = velocity(x, sigmas[i])
        m = rnd(x - sigmas[i] * v)
        if corrector and i > 0:
            m_p = hist[-2] if len(hist) > 1 else None
            x = rnd(correct(x_last, hist[-1], m_p, m, sigmas[i - 1],
                            sigmas[i - 2] if i > 1 else 1.0, sigmas[i], ords[i - 1]))
        hist.append(m)
        x_last = x
        m_p = hist[-2] if len(hist) > 1 else None
        x = rnd(predict(x, m, m_p, sigmas[i], sigmas[i - 1] if i > 0 else 1.0, sigmas[i + 1], ords[i]))
    return x
