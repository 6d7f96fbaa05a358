"""Theorem 1 (Sec. 3, proof in App. A) at the oracle level: for heavy-ball
momentum M_t = mu M_{t-1} + grad F(x_t), x_t = x_{t-1} - eta M_{t-1}, the
statistic the oracle computes from the two momentum norms satisfies

    RMMC_t = | eta kappa_M(x_{t-1}) + B_t | + O(eta^2),
    kappa_M = v^T H v (v = M_{t-1} / ||M_{t-1}||),
    B_t = (1 - mu) - v^T grad F(x_{t-1}) / ||M_{t-1}||.

On a quadratic F(x) = x^T H x / 2 + c^T x the gradient step is exact, so the
only remainder comes from the part of grad F(x_t) orthogonal to v (it adds
||g_perp||^2 / (2 m (mu m + v^T g)) to the norm):
* x and M on one eigendirection of H: the identity is exact;
* grad F(x_{t-1}) along M_{t-1}: g_perp = -eta m (H v)_perp, so the remainder
  is second order in eta (halving eta quarters it) and matches that leading
  term;
* steady state m = ||grad F|| / (1 - mu) with v along grad F: B_t = 0 and the
  statistic measures eta |kappa_M|.
CPU only; eps = 0 in the statistic (the theorem's definition).
"""
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))

import oracle as O  # noqa: E402

MU = 0.95


def _quadratic(d, seed):
    rng = np.random.default_rng(seed)
    A = rng.standard_normal((d, d))
    U, _ = np.linalg.qr(A)
    lam = np.linspace(0.5, 4.0, d)
    H = (U * lam) @ U.T
    c = rng.standard_normal(d)
    return H, c, U, lam


def _step_stat(H, c, x_prev, M_prev, eta):
    """One heavy-ball step; returns the oracle's statistic and the theorem's terms."""
    grad = lambda x: H @ x + c
    x_t = x_prev - eta * M_prev
    M_t = MU * M_prev + grad(x_t)
    m_prev, m_t = O.frobenius_norm(M_prev), O.frobenius_norm(M_t)
    stat = O.rmmc(m_t, m_prev, 0.0)
    v = M_prev / m_prev
    kappa = float(v @ H @ v)
    B = (1.0 - MU) - float(v @ grad(x_prev)) / m_prev
    g_t = grad(x_t)
    g_perp = g_t - (v @ g_t) * v
    lead = float(g_perp @ g_perp) / (2.0 * m_prev * (MU * m_prev + float(v @ g_t)))
    return stat, abs(eta * kappa + B), lead, kappa, B


def test_exact_on_an_eigendirection():
    H, c, U, lam = _quadratic(12, 1)
    u = U[:, 3]
    # x_{t-1} and M_{t-1} in span(u), with c removed along the other directions
    c_u = (u @ c) * u
    for eta in (0.1, 0.03, 0.01):
        x_prev = 0.7 * u
        M_prev = 2.5 * u
        grad = lambda x: H @ x + c_u
        x_t = x_prev - eta * M_prev
        M_t = MU * M_prev + grad(x_t)
        stat = O.rmmc(O.frobenius_norm(M_t), O.frobenius_norm(M_prev), 0.0)
        v = M_prev / np.linalg.norm(M_prev)
        pred = abs(eta * float(v @ H @ v) + (1 - MU) - float(v @ grad(x_prev)) / np.linalg.norm(M_prev))
        assert abs(stat - pred) <= 1e-13 * max(1.0, pred), (eta, stat, pred)
        assert abs(float(v @ H @ v) - lam[3]) < 1e-12


def test_second_order_remainder_when_gradient_follows_momentum():
    H, c, _, _ = _quadratic(16, 2)
    rng = np.random.default_rng(3)
    x_prev = rng.standard_normal(16)
    g0 = H @ x_prev + c
    M_prev = 3.0 * g0 / np.linalg.norm(g0)   # momentum along the gradient, m = 3
    res = []
    for eta in (0.02, 0.01, 0.005, 0.0025):
        stat, pred, lead, _, _ = _step_stat(H, c, x_prev, M_prev, eta)
        res.append(stat - pred)
        # the remainder is the orthogonal-gradient term, to higher order
        assert abs((stat - pred) - lead) <= 0.05 * abs(lead) + 1e-15
    ratios = [res[i] / res[i + 1] for i in range(len(res) - 1)]
    for q in ratios:
        assert 3.8 < q < 4.2, ratios          # O(eta^2)


def test_steady_state_measures_curvature():
    H, c, _, lam = _quadratic(10, 4)
    rng = np.random.default_rng(5)
    x_prev = rng.standard_normal(10)
    g0 = H @ x_prev + c
    M_prev = g0 / (1.0 - MU)                 # equilibrium momentum: B_t = 0
    for eta in (0.004, 0.002):
        stat, pred, _, kappa, B = _step_stat(H, c, x_prev, M_prev, eta)
        assert abs(B) < 1e-12
        assert lam[0] - 1e-12 <= kappa <= lam[-1] + 1e-12
        assert abs(pred - eta * abs(kappa)) < 1e-12
        assert abs(stat - eta * kappa) <= 0.1 * eta * kappa


def test_bias_term_dominates_while_momentum_builds():
    """From M = 0 the first steps have large |B_t| (momentum far below its
    equilibrium), and B_t decays as momentum builds: the early-training regime
    the paper describes."""
    H, c, _, _ = _quadratic(8, 6)
    eta = 1e-3
    x = np.zeros(8)
    M = H @ x + c                               # M_1 = grad F(x_0)
    Bs = []
    for _ in range(60):
        _, _, _, _, B = _step_stat(H, c, x, M, eta)
        Bs.append(abs(B))
        x = x - eta * M
        M = MU * M + (H @ x + c)
    assert Bs[0] > 0.9 and Bs[-1] < 0.1 * Bs[0]
    assert all(Bs[i + 1] <= Bs[i] + 1e-12 for i in range(20))
