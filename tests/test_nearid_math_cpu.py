"""The second CholQR pass of fp32-gradient layers (Orthogonalize of Algorithm
1 / 2) factors a Gram matrix W1 = I + E that is the identity to within
||E||_F <= 2^-10 by the fixed point U = Phi(E - U^T U), T1 = I + U, with
Phi(S) the strict upper triangle of S plus half its diagonal, and inverts the
64 x 64 diagonal blocks of T1 by the series sum_j (-U_kk)^j (Horner's rule,
V <- I - U V).  These tests hold the step counts the kernels use (four
products, the fifth power) to the Cholesky factor and the inverse numpy
computes: at the bound they agree to fp64 rounding, fewer steps do not, and
past the bound the fixed count falls short, which is why such layers take the
blocked factorisation.  No GPU: plain numpy on random symmetric E."""
import numpy as np
import pytest

NID_ITERS, NID_SERIES, BOUND = 4, 5, 2.0 ** -10
BLOCK = 64


def phi(S):
    return np.triu(S, 1) + np.diag(np.diag(S)) / 2


def near_identity_factor(E, iters=NID_ITERS):
    U = phi(E)
    for _ in range(iters):
        U = phi(E - U.T @ U)
    return np.eye(len(E)) + U


def series_inverse(T, terms=NID_SERIES):
    U = T - np.eye(len(T))
    V = np.eye(len(T))
    for _ in range(terms):
        V = np.eye(len(T)) - U @ V
    return V


def random_E(r, norm, seed):
    A = np.random.default_rng(seed).standard_normal((r, r))
    E = (A + A.T) / 2
    return E * (norm / np.linalg.norm(E))


@pytest.mark.parametrize("r", [64, 160, 512])
def test_fixed_point_is_the_cholesky_factor_at_the_bound(r):
    E = random_E(r, BOUND, r)
    T = near_identity_factor(E)
    T_ref = np.linalg.cholesky(np.eye(r) + E).T
    assert np.allclose(np.tril(T, -1), 0.0)
    assert np.abs(T - T_ref).max() <= 1e-15
    assert np.abs(T.T @ T - (np.eye(r) + E)).max() <= 1e-15
    for k0 in range(0, r, BLOCK):
        Tk = T[k0:k0 + BLOCK, k0:k0 + BLOCK]
        assert np.abs(series_inverse(Tk) - np.linalg.inv(Tk)).max() <= 1e-15


def rank_one_E(r, norm, seed, sign=1.0):
    v = np.random.default_rng(seed).standard_normal(r)
    E = sign * np.outer(v, v)
    return E * (norm / np.linalg.norm(E))


@pytest.mark.parametrize("sign", [1.0, -1.0])
def test_fewer_steps_fall_short_at_the_bound(sign):
    """A rank-one E (the slowest case: U^T U is as large as ||U||^2 allows)
    needs three products; the kernels' four leave one step of margin."""
    r = 256
    E = rank_one_E(r, BOUND, 3, sign)
    T_ref = np.linalg.cholesky(np.eye(r) + E).T
    err = [np.abs(near_identity_factor(E, k) - T_ref).max() for k in range(NID_ITERS + 1)]
    assert err[0] > 1e-9 and err[1] > 1e-12 and err[2] > 1e-15
    assert err[3] <= 1e-15 and err[NID_ITERS] <= 1e-15
    Tk = T_ref[:BLOCK, :BLOCK]
    assert np.abs(series_inverse(Tk, 2) - np.linalg.inv(Tk)).max() > 1e-15


@pytest.mark.parametrize("E", [random_E(128, 0.25, 11), rank_one_E(128, 0.25, 5)], ids=["random", "rank-one"])
def test_past_the_bound_the_fixed_count_falls_short(E):
    T_ref = np.linalg.cholesky(np.eye(len(E)) + E).T
    assert np.abs(near_identity_factor(E) - T_ref).max() > 1e-13
