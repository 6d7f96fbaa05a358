"""Pins for the float64 oracle: each check ties it to something other than
itself (a hand-worked example, closed forms, invariants, an explicit SVD, an
independent orthonormaliser, brute force on tiny inputs).

Each ``check_*`` raises AssertionError on failure; the tests call them on the
oracle as written, and ``test_planted_mistakes_are_caught`` re-runs them on
copies of the oracle with plausible mistakes planted, to show that every such
mistake fails at least one pin.
"""
import math
import os
import types

import numpy as np
import pytest

import oracle as O
from oracle import curvadion_oracle as OC

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_2x2.txt")


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _load_golden(path=GOLDEN):
    vals = {}
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, rhs = [s.strip() for s in line.split("=", 1)]
        vals[key] = np.array([eval(tok, {"__builtins__": {}, "sqrt": math.sqrt})
                              for tok in rhs.split()], dtype=np.float64)
    return vals


# ---------------------------------------------------------------------------
# checks (parameterised by the oracle module so mutants can be run through them)
# ---------------------------------------------------------------------------
def check_golden(o):
    """The hand-worked 2x2 example (three steps: sync, local, RMMC = 0)."""
    gv = _load_golden()
    L = o.OracleLayer.from_arrays(np.zeros((2, 2)), np.zeros((2, 2)), gv["Q0"].reshape(2, 1))
    grads = [gv["G1"].reshape(2, 2), gv["G2"].reshape(2, 2), gv["G3"].reshape(2, 2)]
    for t, G in enumerate(grads, start=1):
        res = o.group_step([L], [G], mu=0.5, eta=0.1, tau=0.5, eps=1e-8)
        pre = f"step{t}."
        assert int(res["flag"]) == int(gv[pre + "flag"][0]), (t, res)
        assert abs(res["rmmc"][0] - gv[pre + "rmmc"][0]) <= 1e-12 * max(1.0, abs(gv[pre + "rmmc"][0])), t
        if pre + "norm" in gv:
            assert abs(L.prev_norm - gv[pre + "norm"][0]) <= 1e-13
        np.testing.assert_allclose(L.M.ravel(), gv[pre + "M"], rtol=0, atol=1e-13)
        if pre + "Q" in gv:
            np.testing.assert_allclose(L.Q.ravel(), gv[pre + "Q"], rtol=0, atol=1e-13)
        if pre + "X" in gv:
            np.testing.assert_allclose(L.X.ravel(), gv[pre + "X"], rtol=0, atol=1e-13)
        if pre + "P" in gv:
            np.testing.assert_allclose(L.last["P"].ravel(), gv[pre + "P"], rtol=0, atol=1e-13)
            np.testing.assert_allclose(L.last["R"].ravel(), gv[pre + "R"], rtol=0, atol=1e-13)
    assert res["rmmc"][0] == 0.0


def check_orthogonalize_is_qr_factor(o):
    """P^T P = I and C = P^T P~ is upper triangular with a positive diagonal and
    P C = P~: together these fix P as the unique thin-QR factor."""
    for (m, r, seed) in [(40, 7, 1), (64, 64, 2), (200, 17, 3), (5, 1, 4)]:
        Pt = _rng(seed).standard_normal((m, r)) * np.logspace(0, 3, r)[None, :]
        P = o.orthogonalize(Pt)
        assert P.shape == (m, r)
        assert np.linalg.norm(P.T @ P - np.eye(r)) <= 1e-12
        C = P.T @ Pt
        assert np.max(np.abs(np.tril(C, -1))) <= 1e-11 * np.linalg.norm(Pt)
        assert np.all(np.diag(C) > 0)
        assert np.linalg.norm(P @ np.triu(C) - Pt) <= 1e-12 * np.linalg.norm(Pt)


def _cgs2(A):
    """Classical Gram-Schmidt applied twice per column (an independent thin QR)."""
    A = np.array(A, dtype=np.float64)
    m, r = A.shape
    Qm = np.zeros((m, r))
    for j in range(r):
        v = A[:, j].copy()
        for _ in range(2):
            v -= Qm[:, :j] @ (Qm[:, :j].T @ v)
        Qm[:, j] = v / np.linalg.norm(v)
    return Qm


def check_orthogonalize_matches_gram_schmidt(o):
    for (m, r, seed) in [(30, 5, 11), (128, 32, 12), (9, 9, 13)]:
        Pt = _rng(seed).standard_normal((m, r))
        assert np.max(np.abs(o.orthogonalize(Pt) - _cgs2(Pt))) <= 1e-12


def check_column_normalize(o):
    R = _rng(5).standard_normal((50, 6)) * np.array([1e-3, 1, 10, 1e5, 3, 0.5])
    R[:, 4] = 0.0
    Q = o.column_normalize(R)
    norms = np.sqrt(np.sum(Q * Q, axis=0))
    for j in range(6):
        if j == 4:
            assert np.all(Q[:, j] == 0.0)
        else:
            assert abs(norms[j] - 1.0) <= 1e-14
            # same direction: Q_j is a positive multiple of R_j
            c = (Q[:, j] @ R[:, j]) / (R[:, j] @ R[:, j])
            assert c > 0 and np.linalg.norm(Q[:, j] - c * R[:, j]) <= 1e-14


def check_frobenius_norm(o):
    B = _rng(6).standard_normal((13, 7))
    brute = math.sqrt(math.fsum(float(x) * float(x) for x in B.ravel()))
    assert abs(o.frobenius_norm(B) - brute) <= 1e-15 * brute
    # A norm that is not the Frobenius one (max-abs, spectral) fails this.
    assert abs(o.frobenius_norm(np.full((3, 4), 2.0)) - math.sqrt(48.0)) <= 1e-15


def check_rmmc_definition(o):
    assert o.rmmc(3.0, 2.0, 0.0) == 0.5
    assert o.rmmc(1.0, 2.0, 0.0) == 0.5          # decreases count (absolute value)
    assert abs(o.rmmc(5.0, 0.0, 1e-8) - 5e8) <= 1e-6
    assert o.rmmc(2.0, 2.0, 1e-8) == 0.0


def check_rmmc_zero_when_unchanged(o):
    m, n, r = 24, 16, 4
    rng = _rng(7)
    L = o.OracleLayer.from_arrays(rng.standard_normal((m, n)), np.zeros((m, n)),
                                  o.orthogonalize(rng.standard_normal((n, r))))
    o.group_step([L], [rng.standard_normal((m, n))], 0.9, 0.01, 0.5,
                 policy=o.POLICY_NEVER_SYNC)
    res = o.group_step([L], [np.zeros((m, n))], 0.9, 0.01, 0.5)
    assert res["rmmc"] == [0.0] and res["flag"] is False


def _trajectory(o, scale, eps, policy, steps=6, seed=8):
    m, n, r = 20, 12, 3
    rng = _rng(seed)
    M0, X0 = rng.standard_normal((m, n)), rng.standard_normal((m, n))
    Q0 = o.orthogonalize(rng.standard_normal((n, r)))
    grads = [rng.standard_normal((m, n)) for _ in range(steps)]
    L = o.OracleLayer.from_arrays(M0 * scale, X0 * scale, Q0)
    out = []
    for G in grads:
        out.append(o.group_step([L], [G * scale], 0.9, 0.1, 0.2, eps=eps, policy=policy))
    return [x["rmmc"][0] for x in out], [x["flag"] for x in out]


def check_rmmc_scale_invariance(o):
    """Scaling M0, X0 and every G by c = 2^k leaves RMMC unchanged from step 2 on:
    bit-identical with eps = 0 on the local branch (only exact scalings
    occur), and to rounding when sync steps run."""
    base, _ = _trajectory(o, 1.0, 0.0, o.POLICY_NEVER_SYNC)
    for c in (2.0 ** 7, 2.0 ** -5):
        sc, _ = _trajectory(o, c, 0.0, o.POLICY_NEVER_SYNC)
        assert base[1:] == sc[1:]
    base, fb = _trajectory(o, 1.0, 1e-8, o.POLICY_RMMC)
    for c in (2.0 ** 10, 2.0 ** -3):
        sc, fs = _trajectory(o, c, 1e-8, o.POLICY_RMMC)
        assert fb == fs
        # RMMC_c = |n - p| / (p + eps/c): relative change at most about
        # eps |1 - 1/c| / p, and every layer norm p here exceeds 10.
        tol = 1e-12 + 1e-8 * abs(1.0 - 1.0 / c) / 10.0
        for a, b in zip(base[1:], sc[1:]):
            assert abs(a - b) <= tol * abs(a)


def check_power_iteration_converges(o):
    """Repeating PowerIter on a fixed B (Q <- ColumnNormalize(R)) converges to
    the top-r singular subspace of an explicit SVD at rate (s_{r+1}/s_r)^k, and
    ‖B - P R^T‖_F^2 tends to the Eckart-Young value sum_{i>r} s_i^2."""
    m, n, r = 12, 9, 3
    rng = _rng(9)
    U, _ = np.linalg.qr(rng.standard_normal((m, m)))
    V, _ = np.linalg.qr(rng.standard_normal((n, n)))
    s = np.array([10.0, 8.0, 6.0, 3.0, 1.0, 0.5, 0.2, 0.1, 0.05])
    B = U[:, :9] @ np.diag(s) @ V.T
    Q = o.orthogonalize(rng.standard_normal((n, r)))
    errs = []
    for k in range(40):
        _, P, R = o.power_iteration(B, Q)
        Q = o.column_normalize(R)
        errs.append(np.linalg.norm(P - U[:, :r] @ (U[:, :r].T @ P), 2))
    ratio = s[r] / s[r - 1]
    assert errs[-1] <= 1e-6
    # geometric decay at (about) the predicted rate, checked over 10 iterations
    assert errs[25] / errs[15] <= (ratio ** 10) * 5.0
    _, P, R = o.power_iteration(B, Q)
    resid = np.linalg.norm(B - P @ R.T) ** 2
    assert abs(resid - np.sum(s[r:] ** 2)) <= 1e-9 * np.sum(s ** 2)


def check_full_rank_momentum(o):
    """r = m <= n: P P^T = I, so the error-feedback update gives M = mu B exactly."""
    m, n, mu = 6, 10, 0.8
    rng = _rng(10)
    B = rng.standard_normal((m, n))
    Q0 = o.orthogonalize(rng.standard_normal((n, m)))
    out = o.sync_update(B, np.zeros((m, n)), Q0, mu, 0.1)
    assert np.max(np.abs(out["M"] - mu * B)) <= 1e-13 * np.max(np.abs(B))


def check_rank_one_closed_form(o):
    """B = u v^T, r = 1: M = mu B, Q = sign(v^T q0) v/‖v‖ and
    dX = -eta sqrt(m/n) u v^T / (‖u‖ ‖v‖) whatever q0 (m != n)."""
    m, n, mu, eta = 7, 4, 0.9, 0.05
    rng = _rng(11)
    u, v = rng.standard_normal(m), rng.standard_normal(n)
    B = np.outer(u, v)
    X0 = rng.standard_normal((m, n))
    for q0 in (rng.standard_normal((n, 1)), -rng.standard_normal((n, 1))):
        q0 = q0 / np.linalg.norm(q0)
        out = o.sync_update(B, X0, q0, mu, eta)
        assert np.max(np.abs(out["M"] - mu * B)) <= 1e-13 * np.max(np.abs(B))
        sgn = np.sign(v @ q0[:, 0])
        np.testing.assert_allclose(out["Q"][:, 0], sgn * v / np.linalg.norm(v), atol=1e-14)
        dX = -eta * math.sqrt(m / n) * np.outer(u, v) / (np.linalg.norm(u) * np.linalg.norm(v))
        np.testing.assert_allclose(out["X"] - X0, dX, atol=1e-14)


def check_local_branch_closed_form(o):
    m, n = 9, 5
    rng = _rng(12)
    M0, X0, G = (rng.standard_normal((m, n)) for _ in range(3))
    Q0 = o.orthogonalize(rng.standard_normal((n, 2)))
    # prev_norm equal to ||M0 + G|| makes RMMC (about) zero -> local branch
    L = o.OracleLayer.from_arrays(M0, X0, Q0, prev_norm=np.linalg.norm(M0 + G))
    res = o.group_step([L], [G], 0.9, 0.1, 0.5, eta_local=0.25)
    assert res["flag"] is False
    assert np.array_equal(L.M, M0 + G)
    assert np.array_equal(L.X, X0 - 0.25 * G)
    assert np.array_equal(L.Q, Q0)


def check_gate(o):
    assert o.gate([0.1, 0.7, 0.3], 0.5) == (0.7, True)
    assert o.gate([0.5], 0.5) == (0.5, False)                 # tie skips (strict >)
    g, f = o.gate([0.1, float("nan")], 0.5)
    assert math.isnan(g) and f is False                       # NaN skips
    assert o.gate([0.0], 0.5, o.POLICY_ALWAYS_SYNC)[1] is True
    assert o.gate([9.0], 0.5, o.POLICY_NEVER_SYNC)[1] is False
    assert [o.gate([0.0], 0.5, o.POLICY_EVERY_H, step=t, H=3)[1] for t in range(1, 7)] == \
        [False, False, True, False, False, True]


def check_first_step_syncs_and_global_max(o):
    """prev_norm0 = 0 makes step 1 sync; the gate uses the max over layers, so
    one layer with a large RMMC makes every layer take the sync branch."""
    rng = _rng(13)
    mk = lambda m, n, r, pn: o.OracleLayer.from_arrays(
        np.zeros((m, n)), np.zeros((m, n)), o.orthogonalize(rng.standard_normal((n, r))), prev_norm=pn)
    layers = [mk(8, 6, 2, 0.0), mk(5, 7, 2, 0.0)]
    res = o.group_step(layers, [rng.standard_normal((8, 6)), rng.standard_normal((5, 7))], 0.9, 0.1, 0.5)
    assert res["flag"] is True and all(L.last.get("P") is not None for L in layers)
    # step 2: layer 0 barely moves (its RMMC is only the sync step's shrinkage
    # |‖M_1‖ - ‖B_1‖| / ‖B_1‖, well under tau); layer 1 gets G = 2 M, tripling
    # its norm.  The max decides, so layer 0 takes the sync branch as well.
    for L in layers:
        L.last = {}
    G0 = 1e-9 * rng.standard_normal((8, 6))
    G1 = 2.0 * layers[1].M
    res = o.group_step(layers, [G0, G1], 0.9, 0.1, 0.5)
    assert res["rmmc"][0] < 0.5 < res["rmmc"][1]
    assert res["flag"] is True and res["g"] == max(res["rmmc"])
    assert "P" in layers[0].last


def check_policies_match_algorithms(o):
    """ALWAYS_SYNC reproduces Algorithm 1 (sync_update every step); NEVER_SYNC
    is momentum accumulation plus SGD."""
    m, n, r = 10, 8, 3
    rng = _rng(14)
    M0, X0 = rng.standard_normal((m, n)), rng.standard_normal((m, n))
    Q0 = o.orthogonalize(rng.standard_normal((n, r)))
    grads = [rng.standard_normal((m, n)) for _ in range(4)]
    L = o.OracleLayer.from_arrays(M0, X0, Q0)
    M, X, Q = M0.copy(), X0.copy(), Q0.copy()
    for G in grads:
        o.group_step([L], [G], 0.9, 0.05, 1e30, policy=o.POLICY_ALWAYS_SYNC)
        out = o.sync_update(M + G, X, Q, 0.9, 0.05)
        M, X, Q = out["M"], out["X"], out["Q"]
    assert np.array_equal(L.M, M) and np.array_equal(L.X, X) and np.array_equal(L.Q, Q)
    L = o.OracleLayer.from_arrays(M0, X0, Q0)
    for G in grads:
        o.group_step([L], [G], 0.9, 0.05, 0.0, policy=o.POLICY_NEVER_SYNC)
    np.testing.assert_allclose(L.M, M0 + sum(grads), atol=1e-13)
    np.testing.assert_allclose(L.X, X0 - 0.05 * sum(grads), atol=1e-13)


def check_weight_decay_decoupled(o):
    """Decoupled weight decay: X <- (1 - eta lambda) X before either branch's
    update, M and Q untouched.  A local step with G = 0 and a sync step with
    B = 0 only scale X; with any input, turning the decay on moves X by exactly
    (d - 1) X_{t-1} and nothing else."""
    m, n, r, mu, eta, lam = 7, 5, 2, 0.9, 0.05, 0.3
    d = 1.0 - eta * lam
    rng = _rng(15)
    M0, X0 = rng.standard_normal((m, n)), rng.standard_normal((m, n))
    Q0 = o.orthogonalize(rng.standard_normal((n, r)))
    L = o.OracleLayer.from_arrays(M0, X0, Q0, prev_norm=np.linalg.norm(M0))
    res = o.group_step([L], [np.zeros((m, n))], mu, eta, 0.5, weight_decay=lam)
    assert res["flag"] is False and np.array_equal(L.M, M0) and np.array_equal(L.X, d * X0)
    L = o.OracleLayer.from_arrays(np.zeros((m, n)), X0, Q0)
    o.group_step([L], [np.zeros((m, n))], mu, eta, 0.5, policy=o.POLICY_ALWAYS_SYNC, weight_decay=lam)
    assert np.array_equal(L.X, d * X0) and not np.any(L.M)
    G = rng.standard_normal((m, n))
    for policy in (o.POLICY_ALWAYS_SYNC, o.POLICY_NEVER_SYNC):
        A, Bl = o.OracleLayer.from_arrays(M0, X0, Q0), o.OracleLayer.from_arrays(M0, X0, Q0)
        o.group_step([A], [G], mu, eta, 0.5, policy=policy)
        o.group_step([Bl], [G], mu, eta, 0.5, policy=policy, weight_decay=lam)
        assert np.array_equal(A.M, Bl.M) and np.array_equal(A.Q, Bl.Q)
        np.testing.assert_allclose(Bl.X - A.X, (d - 1.0) * X0, rtol=0, atol=1e-14)


def check_sync_update_equivariance(o):
    """Metamorphic pins of the sync update (no formula retyped): for orthogonal
    U (m x m) and V (n x n) and c > 0,
      B -> U B, X -> U X:            P -> U P, R and Q unchanged, M -> U M, X' -> U X'
      B -> B V, X -> X V, Q0 -> V^T Q0:  P unchanged, R -> V^T R, Q -> V^T Q,
                                          M -> M V, X' -> X' V
      B -> c B:                      P, Q and X' unchanged, R -> c R, M -> c M
    (the positive-diagonal QR factor is equivariant under both rotations and
    invariant under positive scaling; column norms are rotation invariant)."""
    rng = _rng(23)
    mu, eta = 0.9, 0.03
    for m, n, r in ((9, 7, 3), (7, 9, 3), (12, 12, 5)):
        B, X = rng.standard_normal((m, n)), rng.standard_normal((m, n))
        Q0 = np.linalg.qr(rng.standard_normal((n, r)))[0]
        U = np.linalg.qr(rng.standard_normal((m, m)))[0]
        V = np.linalg.qr(rng.standard_normal((n, n)))[0]
        base = o.sync_update(B, X, Q0, mu, eta)

        def close(a, b):
            np.testing.assert_allclose(a, b, rtol=0, atol=1e-11 * max(1.0, np.abs(b).max()))

        left = o.sync_update(U @ B, U @ X, Q0, mu, eta)
        close(left["P"], U @ base["P"])
        close(left["R"], base["R"])
        close(left["Q"], base["Q"])
        close(left["M"], U @ base["M"])
        close(left["X"], U @ base["X"])
        right = o.sync_update(B @ V, X @ V, V.T @ Q0, mu, eta)
        close(right["P"], base["P"])
        close(right["R"], V.T @ base["R"])
        close(right["Q"], V.T @ base["Q"])
        close(right["M"], base["M"] @ V)
        close(right["X"], base["X"] @ V)
        scaled = o.sync_update(3.0 * B, X, Q0, mu, eta)
        close(scaled["P"], base["P"])
        close(scaled["Q"], base["Q"])
        close(scaled["R"], 3.0 * base["R"])
        close(scaled["M"], 3.0 * base["M"])
        close(scaled["X"], base["X"])


ALL_CHECKS = [check_golden, check_orthogonalize_is_qr_factor,
              check_orthogonalize_matches_gram_schmidt, check_column_normalize,
              check_frobenius_norm, check_rmmc_definition, check_rmmc_zero_when_unchanged,
              check_rmmc_scale_invariance, check_power_iteration_converges,
              check_full_rank_momentum, check_rank_one_closed_form,
              check_local_branch_closed_form, check_gate,
              check_first_step_syncs_and_global_max, check_policies_match_algorithms,
              check_weight_decay_decoupled, check_sync_update_equivariance]


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda c: c.__name__)
def test_oracle_pin(check):
    check(O)


def test_nonfinite_gradient_takes_local_branch_and_poisons_prev():
    """A NaN in G: RMMC is NaN, NaN > tau is False (local branch), and
    prev_norm still takes the NaN (the norm update is unconditional)."""
    rng = _rng(15)
    L = O.OracleLayer.from_arrays(np.ones((4, 4)), np.zeros((4, 4)),
                                  O.orthogonalize(rng.standard_normal((4, 2))), prev_norm=4.0)
    G = np.zeros((4, 4))
    G[1, 2] = np.nan
    res = O.group_step([L], [G], 0.9, 0.1, 0.5)
    assert math.isnan(res["rmmc"][0]) and res["flag"] is False and math.isnan(L.prev_norm)


# ---------------------------------------------------------------------------
# planted mistakes: each mutant of the oracle must fail at least one pin
# ---------------------------------------------------------------------------
def _mutant(**overrides):
    """A copy of the oracle module whose functions see ``overrides`` in place of
    the originals (the originals are rebound to the copy's namespace)."""
    mod = types.ModuleType("oracle_mutant")
    mod.__dict__.update({k: v for k, v in OC.__dict__.items() if not k.startswith("__")})
    for name, val in list(mod.__dict__.items()):
        if isinstance(val, types.FunctionType) and val.__module__ == OC.__name__:
            mod.__dict__[name] = types.FunctionType(val.__code__, mod.__dict__, name,
                                                    val.__defaults__, val.__closure__)
    mod.__dict__.update(overrides)
    return mod


def _m_no_sign_fix(P_tilde):
    Qf, _ = np.linalg.qr(np.asarray(P_tilde, dtype=np.float64), mode="reduced")
    return Qf


def _m_r_from_ptilde(B, Q_prev):
    B = np.asarray(B, dtype=np.float64)
    Pt = B @ Q_prev
    P = OC.orthogonalize(Pt)
    return Pt, P, B.T @ Pt


def _m_sqrt_n_over_m(B, X, Q_prev, mu, eta, x_decay=1.0):
    B = np.asarray(B, dtype=np.float64)
    m, n = B.shape
    Pt, P, R = OC.power_iteration(B, Q_prev)
    Q = OC.column_normalize(R)
    return dict(M=B - (1 - mu) * (P @ R.T), X=x_decay * X - eta * math.sqrt(n / m) * (P @ Q.T),
                Q=Q, P=P, P_tilde=Pt, R=R)


def _m_mu_instead_of_one_minus_mu(B, X, Q_prev, mu, eta, x_decay=1.0):
    B = np.asarray(B, dtype=np.float64)
    m, n = B.shape
    Pt, P, R = OC.power_iteration(B, Q_prev)
    Q = OC.column_normalize(R)
    return dict(M=B - mu * (P @ R.T), X=x_decay * X - eta * math.sqrt(m / n) * (P @ Q.T),
                Q=Q, P=P, P_tilde=Pt, R=R)


def _m_x_uses_r(B, X, Q_prev, mu, eta, x_decay=1.0):
    B = np.asarray(B, dtype=np.float64)
    m, n = B.shape
    Pt, P, R = OC.power_iteration(B, Q_prev)
    Q = OC.column_normalize(R)
    return dict(M=B - (1 - mu) * (P @ R.T), X=x_decay * X - eta * math.sqrt(m / n) * (P @ R.T),
                Q=Q, P=P, P_tilde=Pt, R=R)


def _m_row_normalize(R):
    R = np.asarray(R, dtype=np.float64)
    return R / np.sqrt(np.sum(R * R, axis=1))[:, None]


def _m_rmmc_no_abs(norm_b, prev_norm, eps):
    return (norm_b - prev_norm) / (prev_norm + eps)


def _m_rmmc_over_current(norm_b, prev_norm, eps):
    return abs(norm_b - prev_norm) / (norm_b + eps)


def _m_maxabs_norm(B):
    return float(np.max(np.abs(np.asarray(B, dtype=np.float64))))


def _m_gate_ge(rmmc_values, tau, policy=0, step=1, H=1):
    g = float(np.max(rmmc_values))
    return g, bool(g >= tau) if policy == 0 else OC.gate(rmmc_values, tau, policy, step, H)[1]


def _m_gate_mean(rmmc_values, tau, policy=0, step=1, H=1):
    g = float(np.mean(rmmc_values))
    return g, bool(g > tau) if policy == 0 else OC.gate(rmmc_values, tau, policy, step, H)[1]


def _m_local_no_g(B, G, X, eta_local, x_decay=1.0):
    return dict(M=np.asarray(B, dtype=np.float64).copy(), X=x_decay * np.asarray(X, dtype=np.float64))


def _m_local_decays(B, G, X, eta_local, x_decay=1.0):
    return dict(M=0.95 * np.asarray(B, dtype=np.float64),
                X=x_decay * np.asarray(X, dtype=np.float64) - eta_local * np.asarray(G, dtype=np.float64))


def _m_weight_decay_on_m(B, X, Q_prev, mu, eta, x_decay=1.0):
    out = OC.sync_update(B, X, Q_prev, mu, eta, x_decay)
    out["M"] = x_decay * out["M"]
    return out


def _m_weight_decay_after_update(B, X, Q_prev, mu, eta, x_decay=1.0):
    out = OC.sync_update(B, X, Q_prev, mu, eta, 1.0)
    out["X"] = x_decay * out["X"]
    return out


MUTANTS = {
    "no_sign_fix": dict(orthogonalize=_m_no_sign_fix),
    "R_from_P_tilde": dict(power_iteration=_m_r_from_ptilde),
    "sqrt_n_over_m": dict(sync_update=_m_sqrt_n_over_m),
    "mu_for_1_minus_mu": dict(sync_update=_m_mu_instead_of_one_minus_mu),
    "X_update_uses_R": dict(sync_update=_m_x_uses_r),
    "row_normalize": dict(column_normalize=_m_row_normalize),
    "rmmc_no_abs": dict(rmmc=_m_rmmc_no_abs),
    "rmmc_over_current": dict(rmmc=_m_rmmc_over_current),
    "maxabs_norm": dict(frobenius_norm=_m_maxabs_norm),
    "gate_ge": dict(gate=_m_gate_ge),
    "gate_mean": dict(gate=_m_gate_mean),
    "local_drops_G": dict(local_update=_m_local_no_g),
    "local_decays_M": dict(local_update=_m_local_decays),
    "weight_decay_on_M": dict(sync_update=_m_weight_decay_on_m),
    "weight_decay_after_update": dict(sync_update=_m_weight_decay_after_update),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name):
    mod = _mutant(**MUTANTS[name])
    failures = 0
    for check in ALL_CHECKS:
        try:
            check(mod)
        except Exception:
            failures += 1
    assert failures >= 1, f"mutant {name} passed every pin"
