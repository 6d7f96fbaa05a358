"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on
the same seeded inputs.  Per step, teacher-forced unless stated: the oracle's
whole step on the exact buffer B = M + G gives the decision and RMMC; its
branch on the fp32 buffer the kernels hold (B rounded once, as the kernel's
addition rounds it) gives the outputs.  Tolerances (rel-Frobenius):

* sync flag identical; every RMMC-policy case asserts its decision margin
            |g - tau| / tau > 1e-4 (1e-2 with bf16 gradients)
* RMMC:     relative 1e-5 (norms of the fp32 buffer; fp64 accumulation)
* fp32 gradients: M, X, P, Q, dM = B - M (the momentum correction
            (1 - mu) P R^T), dX = X_t - X_{t-1}: 1e-5 each, plus for dX the
            fp32 rounding of X itself (4 u ‖X_t‖ / ‖dX‖: X is rounded up to
            three times per step)
* per tile (128 x 64 tiles of dM and dX, the update kernel's tile; 64-row
            panels of P): the largest tile error within TILE_F32 (fp32) or
            2e-2 (bf16).  One wholly wrong tile gives an error near 1 in its
            tile however large the matrix, where the global norm would dilute
            it by the square root of the tile count
* P^T P - I and |‖Q_j‖ - 1|: 1e-5 (absolute, Frobenius / max)
* local branch: M bit-exact against fp32 M + G, X within 1 ulp of fp32 FMA
* bf16 gradients (the path uses two-piece bf16 products, about 2^-16, for
            the power iteration, plain bf16 products for the rank-r update and
            fp32-accurate arithmetic for the second CholQR pass): M, X, P, Q,
            dM, dX within 2e-2, ‖P^T P - I‖_F <= 1e-4; decisions identical
Free-running trajectories check every decision against the free-running
oracle and every step teacher-forced (the oracle restarted from the GPU
state) with the bounds above; the drift between the two free-running states
is bounded only loosely (it is a property of the dynamics, not of the kernels).
"""
import math
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

import oracle as O  # noqa: E402
import paper_2512_13728_amd as cdl  # noqa: E402
import synthetic as S  # noqa: E402
from gpu_util import (TILE_F32, TOL_BF16, TOL_F32, assert_rmmc_close, buffer_f32, check_errors,  # noqa: E402
                      f32, f64, group_step_and_compare, rel, step_and_compare, sync_errors,
                      tile_rel_max)

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cdl.lib()  # fail loudly if the library is missing
    yield


def _state(w, li, r=None, device=DEV):
    M0, X0, Q0 = S.initial_state(w, li, device="cpu", r=r)
    return M0.to(device), X0.to(device), Q0.to(device).contiguous()


def _print(tag, d):
    keys = ["flag_gpu", "rmmc_gpu", "err_M", "err_X", "err_dM", "err_dX", "err_Q", "err_P", "tile_dM",
            "tile_dX", "tile_P", "orth_P", "kappa"]
    print(tag, {k: (f"{d[k]:.3g}" if isinstance(d.get(k), float) else d.get(k)) for k in keys if k in d},
          flush=True)


def _check_step(d, tau, policy, bf16=False):
    assert d["flag_gpu"] == d["flag_oracle"], d
    assert_rmmc_close(d["rmmc_gpu"], d["rmmc_oracle"])
    if policy == O.POLICY_RMMC and math.isfinite(d["rmmc_oracle"]):
        assert abs(d["rmmc_oracle"] - tau) / tau > (1e-2 if bf16 else 1e-4), "decision too close to tau"
    check_errors(d, bf16)


def _check_group(info, errs, tau, policy, bf16=False, tag=""):
    """A group step: identical decision (with its margin under the RMMC gate),
    every layer's RMMC, and the checked layers' errors."""
    assert info["flag_gpu"] == info["flag_oracle"], (tag, info["rmmc_gpu"], info["rmmc_oracle"])
    if policy == O.POLICY_RMMC and math.isfinite(info["rmmc_oracle"]):
        assert abs(info["rmmc_oracle"] - tau) / tau > (1e-2 if bf16 else 1e-4), (tag, "too close to tau")
    assert len(info["per_gpu"]) == len(info["per_oracle"])
    for a, b in zip(info["per_gpu"], info["per_oracle"]):
        assert_rmmc_close(a, b)
    worst = {}
    for i, e in errs.items():
        for k, v in e.items():
            if k.startswith(("err_", "tile_")):
                worst[k] = max(worst.get(k, 0.0), v)
        check_errors(e, bf16)
    print(f"{tag} flag={info['flag_gpu']} g={info['rmmc_gpu']:.4g} worst "
          + " ".join(f"{k}={v:.2e}" for k, v in sorted(worst.items())), flush=True)


# ---------------------------------------------------------------------------
@pytest.mark.parametrize("m,n,gd", [(13, 7, "f32"), (256, 256, "f32"), (300, 1000, "bf16"),
                                    (1000, 333, "f32"), (8192 + 5, 3, "bf16")])
def test_local_branch_exact(m, n, gd):
    """Local branch: M = M + G bit-exact in fp32; X = X - eta_l G within 1 ulp."""
    w = S.small_workload(m, n, 1, grad_dtype=gd)
    M, X, Q = _state(w, 0)
    L = cdl.Layer(m, n, 1, grad_dtype=gd, policy=cdl.POLICY_NEVER_SYNC, eta_local_scale=0.5)
    stream = S.GradientStream(w, 0, device="cpu")
    for t in range(3):
        G = stream.next().to(DEV)
        M32, X32, G32 = M.cpu().numpy().copy(), X.cpu().numpy().copy(), G.float().cpu().numpy()
        rm, flag, _ = L.step(G, M, X, Q, 0.95, 0.01, 1)
        torch.cuda.synchronize()
        assert flag is False
        assert np.array_equal(M.cpu().numpy(), M32 + G32)
        c = np.float32(np.float32(0.01) * 0.5)
        Xref = (X32.astype(np.float64) - np.float64(c) * G32.astype(np.float64)).astype(np.float32)
        ulp = np.abs(X.cpu().numpy().view(np.int32).astype(np.int64) - Xref.view(np.int32).astype(np.int64))
        assert ulp.max() <= 1
        assert np.array_equal(Q.cpu().numpy(), _state(w, 0)[2].cpu().numpy())


def test_rmmc_exactly_zero_and_deterministic():
    """After a local step, G = 0 leaves ‖B‖ unchanged: RMMC is exactly 0.
    Re-running the same inputs gives bit-identical RMMC and state."""
    w = S.small_workload(777, 1234, 8)
    results = []
    for rep in range(2):
        M, X, Q = _state(w, 0)
        L = cdl.Layer(777, 1234, 8, policy=cdl.POLICY_RMMC, tau=0.5)
        stream = S.GradientStream(w, 0, device="cpu")
        rms = []
        for t in range(3):
            G = stream.next().to(DEV)
            rms.append(L.step(G, M, X, Q, 0.95, 0.01, 8)[0])
        rm0, flag0, _ = L.step(torch.zeros_like(G), M, X, Q, 0.95, 0.01, 8)
        torch.cuda.synchronize()
        results.append((rms, M.cpu().numpy(), X.cpu().numpy(), Q.cpu().numpy()))
        assert rm0 == 0.0 and flag0 is False
    assert results[0][0] == results[1][0]
    for a, b in zip(results[0][1:], results[1][1:]):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("m,n,r", [(256, 256, 16), (300, 1000, 37), (1000, 300, 64), (64, 64, 64),
                                   (97, 513, 1), (2048, 768, 192), (513, 640, 130),
                                   # fp32 vector update (r <= 32): ragged column strips of
                                   # four and of two columns per lane, a tall narrow matrix
                                   (97, 515, 5), (130, 259, 20), (8197, 6, 3), (300, 1000, 32),
                                   (257, 333, 48),
                                   # the four-launch path of small layers at its limits:
                                   # m r = 8192, n r = 8192, r = 64 and r = 1
                                   (128, 128, 64), (8192, 7, 1), (2047, 2048, 4), (33, 8192, 1)])
def test_sync_step_teacher_forced(m, n, r):
    w = S.small_workload(m, n, r, k=max(2, r // 2))
    M, X, Q = _state(w, 0)
    L = cdl.Layer(m, n, r, policy=cdl.POLICY_ALWAYS_SYNC)
    stream = S.GradientStream(w, 0, device="cpu")
    for t in range(3):
        G = stream.next().to(DEV)
        d = step_and_compare(L, G, M, X, Q, 0.95, 0.01, r, 0.5, O.POLICY_ALWAYS_SYNC)
        _print(f"sync {m}x{n} r={r} t={t + 1}", d)
        _check_step(d, 0.5, O.POLICY_ALWAYS_SYNC)
    assert not L.rank_deficient()


def test_full_rank_gives_mu_B():
    """r = m <= n: the sync update leaves M = mu B."""
    m, n = 48, 80
    w = S.small_workload(m, n, m)
    M, X, Q = _state(w, 0)
    L = cdl.Layer(m, n, m, policy=cdl.POLICY_ALWAYS_SYNC)
    G = S.GradientStream(w, 0, device="cpu").next().to(DEV)
    B = f64(M) + f64(G)
    L.step(G, M, X, Q, 0.9, 0.01, m)
    torch.cuda.synchronize()
    assert rel(f64(M), f32(0.9) * B) <= 1e-5


def test_zero_buffer_sync_is_defined():
    """B = 0 on a sync step: P~ = 0 (rank deficient), yet M = 0, Q = 0 and X
    unchanged, as in the oracle; the layer reports the rank deficiency."""
    m, n, r = 64, 96, 8
    L = cdl.Layer(m, n, r, policy=cdl.POLICY_ALWAYS_SYNC)
    M = torch.zeros(m, n, device=DEV)
    X = torch.randn(m, n, device=DEV)
    X0 = X.clone()
    Q = torch.zeros(n, r, device=DEV)
    Q[:r, :r] = torch.eye(r, device=DEV)
    G = torch.zeros(m, n, device=DEV)
    L.step(G, M, X, Q, 0.95, 0.01, r)
    torch.cuda.synchronize()
    assert torch.all(M == 0) and torch.all(Q == 0) and torch.equal(X, X0)
    assert L.rank_deficient()


@pytest.mark.parametrize("gd", ["f32", "bf16"])
@pytest.mark.parametrize("m,n,r,k", [(192, 160, 96, 5), (96, 80, 48, 5), (64, 80, 24, 5), (48, 40, 12, 3)])
def test_rank_deficient_buffer_is_completed(gd, m, n, r, k):
    """B of exact rank k < r (only its first k rows are nonzero, in either
    gradient dtype) on a sync step: P~ = B Q has rank k, so r - k pass-0
    Cholesky pivots fall under the floor: in both 64-column blocks of r = 96
    (the blocked factorisation), and in the one-workgroup factorisation of a
    small layer (r = 48: T^-1 by back substitution; r = 24 and 12: T^-1 formed
    in the pivot loop by the identity's columns).
    Like a Householder QR factor, P still has orthonormal columns: the first k
    are unique and match the oracle (as do those of R and Q, and M = mu B),
    the others complete the basis orthogonally to B's column space (so the
    matching columns of R are zero to rounding).  The completion is not
    unique (the oracle's Q_j there is normalised rounding noise), so X is held
    to the unique part plus at most eta sqrt(m/n) per such column.

    R = B^T P lies in B's k-dimensional row space, and so does every column of
    Q after this step (in the oracle too), so a full-rank gradient next still
    meets a rank-k P~.  The completed P makes R = B^T P full rank again in that
    step, and the step after it is a plain full-rank step that matches the
    oracle: no column of Q is lost for good."""
    from gpu_util import device_to_numpy
    gen = torch.Generator().manual_seed(77)
    G = torch.zeros(m, n)
    G[:k] = torch.randn(k, n, generator=gen) * 0.01
    G = G.to(torch.bfloat16 if gd == "bf16" else torch.float32)
    X0 = torch.randn(m, n, generator=gen) * 0.02
    Q0 = torch.linalg.qr(torch.randn(n, r, generator=gen, dtype=torch.float64))[0].float()
    M = torch.zeros(m, n, device=DEV)
    X, Q = X0.to(DEV), Q0.to(DEV).contiguous()
    mu, eta = 0.95, 0.01
    L = cdl.Layer(m, n, r, grad_dtype=gd, policy=cdl.POLICY_ALWAYS_SYNC)
    _, flag, _ = L.step(G.to(DEV), M, X, Q, mu, eta, r)
    torch.cuda.synchronize()
    assert flag and L.rank_deficient()
    Pa, Ra = L.last_factors()
    Pg = device_to_numpy(Pa, (m, r)).astype(np.float64)
    Rg = device_to_numpy(Ra, (n, r)).astype(np.float64)
    Mg, Xg, Qg = f64(M), f64(X), f64(Q)
    for name, a in (("P", Pg), ("R", Rg), ("M", Mg), ("X", Xg), ("Q", Qg)):
        assert np.isfinite(a).all(), name
    B = f64(G.float())
    _, Po, Ro = O.power_iteration(B, f64(Q0))
    Qo = O.column_normalize(Ro)
    tol = 2e-2 if gd == "bf16" else 1e-5
    orth = np.abs(Pg.T @ Pg - np.eye(r)).max()
    print(f"rank-deficient {gd}: P {rel(Pg[:, :k], Po[:, :k]):.3g} R {rel(Rg[:, :k], Ro[:, :k]):.3g} "
          f"Q {rel(Qg[:, :k], Qo[:, :k]):.3g} M {rel(Mg, mu * B):.3g} |P^T P - I| {orth:.3g} "
          f"|R_j|/|R| past the rank {np.linalg.norm(Rg[:, k:]) / np.linalg.norm(Rg):.3g}", flush=True)
    assert rel(Pg[:, :k], Po[:, :k]) <= tol
    assert rel(Rg[:, :k], Ro[:, :k]) <= tol
    assert rel(Qg[:, :k], Qo[:, :k]) <= tol
    assert rel(Mg, mu * B) <= tol
    assert orth <= (1e-4 if gd == "bf16" else 1e-5)
    assert np.linalg.norm(Rg[:, k:]) <= (1e-3 if gd == "bf16" else 1e-5) * np.linalg.norm(Rg)
    c = eta * math.sqrt(m / n)
    X_unique = f64(X0) - c * Po[:, :k] @ Qo[:, :k].T
    extra = np.linalg.norm(Xg - X_unique)
    assert extra <= c * (r - k) * 1.01 + tol * np.linalg.norm(Xg), extra
    sv = np.linalg.svd(Qo, compute_uv=False)
    assert int(np.sum(sv > 1e-8 * sv[0])) == k      # the oracle's Q spans B's row space only
    for t in range(2):
        Gt = (torch.randn(m, n, generator=gen) * 0.01).to(G.dtype).to(DEV)
        if t == 0:
            L.step(Gt, M, X, Q, mu, eta, r)
            torch.cuda.synchronize()
            for name, a in (("M", M), ("X", X), ("Q", Q)):
                assert torch.isfinite(a).all(), name
            P2 = device_to_numpy(L.last_factors()[0], (m, r)).astype(np.float64)
            assert np.abs(P2.T @ P2 - np.eye(r)).max() <= (1e-4 if gd == "bf16" else 1e-5)
            sv = np.linalg.svd(f64(Q), compute_uv=False)
            assert int(np.sum(sv > 1e-8 * sv[0])) == r   # full rank again
        else:
            d = step_and_compare(L, Gt, M, X, Q, mu, eta, r, 0.5, O.POLICY_ALWAYS_SYNC)
            _print(f"two steps after the deficiency {gd}", d)
            assert not L.rank_deficient()
            _check_step(d, 0.5, O.POLICY_ALWAYS_SYNC, bf16=gd == "bf16")


@pytest.mark.parametrize("m,n,r", [(700, 640, 96), (520, 900, 160)])
def test_second_pass_paths_mixed_in_one_launch(m, n, r):
    """Three fp32 layers of one shape step together (one batch, one launch
    per kernel); the middle one's buffer has exact rank 5.  Its pass-0 pivots
    fall under the floor and the completed columns leave P1^T P1 far from the
    identity, so its second CholQR pass takes the blocked factorisation, while
    the other two layers' second pass takes the near-identity factor (their
    Gram matrices are within 2^-10 of I): both paths in the same launches,
    gated per layer, at r = 96 (two whole blocks) and r = 160 (a partial third
    block).  The full-rank layers match the oracle to the fp32 bounds; the
    deficient one has orthonormal P whose unique columns (and those of R and
    Q, and M = mu B) match the oracle, as test_rank_deficient_buffer_is_completed
    checks for one layer alone."""
    from gpu_util import device_to_numpy
    k = 5
    w = S.small_workload(m, n, r, layers=3, stream_id=131)
    Ls = [cdl.Layer(m, n, r, policy=cdl.POLICY_ALWAYS_SYNC) for _ in range(3)]
    Gp = cdl.Group(Ls)
    st = [list(_state(w, i)) for i in range(3)]
    gen = torch.Generator().manual_seed(131)
    Gd = torch.zeros(m, n)
    Gd[:k] = torch.randn(k, n, generator=gen) * 0.01
    st[1][0] = torch.zeros(m, n, device=DEV)
    st[1][2] = torch.linalg.qr(torch.randn(n, r, generator=gen, dtype=torch.float64))[0].float().contiguous().to(DEV)
    streams = [S.GradientStream(w, i, device="cpu") for i in range(3)]
    Gs = [streams[0].next().to(DEV), Gd.to(DEV), streams[2].next().to(DEV)]
    Q1 = f64(st[1][2])
    info, errs = group_step_and_compare(Gp, Ls, Gs, [s[0] for s in st], [s[1] for s in st],
                                        [s[2] for s in st], w.mu, w.eta, r, w.tau, O.POLICY_ALWAYS_SYNC,
                                        check=[0, 2])
    _check_group(info, errs, w.tau, O.POLICY_ALWAYS_SYNC, tag=f"mixed paths {m}x{n} r={r}")
    assert info["flag_gpu"] and Ls[1].rank_deficient()
    assert not Ls[0].rank_deficient() and not Ls[2].rank_deficient()
    Pa, Ra = Ls[1].last_factors()
    Pg = device_to_numpy(Pa, (m, r)).astype(np.float64)
    Rg = device_to_numpy(Ra, (n, r)).astype(np.float64)
    B = f64(Gd)
    _, Po, Ro = O.power_iteration(B, Q1)
    Qo = O.column_normalize(Ro)
    orth = np.abs(Pg.T @ Pg - np.eye(r)).max()
    print(f"deficient layer: P {rel(Pg[:, :k], Po[:, :k]):.3g} R {rel(Rg[:, :k], Ro[:, :k]):.3g} "
          f"|P^T P - I| {orth:.3g}", flush=True)
    assert rel(Pg[:, :k], Po[:, :k]) <= 1e-5
    assert rel(Rg[:, :k], Ro[:, :k]) <= 1e-5
    assert rel(f64(st[1][2])[:, :k], Qo[:, :k]) <= 1e-5
    assert rel(f64(st[1][0]), w.mu * B) <= 1e-5
    assert orth <= 1e-5


@pytest.mark.parametrize("tau,policy", [(0.5, O.POLICY_RMMC), (0.1, O.POLICY_RMMC),
                                        (0.5, O.POLICY_ALWAYS_SYNC)])
def test_single256_trajectory(tau, policy):
    """The 256 x 256, r = 16 workload for 20 steps.  Decisions match the
    free-running oracle at every step; each step also matches a teacher-forced
    oracle step (started from the GPU's state) within the strict bounds."""
    w = S.WORKLOADS["single256"]
    M, X, Q = _state(w, 0)
    L = cdl.Layer(256, 256, 16, policy=policy, tau=tau)
    free = O.OracleLayer.from_arrays(f64(M), f64(X), f64(Q))
    stream = S.GradientStream(w, 0, device="cpu")
    drift = {"M": 0.0, "Q": 0.0}
    syncs = []
    for t in range(w.steps):
        G = stream.next()
        d = step_and_compare(L, G.to(DEV), M, X, Q, w.mu, w.eta, 16, tau, policy)
        _check_step(d, tau, policy)
        res = O.group_step([free], [f64(G)], f32(w.mu), f32(w.eta), tau, policy=policy)
        assert d["flag_gpu"] == res["flag"], (t + 1, d["rmmc_gpu"], res["g"])
        if res["flag"]:
            syncs.append(t + 1)
        drift["M"] = max(drift["M"], rel(f64(M), free.M))
        drift["Q"] = max(drift["Q"], rel(f64(Q), free.Q))
    print(f"tau={tau} policy={policy} syncs={syncs} free-running drift {drift}", flush=True)
    assert drift["M"] <= 1e-4 and drift["Q"] <= 1e-2


def test_group_mixed_shapes_rmmc_gate():
    """A group of layers of different (and ragged) shapes: per-layer RMMC, one
    decision from the max, sync and local steps, against the oracle."""
    shapes = [(256, 384), (384, 256), (100, 300), (256, 384), (640, 64)]
    r = 32
    tau = 0.3
    w = S.Workload("grp", tuple(shapes), r=r, grad_dtype="f32", steps=6, k=8, tau=tau, stream_id=91)
    Ls = [cdl.Layer(m, n, r, tau=tau) for m, n in shapes]
    Gp = cdl.Group(Ls)
    st = [_state(w, i) for i in range(len(shapes))]
    OLs = [O.OracleLayer.from_arrays(f64(s[0]), f64(s[1]), f64(s[2])) for s in st]
    streams = [S.GradientStream(w, i, device="cpu") for i in range(len(shapes))]
    flags = []
    for t in range(w.steps):
        Gs = [s.next() for s in streams]
        g, flag, per, _ = Gp.step([G.to(DEV) for G in Gs], [s[0] for s in st], [s[1] for s in st],
                                  [s[2] for s in st], w.mu, w.eta, r)
        torch.cuda.synchronize()
        res = O.group_step(OLs, [f64(G) for G in Gs], f32(w.mu), f32(w.eta), tau, with_kappa=True)
        flags.append(flag)
        assert flag == res["flag"]
        assert abs(res["g"] - tau) / tau > 1e-4
        for a, b in zip(per, res["rmmc"]):
            assert_rmmc_close(a, b)
        for s, OL in zip(st, OLs):
            assert rel(f64(s[0]), OL.M) <= 1e-5 * (t + 1)
    assert any(flags) and not all(flags)


def test_group_wider_than_one_launch():
    """More layers than one launch takes: 40 of 96 x 160 and 30 of 130 x 70,
    so the sync branch runs the first shape in two chunks (32 + 8 layers per
    launch) and the streaming passes in two launches (48 + 22 layers, the first
    of mixed shapes); sync and local steps against the oracle, every layer
    checked."""
    shapes = [(96, 160)] * 40 + [(130, 70)] * 30
    r = 16
    tau = 0.3
    w = S.Workload("wide", tuple(shapes), r=r, grad_dtype="f32", steps=6, k=4, tau=tau, stream_id=93)
    Ls = [cdl.Layer(m, n, r, tau=tau) for m, n in shapes]
    Gp = cdl.Group(Ls)
    st = [_state(w, i) for i in range(len(shapes))]
    streams = [S.GradientStream(w, i, device="cpu") for i in range(len(shapes))]
    flags = []
    for t in range(w.steps):
        Gs = [s.next().to(DEV) for s in streams]
        info, errs = group_step_and_compare(Gp, Ls, Gs, [s[0] for s in st], [s[1] for s in st],
                                            [s[2] for s in st], w.mu, w.eta, r, tau, O.POLICY_RMMC)
        _check_group(info, errs, tau, O.POLICY_RMMC, tag=f"wide step {t + 1}")
        flags.append(info["flag_gpu"])
    assert any(flags) and not all(flags)


@pytest.mark.parametrize("gd", ["f32", "bf16"])
def test_more_shape_batches_than_streams(gd):
    """Seven shapes of two layers each: the sync branch runs seven batches on
    four streams (the caller's and three of the group's), three streams taking
    two batches each.  Always-sync steps: every layer's M, X, Q against the
    oracle (teacher-forced), and a second group on the same inputs gives
    bit-identical results (the batches share no memory, so how their kernels
    interleave does not matter)."""
    shapes = [(96, 160), (160, 96), (130, 70), (64, 64), (200, 120), (72, 300), (256, 128)]
    shapes = [s for s in shapes for _ in range(2)]
    r = 16
    w = S.Workload("many", tuple(shapes), r=r, grad_dtype=gd, steps=3, k=4, tau=0.3, stream_id=97)
    runs = []
    for rep in range(2):
        Ls = [cdl.Layer(m, n, r, grad_dtype=gd, policy=cdl.POLICY_ALWAYS_SYNC) for m, n in shapes]
        Gp = cdl.Group(Ls)
        st = [_state(w, i) for i in range(len(shapes))]
        streams = [S.GradientStream(w, i, device="cpu") for i in range(len(shapes))]
        for t in range(w.steps):
            Gs = [s.next().to(DEV) for s in streams]
            args = (Gp, Ls, Gs, [s[0] for s in st], [s[1] for s in st], [s[2] for s in st], w.mu, w.eta, r)
            if rep == 0:
                info, errs = group_step_and_compare(*args, 0.3, O.POLICY_ALWAYS_SYNC)
                _check_group(info, errs, 0.3, O.POLICY_ALWAYS_SYNC, bf16=gd == "bf16",
                             tag=f"{gd} seven batches step {t + 1}")
                assert info["flag_gpu"]
            else:
                _, flag, _, _ = Gp.step(*args[2:])
                torch.cuda.synchronize()
                assert flag
        runs.append([f64(t) for s in st for t in s])
        print(f"{gd} run {rep + 1}: 7 shape batches, {w.steps} sync steps", flush=True)
    for a, b in zip(*runs):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("policy", [O.POLICY_RMMC, O.POLICY_ALWAYS_SYNC])
def test_bf16_fused_buffer_pass_group(policy):
    """Five shapes of two bf16-gradient layers at r = 288.  On a step that
    syncs for certain (every step of the fixed policy; under the RMMC gate the
    first one, where every layer starts from prev_norm = 0) each shape batch
    forms its B inside P~ = B Q on its own stream and the gate adds those
    passes' partial sums; the RMMC gate's later steps take the plain buffer
    pass, so the RMMC statistic mixes both kinds of partial sums.  Every
    layer's RMMC and the decision against the oracle at every step, all
    layers' outputs teacher-forced, and a rerun bit-identical."""
    shapes = [(300, 400), (400, 300), (288, 1030), (700, 320), (320, 320)]
    shapes = [s for s in shapes for _ in range(2)]
    r = 288
    w = S.Workload("fused", tuple(shapes), r=r, grad_dtype="bf16", steps=4, k=8, tau=0.3, stream_id=41)
    pol = cdl.POLICY_RMMC if policy == O.POLICY_RMMC else cdl.POLICY_ALWAYS_SYNC
    runs = []
    for rep in range(2):
        Ls = [cdl.Layer(m, n, r, grad_dtype="bf16", policy=pol, tau=0.3) for m, n in shapes]
        Gp = cdl.Group(Ls)
        st = [_state(w, i) for i in range(len(shapes))]
        streams = [S.GradientStream(w, i, device="cpu") for i in range(len(shapes))]
        flags = []
        for t in range(w.steps):
            Gs = [s.next().to(DEV) for s in streams]
            args = (Gp, Ls, Gs, [s[0] for s in st], [s[1] for s in st], [s[2] for s in st], w.mu, w.eta, r)
            if rep == 0:
                info, errs = group_step_and_compare(*args, 0.3, policy)
                _check_group(info, errs, 0.3, policy, bf16=True, tag=f"fused step {t + 1}")
                flags.append(info["flag_gpu"])
            else:
                _, flag, _, _ = Gp.step(*args[2:])
                torch.cuda.synchronize()
                flags.append(flag)
        runs.append((flags, [f64(t) for s in st for t in s]))
        print(f"run {rep + 1}: decisions {flags}", flush=True)
    assert runs[0][0] == runs[1][0] and runs[0][0][0]
    for a, b in zip(runs[0][1], runs[1][1]):
        assert np.array_equal(a, b)


@pytest.mark.parametrize("policy", [O.POLICY_RMMC, O.POLICY_ALWAYS_SYNC])
@pytest.mark.parametrize("m,n,r", [(512, 1536, 64), (2048, 512, 256), (300, 700, 37), (128, 256, 32),
                                   # 256 < r <= 512: a predicted or fixed sync forms B inside
                                   # P~ = B Q (one workgroup per 128-row band and K slice), with
                                   # ragged bands, an odd rank (scalar loads of Q), a row length
                                   # that is not a multiple of four (scalar loads of M and G), and
                                   # the full 512-wide tile over two K slices
                                   (300, 1000, 300), (257, 700, 257), (1030, 2051, 500), (2048, 2048, 512)])
def test_bf16_gradient_steps(m, n, r, policy):
    """Three steps of one bf16-gradient layer against the oracle (teacher-forced);
    under the RMMC policy step 1 syncs and the later ones follow the gate."""
    gd = "bf16"
    w = S.small_workload(m, n, r, grad_dtype=gd, k=16)
    M, X, Q = _state(w, 0)
    L = cdl.Layer(m, n, r, grad_dtype=gd, policy=policy, tau=0.5)
    stream = S.GradientStream(w, 0, device="cpu")
    for t in range(3):
        G = stream.next().to(DEV)
        d = step_and_compare(L, G, M, X, Q, 0.95, 0.01, r, 0.5, policy)
        _print(f"bf16 {policy} t={t + 1}", d)
        _check_step(d, 0.5, policy, bf16=True)


@pytest.mark.parametrize("m,n,r,gd", [(256, 384, 32, "f32"), (300, 1000, 37, "bf16"),
                                      (2048, 512, 64, "bf16")])
def test_sync_after_skip_reverses_speculation(m, n, r, gd):
    """Under the RMMC gate a skip step makes the next step's buffer pass apply
    the skip-branch X update speculatively; a gradient spike then forces a
    sync, whose X update must first take the speculative change back.
    Decisions [sync, skip, sync, skip]; every step against the oracle."""
    w = S.small_workload(m, n, r, grad_dtype=gd, k=8)
    M, X, Q = _state(w, 0)
    tau = 0.5
    L = cdl.Layer(m, n, r, grad_dtype=gd, policy=cdl.POLICY_RMMC, tau=tau)
    stream = S.GradientStream(w, 0, device="cpu")
    flags = []
    for t in range(4):
        G = stream.next()
        if t == 2:
            G = (G.float() * 40.0).to(G.dtype)   # spike: RMMC far above tau
        d = step_and_compare(L, G.to(DEV), M, X, Q, 0.95, 0.01, r, tau, O.POLICY_RMMC)
        _print(f"spike {gd} t={t + 1}", d)
        _check_step(d, tau, O.POLICY_RMMC, bf16=gd == "bf16")
        flags.append(d["flag_gpu"])
    assert flags == [True, False, True, False]


@pytest.mark.parametrize("m,n,r,gd", [(256, 384, 32, "f32"), (300, 1000, 37, "bf16")])
def test_weight_decay_every_branch(m, n, r, gd):
    """Decoupled weight decay (lambda = 0.1) through every X-writing path:
    a sync step, the stand-alone skip update, the fused speculative skip
    update, and its reversal inside a sync step.  Decisions [sync, skip,
    sync, skip], every step against the oracle with the same decay."""
    w = S.small_workload(m, n, r, grad_dtype=gd, k=8)
    M, X, Q = _state(w, 0)
    tau, lam = 0.5, 0.1
    L = cdl.Layer(m, n, r, grad_dtype=gd, policy=cdl.POLICY_RMMC, tau=tau, weight_decay=lam)
    stream = S.GradientStream(w, 0, device="cpu")
    flags = []
    for t in range(4):
        G = stream.next()
        if t == 2:
            G = (G.float() * 40.0).to(G.dtype)
        d = step_and_compare(L, G.to(DEV), M, X, Q, 0.95, 0.01, r, tau, O.POLICY_RMMC,
                             weight_decay=lam)
        _print(f"decay {gd} t={t + 1}", d)
        _check_step(d, tau, O.POLICY_RMMC, bf16=gd == "bf16")
        flags.append(d["flag_gpu"])
    assert flags == [True, False, True, False]


@pytest.mark.parametrize("gd", ["f32", "bf16"])
def test_local_scale_and_eps_through_every_x_path(gd):
    """eta_local = 0.5 eta, eps = 1e-3 and weight decay 0.05 through
    [sync, skip, skip, sync, skip, skip]: the stand-alone skip update (after a
    sync the branch is predicted sync), the fused speculative skip update kept
    (a skip after a skip), its reversal when a spike (G x 40) makes the
    predicted skip a sync, and both again.  Every step against the oracle
    with the same eps, eta_local and decay."""
    m, n, r = 300, 200, 24
    w = S.small_workload(m, n, r, grad_dtype=gd, k=8)
    M, X, Q = _state(w, 0)
    tau, eps, scale, lam = 0.5, 1e-3, 0.5, 0.05
    L = cdl.Layer(m, n, r, grad_dtype=gd, policy=cdl.POLICY_RMMC, tau=tau, eps=eps,
                  eta_local_scale=scale, weight_decay=lam)
    stream = S.GradientStream(w, 0, device="cpu")
    flags = []
    for t in range(6):
        G = stream.next()
        if t == 3:
            G = (G.float() * 40.0).to(G.dtype)
        d = step_and_compare(L, G.to(DEV), M, X, Q, 0.95, 0.01, r, tau, O.POLICY_RMMC, eps=eps,
                             eta_local_scale=scale, weight_decay=lam)
        _print(f"eta_local x0.5, eps 1e-3, {gd} t={t + 1}", d)
        _check_step(d, tau, O.POLICY_RMMC, bf16=gd == "bf16")
        flags.append(d["flag_gpu"])
    assert flags == [True, False, False, True, False, False]


@pytest.mark.parametrize("gd", ["f32", "bf16"])
def test_eta_local_zero_with_weight_decay(gd):
    """eta_local = 0 (eta_local_scale = 0) with weight decay 0.1 through
    [sync, skip, skip, sync]: after the first skip the buffer pass applies the
    skip branch speculatively, which with eta_local = 0 is the decay alone;
    the spike's sync update must then leave X with that one decay and must
    not decay it again (nor read G).  Every step against the oracle."""
    m, n, r = 300, 500, 24
    w = S.small_workload(m, n, r, grad_dtype=gd, k=8, stream_id=71)
    M, X, Q = _state(w, 0)
    tau, lam = 0.5, 0.1
    L = cdl.Layer(m, n, r, grad_dtype=gd, policy=cdl.POLICY_RMMC, tau=tau, eta_local_scale=0.0,
                  weight_decay=lam)
    stream = S.GradientStream(w, 0, device="cpu")
    flags = []
    for t in range(4):
        G = stream.next()
        if t == 3:
            G = (G.float() * 40.0).to(G.dtype)
        d = step_and_compare(L, G.to(DEV), M, X, Q, 0.95, 0.01, r, tau, O.POLICY_RMMC,
                             eta_local_scale=0.0, weight_decay=lam)
        _print(f"eta_local = 0, decay {lam}, {gd} t={t + 1}", d)
        _check_step(d, tau, O.POLICY_RMMC, bf16=gd == "bf16")
        flags.append(d["flag_gpu"])
    assert flags == [True, False, False, True]


@pytest.mark.parametrize("H", [3, 4])
@pytest.mark.parametrize("gd", ["f32", "bf16"])
def test_every_h_policy_matches_oracle(gd, H):
    """Scheduled Sync Dion (Sec. 4.3): a sync on every H-th step, fixed in
    advance.  The library enqueues the branch before the gate's readback and
    fuses the skip update into the buffer pass on the steps it knows are
    local.  Three layers of two shapes (one group), 2H + 2 steps with weight
    decay 0.05: every step's decision, every layer's RMMC and every layer's
    M, X, Q (and P on sync steps) against the oracle's POLICY_EVERY_H step,
    teacher-forced."""
    shapes = [(256, 384), (320, 200), (256, 384)]
    r = 24
    w = S.Workload(f"everyh{H}", tuple(shapes), r=r, grad_dtype=gd, steps=2 * H + 2, k=8, tau=0.5,
                   stream_id=73)
    lam = 0.05
    Ls = [cdl.Layer(m, n, r, grad_dtype=gd, policy=cdl.POLICY_EVERY_H, H=H, weight_decay=lam)
          for m, n in shapes]
    Gp = cdl.Group(Ls)
    st = [_state(w, i) for i in range(len(shapes))]
    streams = [S.GradientStream(w, i, device="cpu") for i in range(len(shapes))]
    flags = []
    for t in range(w.steps):
        Gs = [s.next().to(DEV) for s in streams]
        info, errs = group_step_and_compare(Gp, Ls, Gs, [s[0] for s in st], [s[1] for s in st],
                                            [s[2] for s in st], w.mu, w.eta, r, 0.5, O.POLICY_EVERY_H,
                                            H=H, weight_decay=lam)
        _check_group(info, errs, 0.5, O.POLICY_EVERY_H, bf16=gd == "bf16", tag=f"every H={H} {gd} step {t + 1}")
        flags.append(info["flag_gpu"])
    assert flags == [(t + 1) % H == 0 for t in range(w.steps)]


def test_packed_pointers_match_lists():
    """Group.step with pointer arrays marshalled once (Group.pack) gives the
    bit-identical result of passing the tensor lists."""
    shapes = [(256, 384), (384, 256), (100, 300)]
    r = 16
    w = S.Workload("pack", tuple(shapes), r=r, grad_dtype="f32", steps=3, k=8, tau=0.3, stream_id=92)
    outs = []
    for packed in (False, True):
        Ls = [cdl.Layer(m, n, r, tau=0.3) for m, n in shapes]
        Gp = cdl.Group(Ls)
        st = [_state(w, i) for i in range(len(shapes))]
        M, X, Q = [s[0] for s in st], [s[1] for s in st], [s[2] for s in st]
        args = (Gp.pack(M), Gp.pack(X), Gp.pack(Q)) if packed else (M, X, Q)
        streams = [S.GradientStream(w, i, device="cpu") for i in range(len(shapes))]
        res = []
        for t in range(w.steps):
            G = [s.next().to(DEV) for s in streams]
            res.append(Gp.step(Gp.pack(G) if packed else G, *args, w.mu, w.eta, r)[:2])
        torch.cuda.synchronize()
        outs.append((res, [f64(t) for t in M + X + Q]))
    assert outs[0][0] == outs[1][0]
    for a, b in zip(outs[0][1], outs[1][1]):
        assert np.array_equal(a, b)
    with pytest.raises(ValueError):
        Gp.pack(M[:1])


def test_kernel_timing_brackets_only_the_named_kinds():
    """Timing restricted to named kernel kinds records only those kinds, with
    the launch counts of the unrestricted run; timing changes no result; an
    unknown kind name is refused."""
    m, n, r = 256, 384, 16
    w = S.small_workload(m, n, r)
    runs = []
    for kinds in (None, "pick"):
        L = cdl.Layer(m, n, r)
        Gp = cdl.Group([L])
        M, X, Q = _state(w, 0)
        stream = S.GradientStream(w, 0, device="cpu")
        if kinds == "pick":
            upd = [k for k in runs[0][0] if k in ("update_f32", "update_bf16", "small_update")]
            assert len(upd) == 1
            kinds = ["gate", upd[0]]
        Gp.set_timing(True, kinds)
        flags = [Gp.step([stream.next().to(DEV)], [M], [X], [Q], w.mu, w.eta, r)[1] for _ in range(3)]
        kt = Gp.kernel_times()
        Gp.set_timing(False)
        torch.cuda.synchronize()
        runs.append((kt, flags, [f64(t) for t in (M, X, Q)]))
        if kinds is not None:
            with pytest.raises(cdl.CurvaDionError):
                Gp.set_timing(True, ["no_such_kind"])
    (k_all, f_all, s_all), (k_sel, f_sel, s_sel) = runs
    assert f_all == f_sel and f_all[0]
    assert set(k_sel) == {"gate", [k for k in k_all if k in ("update_f32", "update_bf16", "small_update")][0]}
    for k, v in k_sel.items():
        assert v["launches"] == k_all[k]["launches"] and v["total_ms"] > 0
    assert len(k_all) > 5 and k_all["gate"]["launches"] == 3
    for a, b in zip(s_all, s_sel):
        assert np.array_equal(a, b)


def test_full_timing_runs_batches_serially_with_identical_results():
    """With every kernel kind timed, the shape batches of the sync branch run
    one after another on the caller's stream; the results are bit-identical
    to the untimed (concurrent) schedule, and the per-kind table covers the
    sync-branch kernels of every batch."""
    shapes = [(256, 384), (384, 256), (100, 300)]
    r = 16
    w = S.Workload("timing", tuple(shapes), r=r, grad_dtype="f32", steps=3, k=8, tau=0.3, stream_id=93)
    outs = []
    for timed in (False, True):
        Gp = cdl.Group([cdl.Layer(m, n, r, tau=0.3) for m, n in shapes])
        st = [_state(w, i) for i in range(len(shapes))]
        M, X, Q = [t[0] for t in st], [t[1] for t in st], [t[2] for t in st]
        streams = [S.GradientStream(w, i, device="cpu") for i in range(len(shapes))]
        if timed:
            Gp.set_timing(True)
        res = [Gp.step([s.next().to(DEV) for s in streams], M, X, Q, w.mu, w.eta, r)[:2]
               for _ in range(w.steps)]
        kt = Gp.kernel_times() if timed else None
        Gp.set_timing(False)
        torch.cuda.synchronize()
        outs.append((res, [f64(t) for t in M + X + Q], kt))
    assert outs[0][0] == outs[1][0] and outs[0][0][0][1]
    for a, b in zip(outs[0][1], outs[1][1]):
        assert np.array_equal(a, b)
    kt = outs[1][2]
    n_sync = sum(f for _, f in outs[0][0])
    # one update launch per shape batch and sync step (these small layers
    # take the four-launch path: P~ = BQ, CholQR2, R = B^T P, update)
    assert kt["small_update"]["launches"] == len(shapes) * n_sync
    assert kt["small_cholqr"]["launches"] == len(shapes) * n_sync


def test_wrong_operands_are_refused_before_any_work():
    """A transposed, mistyped or wrongly-sized operand raises ValueError in the
    binding; the layer's state (prev_norm, step counter) and every buffer stay
    as they were, and a packed array is re-checked for a new rank."""
    m, n, r = 96, 64, 8
    w = S.small_workload(m, n, r)
    L = cdl.Layer(m, n, r)
    M, X, Q = _state(w, 0)
    G = S.GradientStream(w, 0, device="cpu").next().to(DEV)
    before = [t.clone() for t in (M, X, Q)]
    bad = [dict(M=M.t()), dict(X=X.double()), dict(G=G.bfloat16()), dict(Q=Q[:, : r // 2]),
           dict(G=G.cpu())]
    for kw in bad:
        args = dict(G=G, M=M, X=X, Q=Q)
        args.update(kw)
        with pytest.raises(ValueError):
            L.step(args["G"], args["M"], args["X"], args["Q"], 0.95, 0.01, r)
    torch.cuda.synchronize()
    assert L.get_state() == (0.0, 0)
    for a, b in zip(before, (M, X, Q)):
        assert torch.equal(a, b)
    Gp = cdl.Group([L])
    pQ = Gp.pack([Q])
    Gp.step([G], [M], [X], pQ, 0.95, 0.01, r)
    with pytest.raises(ValueError, match="shape"):
        Gp.step([G], [M], [X], pQ, 0.95, 0.01, r // 2)     # Q is n x r, not n x r/2
    with pytest.raises(ValueError, match="shape"):
        Gp.pack([M.t()], "M")                              # checked when packed with a role
    with pytest.raises(ValueError, match="float32"):
        Gp.pack([X.double()], "X")
    torch.cuda.synchronize()
    assert L.get_state()[1] == 1


@pytest.mark.parametrize("gd", ["f32", "bf16"])
def test_plain_c_client_matches_binding_and_oracle(gd, tmp_path):
    """The C99 client (tests/c/cd_c_step.c: the header, the HIP runtime's C
    API and the library, nothing else) steps one layer three times in its own
    process: its M, X, Q are bit-identical to the Python binding's on the same
    inputs, and its decisions and RMMC values match the float64 oracle run
    free from the same start (the first step syncs, as prev_norm starts at 0)."""
    import subprocess
    from paper_2512_13728_amd import build
    exe = build.C_CLIENT
    if not os.path.exists(exe):
        pytest.skip("C client not built (build() compiles it)")
    m, n, r, steps, tau, mu, eta = 96, 160, 8, 3, 0.3, 0.95, 0.01
    w = S.small_workload(m, n, r, grad_dtype=gd, tau=tau, stream_id=31)
    M0, X0, Q0 = S.initial_state(w, 0)
    stream = S.GradientStream(w, 0)
    Gs = [stream.next() for _ in range(steps)]
    M0.numpy().tofile(tmp_path / "M0.bin")
    X0.numpy().tofile(tmp_path / "X0.bin")
    Q0.numpy().tofile(tmp_path / "Q0.bin")
    for t, G in enumerate(Gs):
        (G.view(torch.int16) if gd == "bf16" else G).numpy().tofile(tmp_path / f"G{t}.bin")
    print(f"C client {gd}: {m}x{n} r={r}, {steps} steps", flush=True)
    out = subprocess.run([exe, "run", str(tmp_path), str(m), str(n), str(r), str(steps), gd,
                          str(cdl.POLICY_RMMC), repr(tau), repr(mu), repr(eta)],
                         capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    rows = [ln.split() for ln in (tmp_path / "steps.txt").read_text().splitlines()]
    c_rmmc = [float(a) for a, _, _ in rows]
    c_flag = [b == "1" for _, b, _ in rows]
    cM = np.fromfile(tmp_path / "M.bin", dtype=np.float32).reshape(m, n)
    cX = np.fromfile(tmp_path / "X.bin", dtype=np.float32).reshape(m, n)
    cQ = np.fromfile(tmp_path / "Q.bin", dtype=np.float32).reshape(n, r)
    # the same steps through the Python binding
    L = cdl.Layer(m, n, r, grad_dtype=gd, tau=tau)
    M, X, Q = M0.to(DEV), X0.to(DEV), Q0.to(DEV).contiguous()
    py = [L.step(G.to(DEV), M, X, Q, mu, eta, r)[:2] for G in Gs]
    torch.cuda.synchronize()
    assert [p[0] for p in py] == c_rmmc and [p[1] for p in py] == c_flag
    assert np.array_equal(M.cpu().numpy(), cM) and np.array_equal(X.cpu().numpy(), cX)
    assert np.array_equal(Q.cpu().numpy(), cQ)
    # the free-running oracle from the same start
    OL = O.OracleLayer.from_arrays(f64(M0), f64(X0), f64(Q0))
    for t, G in enumerate(Gs):
        res = O.group_step([OL], [f64(G)], f32(mu), f32(eta), tau)
        assert res["flag"] == c_flag[t], t
        if gd == "f32" or t == 0:
            assert_rmmc_close(c_rmmc[t], res["g"])
        else:
            # free-running bf16: after a sync step the path's M differs from the
            # oracle's by about 1e-4 relative (plain bf16 rank-r update), which
            # moves the next ||B|| and RMMC by a few 1e-5
            assert abs(c_rmmc[t] - res["g"]) <= 1e-3 * abs(res["g"]), (t, c_rmmc[t], res["g"])
        if t > 0:
            assert abs(res["g"] - tau) / tau > 1e-2, "decision too close to tau"
    assert c_flag[0]
    tol = 2e-2 if gd == "bf16" else 1e-4
    assert rel(cM.astype(np.float64), OL.M) <= tol
    assert rel(cX.astype(np.float64), OL.X) <= tol


def test_state_roundtrip_and_every_h_policy():
    m, n, r = 64, 64, 4
    L = cdl.Layer(m, n, r, policy=cdl.POLICY_EVERY_H, H=3)
    w = S.small_workload(m, n, r)
    M, X, Q = _state(w, 0)
    stream = S.GradientStream(w, 0, device="cpu")
    flags = [L.step(stream.next().to(DEV), M, X, Q, 0.95, 0.01, r)[1] for _ in range(6)]
    assert flags == [False, False, True, False, False, True]
    p, s = L.get_state()
    assert s == 6 and p > 0
    L.set_state(123.0, 41)
    assert L.get_state() == (123.0, 41)


def test_nonfinite_gradient_takes_the_local_branch():
    """A NaN (and an Inf) in G: ‖B‖ is not finite, so RMMC is NaN, the gate's
    NaN > tau is false and the local branch runs (the literal IEEE reading of
    Alg. 2); the step reports CD_ENONFINITE, prev_norm becomes NaN and the next
    steps stay local.  In a group the NaN of one layer makes the maximum NaN,
    so every layer takes the local branch; the finite layer's outputs still
    match the oracle exactly as a local step."""
    m, n, r = 200, 300, 8
    w = S.Workload("nan", ((m, n), (m, n)), r=r, grad_dtype="f32", steps=3, k=4, tau=0.5, stream_id=95)
    st = [_state(w, i) for i in range(2)]
    OLs = [O.OracleLayer.from_arrays(f64(s[0]), f64(s[1]), f64(s[2])) for s in st]
    Ls = [cdl.Layer(m, n, r, tau=0.5) for _ in range(2)]
    Gp = cdl.Group(Ls)
    streams = [S.GradientStream(w, i, device="cpu") for i in range(2)]
    for t in range(3):
        Gs = [s.next() for s in streams]
        if t >= 1:
            Gs[1][3, 5] = float("nan")
            Gs[1][7, 11] = float("inf")
        Q0 = [s[2].clone() for s in st]
        X0 = [f64(s[1]) for s in st]
        g, flag, per, status = Gp.step([G.to(DEV) for G in Gs], [s[0] for s in st], [s[1] for s in st],
                                       [s[2] for s in st], w.mu, w.eta, r)
        torch.cuda.synchronize()
        res = O.group_step(OLs, [f64(G) for G in Gs], f32(w.mu), f32(w.eta), 0.5)
        assert flag == res["flag"]
        if t == 0:
            assert flag and status == cdl.CD_OK
            for s, OL in zip(st, OLs):
                OL.M, OL.X, OL.Q = f64(s[0]), f64(s[1]), f64(s[2])
            continue
        assert not flag and status == cdl.CD_ENONFINITE
        assert math.isnan(g) and math.isnan(per[1]) and math.isfinite(per[0])
        assert_rmmc_close(per[0], res["rmmc"][0])
        for i in range(2):
            assert torch.equal(st[i][2], Q0[i])                      # Q untouched
            Mg, Xg = f64(st[i][0]), f64(st[i][1])
            # NaN / Inf positions propagate exactly as in the oracle
            assert np.array_equal(np.isnan(Mg), np.isnan(OLs[i].M))
            assert np.array_equal(np.isnan(Xg), np.isnan(OLs[i].X))
            assert np.array_equal(np.isinf(Xg), np.isinf(OLs[i].X))
            fin = np.isfinite(OLs[i].M)
            assert rel(Mg[fin], OLs[i].M[fin]) <= 1e-6
            finx = np.isfinite(OLs[i].X)
            scale = np.max(np.abs(X0[i][np.isfinite(X0[i])]))
            assert np.max(np.abs(Xg[finx] - OLs[i].X[finx])) <= 1e-6 * scale
            OLs[i].M, OLs[i].X = Mg, Xg
    p, _ = Ls[1].get_state()
    assert math.isnan(p)
    assert math.isfinite(Ls[0].get_state()[0])


def _random_cases(count, seed):
    rng = np.random.default_rng(seed)
    cases = []
    for _ in range(count):
        m, n = (int(x) for x in rng.integers(1, 700, size=2))
        r = int(rng.integers(1, min(m, n, 96) + 1))
        cases.append((m, n, r, "bf16" if rng.random() < 0.4 else "f32"))
    # the degenerate corners: one row, one column, r = min(m, n)
    cases += [(1, 257, 1, "f32"), (333, 1, 1, "bf16"), (40, 40, 40, "f32"), (65, 129, 65, "f32")]
    return cases


@pytest.mark.parametrize("m,n,r,gd", _random_cases(14, 2026))
def test_random_shapes_sync_then_skip(m, n, r, gd):
    """Seeded random shapes (every tile size hits a ragged tail somewhere):
    an always-sync step, then two RMMC-gated steps, teacher-forced against
    the oracle with the bounds of this module."""
    w = S.small_workload(m, n, r, grad_dtype=gd, k=3, stream_id=97)
    M, X, Q = _state(w, 0)
    bf = gd == "bf16"
    stream = S.GradientStream(w, 0, device="cpu")
    L = cdl.Layer(m, n, r, grad_dtype=gd, policy=cdl.POLICY_ALWAYS_SYNC)
    d = step_and_compare(L, stream.next().to(DEV), M, X, Q, 0.95, 0.01, r, 0.5, O.POLICY_ALWAYS_SYNC)
    _print(f"random {m}x{n} r={r} {gd} sync", d)
    _check_step(d, 0.5, O.POLICY_ALWAYS_SYNC, bf16=bf)
    # the same state under the RMMC gate (a fresh layer: prev_norm = 0 syncs
    # first, then the statistic decides)
    L2 = cdl.Layer(m, n, r, grad_dtype=gd, policy=cdl.POLICY_RMMC, tau=0.5)
    for t in range(2):
        d = step_and_compare(L2, stream.next().to(DEV), M, X, Q, 0.95, 0.01, r, 0.5, O.POLICY_RMMC)
        _print(f"random {m}x{n} r={r} {gd} rmmc t={t + 1}", d)
        if math.isfinite(d["rmmc_oracle"]) and abs(d["rmmc_oracle"] - 0.5) / 0.5 <= (1e-2 if bf else 1e-4):
            continue   # too close to tau to compare decisions
        _check_step(d, 0.5, O.POLICY_RMMC, bf16=bf)


# --- asynchronous steps -------------------------------------------------------
def _spiky_grads(w, L, steps, spikes=(5,), scale=40.0):
    streams = [S.GradientStream(w, i, device="cpu") for i in range(L)]
    out = []
    for t in range(steps):
        gs = [s.next() for s in streams]
        if t in spikes:
            gs = [(g.float() * scale).to(g.dtype) for g in gs]
        out.append([g.to(DEV) for g in gs])
    return out


@pytest.mark.parametrize("mode", ["end", "each", "alternate"])
@pytest.mark.parametrize("gd", ["f32", "bf16"])
def test_async_group_steps_bit_identical_to_blocking(gd, mode):
    """Asynchronous group steps (no host output: both branches enqueued,
    every kernel predicated on the gate's decision in device memory, the
    speculative skip update taken from the device's prediction) against
    blocking steps over the same inputs: a group of three shapes (three units
    on three streams), the RMMC gate with a spike (G x 40) at step 6 after
    skips, so the run has syncs, skips, fused skips and a reversed
    speculation; weight decay on.  `mode`: every step asynchronous with one
    last-result read at the end; a last-result read after each asynchronous
    step (its outcome equals the blocking step's); asynchronous and blocking
    steps alternating.  The final M, X, Q are bit-identical in every mode."""
    shapes = [(256, 384), (384, 256), (130, 70), (256, 384)]
    r, tau, steps = 24, 0.5, 10
    w = S.Workload("async", tuple(shapes), r=r, grad_dtype=gd, steps=steps, k=6, tau=tau, stream_id=81)
    grads = _spiky_grads(w, len(shapes), steps)
    runs = []
    for asyn in (False, True):
        Ls = [cdl.Layer(m, n, r, grad_dtype=gd, tau=tau, weight_decay=0.05) for m, n in shapes]
        Gp = cdl.Group(Ls)
        st = [_state(w, i) for i in range(len(shapes))]
        M, X, Q = ([s[k] for s in st] for k in range(3))
        res = []
        for t in range(steps):
            blocking = (not asyn) or (mode == "alternate" and t % 2 == 1)
            if blocking:
                g, flag, per, status = Gp.step(grads[t], M, X, Q, w.mu, w.eta, r)
                res.append((g, flag, per, status))
            else:
                assert Gp.step(grads[t], M, X, Q, w.mu, w.eta, r, wait=False) is None
                if mode == "each":
                    res.append(Gp.last_result())
        if asyn and mode == "end":
            res.append(Gp.last_result())
        torch.cuda.synchronize()
        runs.append((res, [f64(t) for t in M + X + Q]))
    (rb, sb), (ra, sa) = runs
    flags = [x[1] for x in rb]
    print(f"{gd} async ({mode}): decisions {flags}", flush=True)
    assert flags[0] and flags[5] and not all(flags) and not flags[4]
    if mode == "each":
        assert ra == rb
    elif mode == "end":
        assert ra[-1] == rb[-1]
    for a, b in zip(sa, sb):
        assert np.array_equal(a, b)


def test_async_every_h_and_status_reports():
    """Scheduled Sync (fixed branches) asynchronously equals blocking; an
    asynchronous step on a rank-deficient buffer reports CD_ERANKDEF through
    last_result, and one on a NaN gradient CD_ENONFINITE (the local branch ran)."""
    m, n, r = 192, 160, 24
    w = S.small_workload(m, n, r, k=4, stream_id=83)
    grads = _spiky_grads(w, 1, 7, spikes=())
    outs = []
    for asyn in (False, True):
        L = cdl.Layer(m, n, r, policy=cdl.POLICY_EVERY_H, H=3)
        M, X, Q = _state(w, 0)
        for t in range(7):
            L.step(grads[t][0], M, X, Q, 0.95, 0.01, r, wait=not asyn)
        rm, flag, st = L.last_result()
        torch.cuda.synchronize()
        outs.append((rm, flag, st, f64(M), f64(X), f64(Q)))
    assert outs[0][:3] == outs[1][:3] and outs[0][1] is False
    for a, b in zip(outs[0][3:], outs[1][3:]):
        assert np.array_equal(a, b)
    # B of rank 5 at r = 24: floored pivots
    gen = torch.Generator().manual_seed(5)
    G = torch.zeros(m, n)
    G[:5] = torch.randn(5, n, generator=gen) * 0.01
    L = cdl.Layer(m, n, r, policy=cdl.POLICY_ALWAYS_SYNC)
    M = torch.zeros(m, n, device=DEV)
    X = torch.randn(m, n, device=DEV) * 0.02
    Q = torch.linalg.qr(torch.randn(n, r, generator=gen, dtype=torch.float64))[0].float().to(DEV).contiguous()
    L.step(G.to(DEV), M, X, Q, 0.95, 0.01, r, wait=False)
    rm, flag, st = L.last_result()
    assert flag and st == cdl.CD_ERANKDEF and L.rank_deficient()
    # a full-rank step afterwards clears it
    L.step((torch.randn(m, n, generator=gen) * 0.01).to(DEV), M, X, Q, 0.95, 0.01, r, wait=False)
    L.step((torch.randn(m, n, generator=gen) * 0.01).to(DEV), M, X, Q, 0.95, 0.01, r, wait=False)
    assert L.last_result()[2] == cdl.CD_OK and not L.rank_deficient()
    # a NaN in G
    L2 = cdl.Layer(m, n, r, tau=0.5)
    M, X, Q = _state(w, 0)
    L2.step(grads[0][0], M, X, Q, 0.95, 0.01, r)
    Gn = grads[1][0].clone()
    Gn[3, 4] = float("nan")
    L2.step(Gn, M, X, Q, 0.95, 0.01, r, wait=False)
    rm, flag, st = L2.last_result()
    assert st == cdl.CD_ENONFINITE and not flag and math.isnan(rm)


@pytest.mark.parametrize("gd", ["f32", "bf16"])
def test_c_client_async_steps_match_blocking(gd, tmp_path):
    """The C99 client steps one layer ten times asynchronously (cd_step with
    no result pointer, each gradient in its own buffer), then reads
    cd_layer_last_result: M, X, Q and the last outcome are bit-identical to
    its blocking run over the same inputs, which syncs at step 1 and at the
    step-6 spike (a predicted skip reversed) and skips otherwise."""
    import shutil
    import subprocess
    from paper_2512_13728_amd import build
    exe = build.C_CLIENT
    if not os.path.exists(exe):
        pytest.skip("C client not built (build() compiles it)")
    m, n, r, steps, tau, mu, eta = 130, 200, 12, 10, 0.5, 0.95, 0.01
    w = S.small_workload(m, n, r, grad_dtype=gd, tau=tau, stream_id=35)
    M0, X0, Q0 = S.initial_state(w, 0)
    stream = S.GradientStream(w, 0)
    d1, d2 = tmp_path / "blocking", tmp_path / "async"
    d1.mkdir()
    M0.numpy().tofile(d1 / "M0.bin")
    X0.numpy().tofile(d1 / "X0.bin")
    Q0.numpy().tofile(d1 / "Q0.bin")
    for t in range(steps):
        G = stream.next()
        if t == 5:
            G = (G.float() * 40.0).to(G.dtype)
        (G.view(torch.int16) if gd == "bf16" else G).numpy().tofile(d1 / f"G{t}.bin")
    shutil.copytree(d1, d2)
    args = [str(m), str(n), str(r), str(steps), gd, str(cdl.POLICY_RMMC), repr(tau), repr(mu), repr(eta)]
    for mode, d in (("run", d1), ("async", d2)):
        print(f"C client {mode} {gd}", flush=True)
        out = subprocess.run([exe, mode, str(d)] + args, capture_output=True, text=True, timeout=120)
        assert out.returncode == 0, out.stdout + out.stderr
    rows = (d1 / "steps.txt").read_text().splitlines()
    flags = [ln.split()[1] == "1" for ln in rows]
    print(f"C client {gd}: blocking decisions {flags}", flush=True)
    assert flags[0] and flags[5] and not any(flags[1:5]) and not any(flags[6:])
    assert (d2 / "steps.txt").read_text().splitlines() == [rows[-1]]
    for f in ("M.bin", "X.bin", "Q.bin"):
        assert (d1 / f).read_bytes() == (d2 / f).read_bytes(), f
