"""GPU parity at the workloads' full sizes, in the launch configuration the
benchmark uses (one group per workload).  Where the oracle cannot afford the
whole set it checks what it can compute one layer at a time: every layer's
RMMC and the common decision at every step (the oracle's norms of all layers,
evaluated a layer per thread), and the full update of sampled layers (one of
each shape), teacher-forced from the GPU state, at every step.  Bounds as in
test_gpu_parity.py (gpu_util.check_errors), decision margins asserted."""
import concurrent.futures as cf
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
from gpu_util import (assert_rmmc_close, buffer_f32, check_errors, device_to_numpy, f32, f64,  # noqa: E402
                      rel, speculated, sync_errors, x_floor)

pytestmark = pytest.mark.gpu
DEV = "cuda"
POOL = cf.ThreadPoolExecutor(max_workers=min(16, len(os.sched_getaffinity(0))))


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cdl.lib()
    yield


def _sample_one_per_shape(w):
    seen, idx = set(), []
    for i, s in enumerate(w.shapes):
        if s not in seen:
            seen.add(s)
            idx.append(i)
    return idx


def _oracle_norm(Mi, Gi):
    """The oracle's ‖M + G‖_F of one layer (copied to the host first)."""
    return O.frobenius_norm(O.buffer_update(f64(Mi), f64(Gi)))


def _group_case(w, policy, steps, tau=None, sample=None, log="", H=1, margin=None, check_every=1):
    """Run `steps` group steps of workload w on the GPU; per step compare every
    layer's RMMC and the decision with the oracle (norms from the same inputs),
    and the sampled layers' full update teacher-forced on every sync step and
    on every check_every-th step.  Returns the decisions."""
    tau = w.tau if tau is None else tau
    L = len(w.shapes)
    layers = [cdl.Layer(m, n, w.r, grad_dtype=w.grad_dtype, tau=tau, policy=policy, H=H) for m, n in w.shapes]
    grp = cdl.Group(layers)
    st = [S.initial_state(w, i, device=DEV) for i in range(L)]
    M = [s[0] for s in st]
    X = [s[1] for s in st]
    Q = [s[2].contiguous() for s in st]
    streams = [S.GradientStream(w, i, device=DEV) for i in range(L)]
    prev = [0.0] * L
    sample = _sample_one_per_shape(w) if sample is None else sample
    bf16 = w.grad_dtype == "bf16"
    margin = (1e-2 if bf16 else 1e-4) if margin is None else margin
    flags, worst_margin = [], math.inf
    for t in range(steps):
        G = [s.next() for s in streams]
        # the oracle's statistic for every layer, from the same inputs
        nb = list(POOL.map(_oracle_norm, M, G))
        rm_or = [O.rmmc(nb[i], prev[i], w.eps) for i in range(L)]
        prev = nb
        g_or, flag_or = O.gate(rm_or, tau, policy, step=t + 1, H=H)
        checked = sample if (flag_or or t % check_every == 0) else []
        snap = {i: (f64(M[i]), f64(X[i]), f64(Q[i])) for i in checked}
        spec = speculated(grp, policy, t, 0.0 if t == 0 else 1.0, H)
        g, flag, per, _ = grp.step(G, M, X, Q, w.mu, w.eta, w.r)
        torch.cuda.synchronize()
        grp._last_sync = flag
        assert flag == flag_or, (t + 1, g, g_or)
        if policy == O.POLICY_RMMC and math.isfinite(g_or):
            worst_margin = min(worst_margin, abs(g_or - tau) / tau)
            assert abs(g_or - tau) / tau > margin, (t + 1, g_or, tau)
        for a, b in zip(per, rm_or):
            assert_rmmc_close(a, b)
        flags.append(flag)
        for i in checked:
            M0, X0, Q0 = snap[i]
            Gi = f64(G[i])
            B = buffer_f32(M0, Gi)
            Mg, Xg, Qg = f64(M[i]), f64(X[i]), f64(Q[i])
            if flag:
                out = O.sync_update(B, X0, Q0, f32(w.mu), f32(w.eta))
                m, n = w.shapes[i]
                P = device_to_numpy(layers[i].last_factors()[0], (m, w.r)).astype(np.float64)
                e = sync_errors(out, M0, X0, B, Mg, Xg, Qg, P, spec, f32(w.eta), Gi)
                e["kappa"] = float(np.linalg.cond(out["P_tilde"]))
            else:
                out = O.local_update(B, Gi, X0, f32(w.eta))
                e = {"err_M": rel(Mg, out["M"]), "err_X": rel(Xg, out["X"]), "err_Q": rel(Qg, Q0)}
                dX = out["X"] - X0
                e["err_dX"] = rel(Xg - X0, dX)
                e["dx_floor"] = x_floor(out["X"], dX, False)
            e["flag_oracle"] = flag
            print(f"{log} step {t + 1} layer {i} {w.shapes[i]} flag={flag} g={g:.4g} "
                  + " ".join(f"{k}={v:.2e}" for k, v in e.items()
                             if k.startswith(("err_", "tile_", "orth", "kappa"))), flush=True)
            check_errors(e, bf16)
    if policy == O.POLICY_RMMC:
        print(f"{log}: syncs at {[t + 1 for t, f in enumerate(flags) if f]}, smallest decision margin "
              f"|g - tau| / tau = {worst_margin:.3g}", flush=True)
    return flags


@pytest.mark.timeout(400)
def test_gpt1p3b_full_set_trajectory():
    """All 96 matrices of the 1.3B-shaped set, r = 512, bf16 gradients, its
    20 steps under tau = 0.5: step 1 syncs (prev_norm = 0), the others take
    the local branch.  Every step: the decision (margin > 1e-2) and every
    layer's RMMC; one layer per shape teacher-forced at every step."""
    w = S.WORKLOADS["gpt1p3b"]
    flags = _group_case(w, O.POLICY_RMMC, w.steps, log="gpt1p3b")
    assert flags == [True] + [False] * (w.steps - 1)


@pytest.mark.timeout(300)
def test_gpt1p3b_always_sync_second_step():
    """Two always-sync steps on one layer of each shape of the 1.3B set: the
    second has an ill-conditioned P~ (Q aligned with the previous signal)."""
    w = S.WORKLOADS["gpt1p3b"]
    w4 = S.Workload("gpt1p3b-4", tuple(w.shapes[:4]), r=w.r, grad_dtype="bf16", steps=2, k=w.k,
                    sigma=w.sigma, tau=w.tau, stream_id=w.stream_id)
    _group_case(w4, O.POLICY_ALWAYS_SYNC, 2, log="gpt1p3b-always")


@pytest.mark.timeout(300)
def test_gpt1p3b_block_every_h():
    """Scheduled Sync Dion (Sec. 4.3, sync every H = 4 steps) on one block of
    the 1.3B set (its four shapes), 9 steps: the three fixed syncs and the
    fused skip steps between them, all four layers teacher-forced at every
    step."""
    w = S.WORKLOADS["gpt1p3b"]
    w4 = S.Workload("gpt1p3b-4", tuple(w.shapes[:4]), r=w.r, grad_dtype="bf16", steps=9, k=w.k,
                    sigma=w.sigma, tau=w.tau, stream_id=w.stream_id)
    flags = _group_case(w4, O.POLICY_EVERY_H, 9, H=4, log="gpt1p3b-every4")
    assert flags == [(t + 1) % 4 == 0 for t in range(9)]


@pytest.mark.timeout(300)
def test_mixed1p3b_block_trajectory():
    """The mixed-phase generator (25-step flat and curved phases) on one block
    of the 1.3B set (its four shapes), all 200 steps under tau = 0.5: every
    step's decision (margin > 1e-2) and all four layers' RMMC; the layers
    teacher-forced on every sync step and every 10th step."""
    w = S.WORKLOADS["mixed1p3b"]
    w4 = S.Workload("mixed1p3b-4", tuple(w.shapes[:4]), r=w.r, grad_dtype="bf16", steps=w.steps, k=w.k,
                    sigma=w.sigma, tau=w.tau, kind="mixed", phase_len=w.phase_len, drift=w.drift,
                    sigma_flat=w.sigma_flat, curved_scale=w.curved_scale, stream_id=w.stream_id)
    flags = _group_case(w4, O.POLICY_RMMC, w.steps, log="mixed1p3b-4", check_every=10)
    assert flags[0]


@pytest.mark.timeout(300)
def test_gpt160m_full_set_spikes():
    """All 48 matrices of the 160M-shaped set (fp32, r = 192) for its 50
    steps, through both spikes (steps 10 and 30, tau = 0.3): every step's
    decision (margin > 1e-4) and every layer's RMMC, and the fp32 bounds on
    one layer per shape at every step."""
    w = S.WORKLOADS["gpt160m"]
    flags = _group_case(w, O.POLICY_RMMC, w.steps, log="gpt160m")
    assert flags[0] and flags[9] and flags[29]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("r", [16, 64, 256, 1024])
def test_sweep4096_ranks(r):
    """One 4096 x 16384 fp32 matrix at each rank of the sweep: two always-sync
    steps, strict fp32 bounds."""
    w = S.WORKLOADS["sweep4096"]
    w1 = S.Workload(f"sweep4096-r{r}", w.shapes, r=r, grad_dtype="f32", steps=2, k=w.k, sigma=w.sigma,
                    tau=w.tau, stream_id=w.stream_id)
    _group_case(w1, O.POLICY_ALWAYS_SYNC, 2, log=f"sweep r={r}")


def _chunked_norm(M, G, rows=2048):
    """||M + float(G)||_F in fp64, a row block at a time."""
    s = 0.0
    for i in range(0, M.shape[0], rows):
        s += float(torch.sum((M[i:i + rows] + G[i:i + rows].float()).double() ** 2))
    return math.sqrt(s)


@pytest.mark.parametrize("gd", ["bf16", "f32"])
def test_layer_past_32bit_indexing(gd):
    """One layer of 46341 x 46341 = 2^31 + 4633 elements (25-26 GB with M, X
    and G), r = 8, for either gradient dtype (their sync paths use different
    kernels): every kernel's element index exceeds 32 bits.
    The oracle cannot run at this size, so the check uses what holds at any
    size.  Step 1 syncs (prev_norm starts at 0): ||B|| against a chunked fp64
    norm; P orthonormal and spanning P~ = B Q0 with an upper-triangular,
    positive-diagonal factor P^T P~; R = B^T P on sampled columns; M =
    B - (1 - mu) P R^T and X = X0 - eta sqrt(m/n) P Q^T on sampled rows;
    Q = ColumnNormalize(R).  Step 2 takes the local branch: M = M + G and
    X = X - eta G bit-exact on sampled rows, RMMC from the two fp64 norms."""
    m = n = 46341
    r, mu, eta = 8, 0.95, 0.01
    assert m * n > 2 ** 31
    gen = torch.Generator(device=DEV).manual_seed(4242)
    M = torch.randn(m, n, generator=gen, device=DEV) * 0.02
    X = torch.randn(m, n, generator=gen, device=DEV) * 0.02
    gdt = torch.bfloat16 if gd == "bf16" else torch.float32
    G = (torch.randn(m, n, generator=gen, device=DEV) * 0.01).to(gdt)
    Q0 = torch.linalg.qr(torch.randn(n, r, generator=gen, device=DEV, dtype=torch.float64))[0]
    Q = Q0.float().contiguous()
    rows = [0, 1, m // 2, m - 2, m - 1]
    cols = [0, 3, n // 2, n - 1]
    B_rows = (M[rows] + G[rows].float()).double()
    B_cols = (M[:, cols] + G[:, cols].float()).double()
    X0_rows = X[rows].double()
    nb1 = _chunked_norm(M, G)
    # P~ = B Q0 in fp64, a row block at a time
    Pt = torch.empty(m, r, dtype=torch.float64, device=DEV)
    for i in range(0, m, 2048):
        Pt[i:i + 2048] = (M[i:i + 2048] + G[i:i + 2048].float()).double() @ Q0
    L = cdl.Layer(m, n, r, grad_dtype=gd, tau=1e6)
    print(f"32-bit-index case: {m} x {n} {gd}, r = {r}", flush=True)
    # bf16 layers: two-piece products for the power iteration, plain bf16 for
    # the rank-r corrections; fp32 layers: fp64 and six-piece products (their
    # corrections are then bounded by the fp32 rounding of M and X themselves)
    tol_pow, tol_corr = (1e-3, 2e-2) if gd == "bf16" else (1e-5, 1e-3)
    rm, flag, st = L.step(G, M, X, Q, mu, eta, r)
    torch.cuda.synchronize()
    assert flag and st == cdl.CD_OK
    prev1, step1 = L.get_state()
    assert step1 == 1 and abs(prev1 - nb1) <= 1e-6 * nb1, (prev1, nb1)
    Pa, Ra = L.last_factors()
    P = torch.from_numpy(device_to_numpy(Pa, (m, r))).double().to(DEV)
    R = torch.from_numpy(device_to_numpy(Ra, (n, r))).double().to(DEV)
    assert float((P.T @ P - torch.eye(r, device=DEV, dtype=torch.float64)).abs().max()) <= (1e-4 if gd == "bf16" else 1e-5)
    C = P.T @ Pt                                   # the R-factor of P~ = P C
    assert float(torch.linalg.norm(Pt - P @ C) / torch.linalg.norm(Pt)) <= tol_pow
    assert float(torch.tril(C, -1).abs().max()) <= tol_pow * float(C.abs().max())
    assert bool((torch.diagonal(C) > 0).all())
    # R = B^T P on sampled columns (two-piece bf16 products: about 2^-16)
    R_cols = B_cols.T @ P
    assert float(torch.linalg.norm(R[cols] - R_cols) / torch.linalg.norm(R_cols)) <= tol_pow
    # M and X on sampled rows (plain bf16 products in the rank-r update)
    Qd = Q.double()
    colnrm = torch.linalg.norm(R, dim=0)
    assert float((Qd - R / colnrm).abs().max()) <= 1e-5
    # (the corrections are about 1e-4 of B and X here, so they are compared
    # themselves, at the bound of plain bf16 products)
    dM = (1 - f32(mu)) * P[rows] @ R.T
    dX = f32(eta) * math.sqrt(m / n) * P[rows] @ Qd.T
    assert float(torch.linalg.norm((B_rows - M[rows].double()) - dM) / torch.linalg.norm(dM)) <= tol_corr
    assert float(torch.linalg.norm((X0_rows - X[rows].double()) - dX) / torch.linalg.norm(dX)) <= tol_corr
    # step 2: the local branch, bit-exact on sampled rows
    M1_rows, X1_rows = M[rows].clone(), X[rows].clone()
    G.copy_((torch.randn(m, n, generator=gen, device=DEV) * 0.01).to(gdt))
    nb2 = _chunked_norm(M, G)
    rm2, flag2, _ = L.step(G, M, X, Q, mu, eta, r)
    torch.cuda.synchronize()
    assert not flag2
    assert abs(rm2 - abs(nb2 - prev1) / (prev1 + 1e-8)) <= 1e-5 * rm2 + 1e-9
    Gr = G[rows].float()
    assert torch.equal(M[rows], M1_rows + Gr)
    # X - eta G is one fused multiply-add in fp32: within 1 ulp of the fp64 value
    Xref = X1_rows.double() - f32(eta) * Gr.double()
    assert bool(((X[rows].double() - Xref).abs() <= Xref.abs() * 2.0 ** -23 + 1e-30).all())
