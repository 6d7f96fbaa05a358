"""Helpers for the GPU parity tests: device <-> host copies of library-owned
buffers, error norms, and one teacher-forced step against the oracle."""
from __future__ import annotations

import ctypes
import math

import numpy as np
import torch

import oracle as O
import paper_2512_13728_amd as cdl

U32 = 2.0 ** -24  # unit roundoff of fp32

# Bounds (rel-Frobenius against the oracle; the largest measured values over
# the GPU suite in brackets).  fp32 gradients: the power iteration, both
# CholQR passes and R = B^T P run in fp64 and everything is stored in fp32,
# so P, Q and M carry a few fp32 roundings [P 2.7e-8 at kappa 1.2e6, Q 5.2e-8,
# M 3.7e-8]; the rank-r corrections use fp32-accurate split products
# [dM 1.1e-6, its largest 128 x 64 tile 1.5e-6]; X [8.3e-7] and dX carry
# the fp32 rounding of X itself (x_floor).
TIGHT_F32 = 5e-7   # P, Q, M with fp32 gradients
TOL_F32 = 1e-5     # X, dM, dX with fp32 gradients (the stated fp32 tolerance)
TILE_F32 = 1.5e-5  # the largest tile of dM, dX, P with fp32 gradients
# bf16 gradients: the power products use two-piece splits (about 2^-16), so
# P, Q and dX move by about kappa(P~) 2^-16 times a small factor [1.5e-2 at
# kappa 2e6]: the stated 2e-2; the rank-r corrections use plain bf16
# products [dM 2.9e-3, tile 3.0e-3], which reach M and X only through that
# (1 - mu) and eta-scaled correction [M 1.5e-4, X 7.1e-4].
TOL_BF16 = 2e-2    # P, Q, dM, dX and every tile with bf16 gradients
M_BF16 = 2e-3
X_BF16 = 5e-3

_hip = None


def hip():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        _hip.hipMemcpy.restype = ctypes.c_int
    return _hip


def device_to_numpy(addr: int, shape, dtype=np.float32) -> np.ndarray:
    """Copy a library-owned device buffer to the host (after a sync)."""
    torch.cuda.synchronize()
    out = np.empty(shape, dtype=dtype)
    st = hip().hipMemcpy(out.ctypes.data, addr, out.nbytes, 2)  # hipMemcpyDeviceToHost
    assert st == 0, f"hipMemcpy failed: {st}"
    return out


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to("cpu").to(torch.float64).numpy()


def rel(a, b) -> float:
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (nb if nb > 0 else 1.0))


def f32(x: float) -> float:
    """The fp32 value the library receives for a Python float argument."""
    return float(np.float32(x))


def qr_tol(kappa: float, c: float = 8.0) -> float:
    """Tolerance for P, Q and dX when the oracle starts from the exact buffer
    B = M + G: the QR factor of P~ = B Q then moves by about kappa_2(P~) u
    under the fp32 rounding of B the kernels store (Higham, ch. 19); never
    below 1e-5."""
    return max(1e-5, c * kappa * U32)


def buffer_f32(M0: np.ndarray, G: np.ndarray) -> np.ndarray:
    """The buffer the kernels hold after the buffer pass: B = M + G rounded to
    fp32 (one IEEE addition per element, as the kernel's), widened to fp64.
    Fed to the oracle's sync branch so that the comparison measures the
    kernels' arithmetic and not the fp32 storage of the state (the momentum
    is fp32 state, and B overwrites it in place)."""
    return (np.asarray(M0, np.float32) + np.asarray(G, np.float64).astype(np.float32)).astype(np.float64)


def tile_rel_max(a, b, tm: int = 128, tn: int = 64) -> float:
    """Largest relative Frobenius error over tm x tn tiles (the update
    kernel's tile shape for matrices; 64-row panels for P).  A tile whose
    reference norm is below a tenth of the RMS tile norm is measured against
    that tenth, so near-zero tiles compare on the matrix's own scale.  One
    wholly wrong tile gives a value near 1 or above, whatever the matrix size."""
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    m, n = b.shape
    ti, tj = -(-m // tm), -(-n // tn)
    pad = ((0, ti * tm - m), (0, tj * tn - n))
    d = np.pad(a - b, pad).reshape(ti, tm, tj, tn)
    r = np.pad(b, pad).reshape(ti, tm, tj, tn)
    en = np.sqrt(np.einsum("iajb,iajb->ij", d, d))
    rn = np.sqrt(np.einsum("iajb,iajb->ij", r, r))
    rms = np.linalg.norm(b) / math.sqrt(ti * tj)
    den = np.maximum(rn, 0.1 * rms)
    if rms == 0:
        return float(np.max(en))
    return float(np.max(en / den))


def speculated(obj, policy: int, step0: int, prev0: float, H: int = 1) -> bool:
    """Whether the library's buffer pass applied the skip branch's X update
    ahead of the gate (its documented prediction): fixed policies know the
    branch; the RMMC policy predicts the previous step's branch, except when
    a prev_norm is 0.  `obj` is the Layer or Group; the tests record its last
    decision on it as `_last_sync`."""
    if policy == O.POLICY_NEVER_SYNC:
        return True
    if policy == O.POLICY_ALWAYS_SYNC:
        return False
    if policy == O.POLICY_EVERY_H:
        return (step0 + 1) % H != 0
    return prev0 != 0.0 and getattr(obj, "_last_sync", None) is False


def x_floor(X_new, dX, spec_reversed: bool, eta_l: float = 0.0, G=None) -> float:
    """The fp32 rounding floor of dX = X_t - X_{t-1}, relative to ‖dX‖: X is
    rounded up to three times in a step (the speculative X - eta_l G, its
    reversal, the rank-r update), each by at most u times the magnitude then
    held, which after a speculative update includes ‖eta_l G‖."""
    ndx = float(np.linalg.norm(dX))
    if ndx == 0:
        return 0.0
    mag = float(np.linalg.norm(X_new))
    if spec_reversed and G is not None:
        mag += eta_l * float(np.linalg.norm(G))
    return 4.0 * U32 * mag / ndx


def sync_errors(out: dict, M0, X0, B, Mg, Xg, Qg, Pg, spec=False, eta_l=0.0, G=None) -> dict:
    """Errors of one sync step against the oracle's sync branch `out` (run on
    the buffer B the kernels hold): M, X, Q, P globally; the momentum
    correction dM = B - M against (1 - mu) P R^T and the weight change
    dX = X_t - X_{t-1} as quantities of their own; and the largest per-tile
    error of dM, dX (128 x 64 tiles, the update's tile) and P (64-row panels)."""
    e = {"err_M": rel(Mg, out["M"]), "err_X": rel(Xg, out["X"]), "err_Q": rel(Qg, out["Q"])}
    dM_or, dM = B - out["M"], B - Mg
    dX_or, dX = out["X"] - X0, Xg - X0
    e["err_dM"] = rel(dM, dM_or)
    e["err_dX"] = rel(dX, dX_or)
    e["tile_dM"] = tile_rel_max(dM, dM_or)
    e["tile_dX"] = tile_rel_max(dX, dX_or)
    if Pg is not None:
        e["err_P"] = rel(Pg, out["P"])
        e["tile_P"] = tile_rel_max(Pg, out["P"], 64, Pg.shape[1])
        r = Pg.shape[1]
        e["orth_P"] = float(np.linalg.norm(Pg.T @ Pg - np.eye(r)))
    qn = np.sqrt(np.sum(np.asarray(Qg, np.float64) ** 2, axis=0))
    e["colnorm_dev"] = float(np.max(np.abs(qn - 1.0)))
    e["dx_floor"] = x_floor(out["X"], dX_or, spec, eta_l, G)
    return e


def step_and_compare(layer: cdl.Layer, G, M, X, Q, mu, eta, r, tau, policy, eps=1e-8,
                     eta_local_scale=1.0, weight_decay=0.0, H=1):
    """Run one library step on (G, M, X, Q) and the oracle on the same inputs.
    The decision and RMMC come from the oracle's whole step on the exact
    buffer M + G; the branch's outputs from the oracle's branch on the
    fp32 buffer the kernels hold (buffer_f32).  Returns a dict of errors and
    both decisions.  M, X, Q are updated in place (the device state becomes
    the next step's input)."""
    M0, X0, Q0 = f64(M), f64(X), f64(Q)
    prev0, step0 = layer.get_state()
    spec = speculated(layer, policy, step0, prev0, H)
    rm, flag, st = layer.step(G, M, X, Q, mu, eta, r)
    torch.cuda.synchronize()
    layer._last_sync = flag
    G64 = f64(G)
    OL = O.OracleLayer.from_arrays(M0, X0, Q0, prev_norm=prev0, step=step0)
    res = O.group_step([OL], [G64], f32(mu), f32(eta), tau, eps=eps, policy=policy, H=H,
                       eta_local=f32(eta) * eta_local_scale, with_kappa=True,
                       weight_decay=weight_decay)
    out = dict(flag_gpu=flag, flag_oracle=res["flag"], rmmc_gpu=rm, rmmc_oracle=res["g"],
               status=st)
    B = buffer_f32(M0, G64)
    x_decay = 1.0 - f32(eta) * weight_decay
    Mg, Xg, Qg = f64(M), f64(X), f64(Q)
    if res["flag"]:
        ref = O.sync_update(B, X0, Q0, f32(mu), f32(eta), x_decay)
        m, n = M.shape
        Pa, _ = layer.last_factors()
        P = device_to_numpy(Pa, (m, r)).astype(np.float64)
        out.update(sync_errors(ref, M0, X0, B, Mg, Xg, Qg, P, spec, f32(eta) * eta_local_scale, G64))
        out["kappa"] = res["kappa"][0]
    else:
        ref = O.local_update(B, G64, X0, f32(eta) * eta_local_scale, x_decay)
        out["err_M"] = rel(Mg, ref["M"])
        out["err_X"] = rel(Xg, ref["X"])
        out["err_Q"] = rel(Qg, Q0)
        dX = ref["X"] - X0
        ndx = np.linalg.norm(dX)
        out["err_dX"] = rel(Xg - X0, dX) if ndx > 0 else float(np.max(np.abs(Xg - X0)))
        out["dx_floor"] = x_floor(ref["X"], dX, False)
    out["ref"] = ref
    return out


def assert_rmmc_close(g, o):
    if math.isinf(o) or math.isinf(g):
        assert g == o
        return
    assert abs(g - o) <= 1e-5 * abs(o) + 1e-7, (g, o)
def group_step_and_compare(group: cdl.Group, layers, G, M, X, Q, mu, eta, r, tau, policy, *, H=1,
                           eps=1e-8, eta_local_scale=1.0, weight_decay=0.0, check=None):
    """One group step on the GPU and, teacher-forced from the GPU's state, the
    oracle's: its whole step (the exact buffers) gives every layer's RMMC and
    the decision; its branch on the fp32 buffers the kernels hold gives the
    outputs of the layers in `check` (default: all), compared as in
    step_and_compare.  Returns (decision info, {layer: errors})."""
    L = len(layers)
    check = range(L) if check is None else check
    snap = {i: (f64(M[i]), f64(X[i]), f64(Q[i])) for i in check}
    states = [lay.get_state() for lay in layers]
    spec = speculated(group, policy, states[0][1], min(st[0] for st in states), H)
    OLs = []
    for i in range(L):
        M0, X0, Q0 = snap[i] if i in snap else (f64(M[i]), None, None)
        OLs.append(O.OracleLayer(M0, X0, Q0, prev_norm=states[i][0], step=states[i][1]))
    g, flag, per, st = group.step(G, M, X, Q, mu, eta, r)
    torch.cuda.synchronize()
    group._last_sync = flag
    G64 = [f64(t) for t in G]
    # the decision and every RMMC: buffers and norms only (the branch of the
    # layers that are not checked is not needed)
    rm = []
    for i, OL in enumerate(OLs):
        B = O.buffer_update(OL.M, G64[i])
        rm.append(O.rmmc(O.frobenius_norm(B), OL.prev_norm, eps))
    g_or, flag_or = O.gate(rm, tau, policy, step=states[0][1] + 1, H=H)
    info = dict(flag_gpu=flag, flag_oracle=flag_or, rmmc_gpu=g, rmmc_oracle=g_or, per_gpu=per,
                per_oracle=rm, status=st)
    errs = {}
    x_decay = 1.0 - f32(eta) * weight_decay
    for i in check:
        M0, X0, Q0 = snap[i]
        B = buffer_f32(M0, G64[i])
        Mg, Xg, Qg = f64(M[i]), f64(X[i]), f64(Q[i])
        if flag_or:
            ref = O.sync_update(B, X0, Q0, f32(mu), f32(eta), x_decay)
            m, n = M0.shape
            P = device_to_numpy(layers[i].last_factors()[0], (m, r)).astype(np.float64)
            e = sync_errors(ref, M0, X0, B, Mg, Xg, Qg, P, spec, f32(eta) * eta_local_scale, G64[i])
            e["kappa"] = float(np.linalg.cond(ref["P_tilde"]))
        else:
            ref = O.local_update(B, G64[i], X0, f32(eta) * eta_local_scale, x_decay)
            e = {"err_M": rel(Mg, ref["M"]), "err_X": rel(Xg, ref["X"]), "err_Q": rel(Qg, Q0)}
            dX = ref["X"] - X0
            ndx = np.linalg.norm(dX)
            e["err_dX"] = rel(Xg - X0, dX) if ndx > 0 else float(np.max(np.abs(Xg - X0)))
            e["dx_floor"] = x_floor(ref["X"], dX, False)
        e["flag_gpu"], e["flag_oracle"] = flag, flag_or
        e["rmmc_gpu"], e["rmmc_oracle"] = per[i], rm[i]
        errs[i] = e
    return info, errs


def check_errors(d, bf16=False):
    """The bounds of this module on one layer's step errors (sync_errors or
    the local-branch errors), given the decision the step took."""
    d = {k: v for k, v in d.items() if k != "ref"}
    if bf16:
        assert d["err_M"] <= M_BF16, d
        assert d["err_X"] <= X_BF16, d
        for k in ("err_P", "err_Q", "err_dM", "err_dX", "tile_dM", "tile_dX", "tile_P"):
            if k in d:
                assert d[k] <= TOL_BF16, (k, d)
        if d["flag_oracle"]:
            assert d["orth_P"] <= 1e-4 and d["colnorm_dev"] <= 1e-5, d
        return
    assert d["err_M"] <= TIGHT_F32, d
    assert d["err_X"] <= TOL_F32, d
    if d["flag_oracle"]:
        assert d["orth_P"] <= 1e-5, d
        assert d["colnorm_dev"] <= 1e-5, d
        for k in ("err_P", "err_Q"):
            assert d[k] <= TIGHT_F32, (k, d)
        assert d["err_dM"] <= TOL_F32, d
        assert d["err_dX"] <= TOL_F32 + d["dx_floor"], d
        for k in ("tile_dM", "tile_P"):
            assert d[k] <= TILE_F32, (k, d)
        assert d["tile_dX"] <= TILE_F32 + 4 * d["dx_floor"], d
    else:
        assert d["err_Q"] == 0.0
        assert d["err_dX"] <= 1e-6 + d["dx_floor"], d
