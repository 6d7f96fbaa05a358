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
    """Tolerance for P, Q and dX: the QR factor of an fp32 P~ is determined only
    to about kappa_2(P~) * u (Higham, ch. 19); never below 1e-5."""
    return max(1e-5, c * kappa * U32)


def step_and_compare(layer: cdl.Layer, G, M, X, Q, mu, eta, r, tau, policy, eps=1e-8,
                     eta_local_scale=1.0, weight_decay=0.0):
    """Run one library step on (G, M, X, Q) and the oracle on the same inputs.
    Returns a dict of errors and both decisions.  M, X, Q are updated in place
    (the device state becomes the next step's input)."""
    M0, X0, Q0 = f64(M), f64(X), f64(Q)
    prev0, step0 = layer.get_state()
    rm, flag, st = layer.step(G, M, X, Q, mu, eta, r)
    torch.cuda.synchronize()
    OL = O.OracleLayer.from_arrays(M0, X0, Q0, prev_norm=prev0, step=step0)
    res = O.group_step([OL], [f64(G)], f32(mu), f32(eta), tau, eps=eps, policy=policy,
                       eta_local=f32(eta) * eta_local_scale, with_kappa=True,
                       weight_decay=weight_decay)
    out = dict(flag_gpu=flag, flag_oracle=res["flag"], rmmc_gpu=rm, rmmc_oracle=res["g"],
               status=st)
    out["err_M"] = rel(f64(M), OL.M)
    out["err_X"] = rel(f64(X), OL.X)
    dX = OL.X - X0
    ndx = np.linalg.norm(dX)
    out["err_dX"] = rel(f64(X) - X0, dX) if ndx > 0 else float(np.max(np.abs(f64(X) - X0)))
    # X is stored in fp32: each rounding of X moves dX by up to u |X| per entry;
    # a sync step that follows a predicted skip rounds X three times (the
    # speculative X -= eta_l G, its reversal, the rank-r update)
    out["dx_floor"] = 4.0 * U32 * float(np.linalg.norm(OL.X)) / ndx if ndx > 0 else 0.0
    out["err_Q"] = rel(f64(Q), OL.Q)
    if res["flag"]:
        m, n = M.shape
        Pg, _ = layer.last_factors()
        P = device_to_numpy(Pg, (m, r)).astype(np.float64)
        out["err_P"] = rel(P, OL.last["P"])
        out["orth_P"] = float(np.linalg.norm(P.T @ P - np.eye(r)))
        out["kappa"] = res["kappa"][0]
        qn = np.sqrt(np.sum(f64(Q) ** 2, axis=0))
        out["colnorm_dev"] = float(np.max(np.abs(qn - 1.0)))
    return out


def assert_rmmc_close(g, o):
    if math.isinf(o) or math.isinf(g):
        assert g == o
        return
    assert abs(g - o) <= 1e-5 * abs(o) + 1e-7, (g, o)
