"""Float64 CPU oracle for one CurvaDion optimizer step (TEST INFRASTRUCTURE ONLY).

This module is the checker, not the product.  Only the tests, the smoke check
and the benchmark's CPU-baseline leg may import it; the library itself never
calls it, and it shares no code with the HIP path.

It follows the paper's Algorithm 2 (CurvaDion, Sec. 2.2), which wraps the Dion
step of Algorithm 1 (Sec. 1.1) in a gate driven by the RMMC statistic (Eq. 1,
Sec. 2.1).  Everything is numpy float64; inputs in fp32 or bf16 widen exactly.
At one worker every data-parallel all-reduce of Algorithm 2 is the identity.

Readings of points the paper leaves open (each is also listed in the design
notes of the repository):

* Norm: Frobenius norm of the whole matrix (the proof expands ||M||^2 = M^T M).
* RMMC uses the executed form of Algorithm 2: |‖B_t‖ - prev| / (prev + eps),
  prev <- ‖B_t‖ on every step, prev_0 = 0, eps = 1e-8 unless given.
* Gate: global max over layers, strict ``>`` against tau (a tie skips, a NaN
  skips).
* PowerIter computes P~ = B Q_{t-1}; R is formed from the *orthonormalised* P,
  R = B^T P, so that P R^T = P P^T B is the rank-r projection of B.
* Orthogonalize: the thin-QR Q-factor whose R-factor has a positive diagonal
  (unique for full-rank P~).  Implemented with Householder QR
  (numpy.linalg.qr) and a column sign fix.
* ColumnNormalize: unit 2-norm columns, Q_j = R_j / max(‖R_j‖, 1e-30).
* Weight update scale sqrt(m/n) with m = rows, n = columns of the matrix.
* Local (skip) branch: M = B, X -= eta_local * G, Q unchanged; eta_local = eta
  unless given.
* Weight decay (the experiments of Sec. 4 use 0.01 and leave the form open):
  decoupled, X <- (1 - eta * weight_decay) X before either branch's update; M
  is untouched.  weight_decay = 0 (the default) is Algorithm 2 exactly.

Parity pins for every function live in tests/test_oracle_pins.py.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np

POLICY_RMMC = 0          # Algorithm 2: sync when max RMMC > tau
POLICY_ALWAYS_SYNC = 1   # Algorithm 1 (Dion baseline): every step syncs
POLICY_NEVER_SYNC = 2    # every step takes the local branch
POLICY_EVERY_H = 3       # Scheduled Sync Dion (Sec. 4.3): sync on every H-th step

COLNORM_FLOOR = 1e-30


def _f64(a) -> np.ndarray:
    return np.asarray(a, dtype=np.float64)


# --- Algorithm 2, local buffer update --------------------------------------
def buffer_update(M, G) -> np.ndarray:
    """B_t = M_{t-1} + G_t (Algorithm 2; the same step opens Algorithm 1)."""
    return _f64(M) + _f64(G)


# --- Eq. (1) as executed in Algorithm 2 -------------------------------------
def frobenius_norm(B) -> float:
    """‖B‖_F = sqrt(sum_ij B_ij^2), the layer norm the RMMC statistic compares."""
    B = _f64(B)
    return float(np.sqrt(np.sum(B * B)))


def rmmc(norm_b: float, prev_norm: float, eps: float) -> float:
    """RMMC_l = |‖B_t‖ - prev_norm| / (prev_norm + eps) (Eq. 1 in the form
    Algorithm 2 evaluates it)."""
    with np.errstate(divide="ignore", invalid="ignore"):
        return float(np.float64(abs(norm_b - prev_norm)) / np.float64(prev_norm + eps))


def gate(rmmc_values: Sequence[float], tau: float, policy: int = POLICY_RMMC,
         step: int = 1, H: int = 1):
    """Global max over layers and the sync decision (Algorithm 2, gate).

    Returns (global_max, sync_flag).  The max over workers is the identity at
    one worker.  ``max`` propagates a NaN, and NaN > tau is False, so a
    non-finite statistic takes the local branch.
    """
    vals = np.asarray(list(rmmc_values), dtype=np.float64)
    g = float(np.max(vals)) if vals.size else float("-inf")
    if np.isnan(vals).any():
        g = float("nan")
    if policy == POLICY_RMMC:
        flag = bool(g > tau)
    elif policy == POLICY_ALWAYS_SYNC:
        flag = True
    elif policy == POLICY_NEVER_SYNC:
        flag = False
    elif policy == POLICY_EVERY_H:
        flag = (step % H) == 0
    else:
        raise ValueError(f"unknown policy {policy}")
    return g, flag


# --- Dion synchronised branch (Algorithm 1 / Algorithm 2 sync branch) -------
def orthogonalize(P_tilde) -> np.ndarray:
    """Thin-QR Q-factor of P~ with a positive-diagonal R-factor.

    Householder QR (LAPACK via numpy), then each column j is multiplied by the
    sign of R_jj (a zero diagonal keeps sign +1).
    """
    Qf, Rf = np.linalg.qr(_f64(P_tilde), mode="reduced")
    s = np.sign(np.diag(Rf))
    s[s == 0] = 1.0
    return Qf * s[None, :]


def column_normalize(R) -> np.ndarray:
    """Q_j = R_j / max(‖R_j‖_2, 1e-30) for every column j."""
    R = _f64(R)
    norms = np.sqrt(np.sum(R * R, axis=0))
    return R / np.maximum(norms, COLNORM_FLOOR)[None, :]


def power_iteration(B, Q_prev):
    """PowerIter with the orthonormalisation between its two halves.

    P~ = B Q_{t-1}; P = Orthogonalize(P~); R = B^T P.  Returns (P~, P, R).
    """
    B = _f64(B)
    P_tilde = B @ _f64(Q_prev)
    P = orthogonalize(P_tilde)
    R = B.T @ P
    return P_tilde, P, R


def sync_update(B, X, Q_prev, mu: float, eta: float, x_decay: float = 1.0):
    """The full Dion update for one layer (Algorithm 2, sync branch).

    M_t = B_t - (1 - mu) P R^T;  Q_t = ColumnNormalize(R);
    X_t = x_decay X_{t-1} - eta sqrt(m/n) P Q_t^T  (x_decay = 1 - eta * weight decay).
    Returns dict with M, X, Q, P, P_tilde, R.
    """
    B = _f64(B)
    m, n = B.shape
    P_tilde, P, R = power_iteration(B, Q_prev)
    M = B - (1.0 - mu) * (P @ R.T)
    Q = column_normalize(R)
    Xn = x_decay * _f64(X) - eta * math.sqrt(m / n) * (P @ Q.T)
    return dict(M=M, X=Xn, Q=Q, P=P, P_tilde=P_tilde, R=R)


def local_update(B, G, X, eta_local: float, x_decay: float = 1.0):
    """Local branch of Algorithm 2: M_t = B_t; X_t = x_decay X_{t-1} - eta_local G_t."""
    return dict(M=_f64(B).copy(), X=x_decay * _f64(X) - eta_local * _f64(G))


# --- whole step over a set of layers -----------------------------------------
@dataclass
class OracleLayer:
    """Per-layer optimizer state: momentum M, weights X, right factor Q and
    the previous buffer norm (prev_norm_0 = 0 as in Algorithm 2)."""
    M: np.ndarray
    X: np.ndarray
    Q: np.ndarray
    prev_norm: float = 0.0
    step: int = 0
    last: dict = field(default_factory=dict)

    @classmethod
    def from_arrays(cls, M, X, Q, prev_norm: float = 0.0, step: int = 0):
        return cls(_f64(M).copy(), _f64(X).copy(), _f64(Q).copy(), float(prev_norm), step)

    @property
    def shape(self):
        return self.M.shape


def group_step(layers: List[OracleLayer], grads, mu: float, eta: float, tau: float,
               eps: float = 1e-8, policy: int = POLICY_RMMC, H: int = 1,
               eta_local: Optional[float] = None, with_kappa: bool = False,
               weight_decay: float = 0.0):
    """One CurvaDion step over all layers (Algorithm 2), updating ``layers``.
    weight_decay > 0 adds the decoupled decay X <- (1 - eta weight_decay) X.

    Every layer forms its buffer and RMMC first; the global max then decides one
    branch for all layers.  Returns dict(rmmc=[...], g=global max, flag=bool,
    kappa=[cond(P~) per layer] when requested and synced).
    """
    eta_local = eta if eta_local is None else eta_local
    x_decay = 1.0 - eta * weight_decay
    Bs, vals = [], []
    for L, G in zip(layers, grads):
        B = buffer_update(L.M, G)
        nb = frobenius_norm(B)
        vals.append(rmmc(nb, L.prev_norm, eps))
        L.prev_norm = nb
        L.step += 1
        Bs.append(B)
    step = layers[0].step if layers else 0
    g, flag = gate(vals, tau, policy, step, H)
    kappa = []
    for L, G, B in zip(layers, grads, Bs):
        if flag:
            out = sync_update(B, L.X, L.Q, mu, eta, x_decay)
            L.M, L.X, L.Q = out["M"], out["X"], out["Q"]
            L.last = out
            if with_kappa:
                kappa.append(float(np.linalg.cond(out["P_tilde"])))
        else:
            out = local_update(B, G, L.X, eta_local, x_decay)
            L.M, L.X = out["M"], out["X"]
            L.last = out
    return dict(rmmc=vals, g=g, flag=flag, kappa=kappa)
