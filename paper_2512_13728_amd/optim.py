"""torch.optim front end for the CurvaDion step (Algorithm 2, Sec. 2.2).

Every 2-D parameter is one layer of the method: the optimizer keeps its
momentum M (fp32, m x n) and right factor Q (fp32, n x r) on the device and
hands p.grad, M, p and Q to the library once per step (one cd_group_step over
all matrices, so the sync decision is the max of RMMC over all of them).  The
arithmetic runs in the library's HIP kernels; this module only allocates the
state and marshals pointers.

Parameters must be contiguous fp32 CUDA matrices; gradients fp32 or bf16
(matrices whose gradients differ in dtype step in separate groups, each with
its own decision).  The learning rate is read from the param group on every
step, so torch.optim.lr_scheduler schedules apply.  Non-matrix parameters
(biases, norms, embeddings if wanted) belong to another optimizer, as in the
paper's setup, where Dion handles the weight matrices.
"""
from __future__ import annotations

import math
from typing import Iterable, Optional

import torch

from . import (POLICY_ALWAYS_SYNC, POLICY_EVERY_H, POLICY_NEVER_SYNC, POLICY_RMMC, Group, Layer)

_POLICIES = {"rmmc": POLICY_RMMC, "always": POLICY_ALWAYS_SYNC, "never": POLICY_NEVER_SYNC,
             "every_h": POLICY_EVERY_H}


def orthonormal_start(n: int, r: int, device, seed: int = 0) -> torch.Tensor:
    """n x r matrix with orthonormal columns and no QR: r distinct columns of
    the orthonormal DCT-II basis (frequencies spread over 0..n-1, chosen by
    the seed), so Q_0 is deterministic and dense."""
    g = torch.Generator().manual_seed(seed)
    freqs = torch.randperm(n, generator=g)[:r].to(torch.float64)
    i = torch.arange(n, dtype=torch.float64)[:, None]
    q = torch.cos(math.pi * (i + 0.5) * freqs[None, :] / n)
    q *= torch.where(freqs == 0, math.sqrt(1.0 / n), math.sqrt(2.0 / n))[None, :]
    return q.to(torch.float32).to(device).contiguous()


class CurvaDion(torch.optim.Optimizer):
    """CurvaDion over the given 2-D parameters.

    lr: eta;  momentum: mu;  rank: r per matrix (int), or a fraction of
    min(m, n) (float < 1, at least 1);  tau: gate threshold;  policy: "rmmc"
    (Algorithm 2), "always" (Dion, Algorithm 1), "never", or "every_h" with H;
    weight_decay: decoupled lambda (X <- (1 - lr lambda) X each step);
    eta_local_scale: eta_local / eta for the skip branch.
    """

    def __init__(self, params: Iterable[torch.nn.Parameter], lr: float = 0.02, momentum: float = 0.95,
                 rank=0.125, tau: float = 0.5, eps: float = 1e-8, policy: str = "rmmc", H: int = 1,
                 weight_decay: float = 0.0, eta_local_scale: float = 1.0, seed: int = 0):
        if policy not in _POLICIES:
            raise ValueError(f"policy must be one of {sorted(_POLICIES)}")
        defaults = dict(lr=lr, momentum=momentum)
        super().__init__(params, defaults)
        self._cfg = dict(rank=rank, tau=tau, eps=eps, policy=_POLICIES[policy], H=H,
                         weight_decay=weight_decay, eta_local_scale=eta_local_scale, seed=seed)
        for grp in self.param_groups:
            for p in grp["params"]:
                if p.dim() != 2 or p.dtype != torch.float32 or not p.is_contiguous():
                    raise ValueError("CurvaDion takes contiguous fp32 matrices "
                                     f"(got {tuple(p.shape)} {p.dtype})")
        self._groups = {}          # grad dtype -> (Group, params, packed M, X, Q, ranks)
        self.last = {}             # grad dtype -> (rmmc, synced)

    def _rank(self, m: int, n: int) -> int:
        rk = self._cfg["rank"]
        if isinstance(rk, float) and rk < 1.0:
            return max(1, int(round(rk * min(m, n))))
        return max(1, min(int(rk), m, n))

    def _build(self, gdtype, params):
        c = self._cfg
        layers, Ms, Qs, ranks = [], [], [], []
        for k, p in enumerate(params):
            m, n = p.shape
            r = self._rank(m, n)
            st = self.state[p]
            if "M" not in st:
                st["M"] = torch.zeros_like(p)
                st["Q"] = orthonormal_start(n, r, p.device, seed=c["seed"] + k)
            layers.append(Layer(m, n, r, grad_dtype="bf16" if gdtype == torch.bfloat16 else "f32",
                                tau=c["tau"], eps=c["eps"], eta_local_scale=c["eta_local_scale"],
                                policy=c["policy"], H=c["H"], weight_decay=c["weight_decay"]))
            Ms.append(st["M"]); Qs.append(st["Q"]); ranks.append(r)
        grp = Group(layers)
        if len(set(ranks)) != 1:
            # one cd_group_step takes one r: step matrices of each rank separately
            raise ValueError("all matrices of one gradient dtype must share the rank; pass an int rank")
        return dict(group=grp, layers=layers, params=list(params), M=grp.pack(Ms, "M"),
                    X=grp.pack(list(params), "X"), Q=grp.pack(Qs, "Q", ranks[0]), r=ranks[0])

    @torch.no_grad()
    def step(self, closure: Optional[callable] = None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        by_dtype = {}
        lr = mu = None
        for grp in self.param_groups:
            lr = grp["lr"] if lr is None else lr
            mu = grp["momentum"] if mu is None else mu
            if grp["lr"] != lr or grp["momentum"] != mu:
                raise ValueError("one lr and momentum for all matrices (one group step)")
            for p in grp["params"]:
                if p.grad is None:
                    raise ValueError("every CurvaDion matrix needs a gradient each step")
                by_dtype.setdefault(p.grad.dtype, []).append(p)
        for gdtype, params in by_dtype.items():
            g = self._groups.get(gdtype)
            if g is None or [id(q) for q in g["params"]] != [id(q) for q in params]:
                g = self._groups[gdtype] = self._build(gdtype, params)
            grads = [p.grad if p.grad.is_contiguous() else p.grad.contiguous() for p in params]
            rm, flag, _, _ = g["group"].step(grads, g["M"], g["X"], g["Q"], float(mu), float(lr), g["r"])
            self.last[gdtype] = (rm, flag)
        return loss
