"""Seeded synthetic inputs for the CurvaDion optimizer step.

The paper trains GPT-style models on FineWeb (Sec. 4); neither the data nor the
trained checkpoints are available, so seeded synthetic gradient streams stand in
for them.  Layer shapes follow the model sizes of Table 1 (d_model 768 / 2048):
per transformer block a QKV matrix d x 3d, an output projection d x d and the two
MLP matrices d x 4d and 4d x d.

This module only *draws* inputs: layer shapes, initial states (M0, X0, Q0) and
per-step gradients G_t.  It contains none of the optimizer's arithmetic and is
imported by both the float64 oracle side and the GPU side of the tests, so that
the two see the same bits.  Gradients are built as

    G_t = U_t V_t^T + sigma * N_t          (U: m x k, V: n x k, N: m x n)

with all factors i.i.d. standard normal and a fresh seed per (stream, layer,
step).  Variants per workload are documented on ``WORKLOADS``.

Randomness comes from ``torch.Generator`` on the device the tensors are made on.
CPU and GPU generators give different streams, so a parity test draws once and
copies the tensor to the other side; it never re-draws.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

__all__ = [
    "Workload", "WORKLOADS", "gpt_layer_shapes", "seed_for", "initial_state",
    "random_orthonormal", "GradientStream",
]


def gpt_layer_shapes(d_model: int, blocks: int) -> List[Tuple[int, int]]:
    """The four 2-D weight matrices of each GPT block, rows x cols, per block."""
    d = d_model
    one = [(d, 3 * d), (d, d), (d, 4 * d), (4 * d, d)]
    return one * blocks


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: shapes, rank, dtypes, hyper-parameters and the
    gradient recipe.  ``kind`` selects the stream variant:

    * ``lowrank``: fresh U, V every step.
    * ``spikes``: as ``lowrank``; at the steps in ``spike_steps`` the low-rank
      part is drawn from an independent stream and scaled by ``spike_scale``
      (a sudden rotation of the gradient direction with a larger magnitude).
    * ``mixed``: blocks of ``phase_len`` steps, flat first.  Flat phases keep a
      slowly drifting subspace, U_t = U_{t-1} + drift * N (same for V), with
      noise ``sigma_flat``; curved phases redraw U, V each step and scale the
      low-rank part by ``curved_scale``.
    """
    name: str
    shapes: Tuple[Tuple[int, int], ...]
    r: int
    grad_dtype: str            # "f32" | "bf16"
    steps: int
    mu: float = 0.95
    eta: float = 0.01
    tau: float = 0.5
    eps: float = 1e-8
    k: int = 8                 # rank of the low-rank gradient part
    sigma: float = 0.1         # std of the i.i.d. noise part
    init_std: float = 0.02     # std of M0 and X0
    kind: str = "lowrank"
    spike_steps: Tuple[int, ...] = ()
    spike_scale: float = 10.0
    phase_len: int = 25
    drift: float = 0.01
    sigma_flat: float = 0.05
    curved_scale: float = 5.0
    stream_id: int = 0

    @property
    def params(self) -> int:
        return sum(m * n for m, n in self.shapes)


_C2 = tuple(gpt_layer_shapes(768, 12))
_C3 = tuple(gpt_layer_shapes(2048, 24))

#: The workloads the library is tested and measured on (names describe them).
WORKLOADS: Dict[str, Workload] = {
    # one 256 x 256 fp32 matrix, r = 16, rank-8 gradients, 20 steps
    "single256": Workload("single256", ((256, 256),), r=16, grad_dtype="f32",
                          steps=20, k=8, sigma=0.1, tau=0.5, stream_id=1),
    # 160M-shaped set: 48 fp32 matrices, r = d/4 = 192, spikes at 10 and 30
    "gpt160m": Workload("gpt160m", _C2, r=192, grad_dtype="f32", steps=50,
                        k=64, sigma=0.1, tau=0.3, kind="spikes",
                        spike_steps=(10, 30), spike_scale=10.0, stream_id=2),
    # 1.3B-shaped set: 96 matrices, r = 512, bf16 gradients, fp32 state
    "gpt1p3b": Workload("gpt1p3b", _C3, r=512, grad_dtype="bf16", steps=20,
                        k=64, sigma=0.1, tau=0.5, stream_id=3),
    # rank sweep on one 4096 x 16384 fp32 matrix (r set per run)
    "sweep4096": Workload("sweep4096", ((4096, 16384),), r=64, grad_dtype="f32",
                          steps=6, k=32, sigma=0.1, tau=0.5, stream_id=4),
    # mixed flat / curved phases on the 1.3B-shaped set, 200 steps
    "mixed1p3b": Workload("mixed1p3b", _C3, r=512, grad_dtype="bf16", steps=200,
                          k=64, sigma=0.1, tau=0.5, kind="mixed", phase_len=25,
                          drift=0.01, sigma_flat=0.05, curved_scale=5.0,
                          stream_id=5),
}


def seed_for(stream_id: int, layer: int, step: int, salt: int = 0) -> int:
    """Deterministic 63-bit seed for one (stream, layer, step, salt) draw."""
    h = (stream_id * 0x9E3779B97F4A7C15 + layer * 0xBF58476D1CE4E5B9
         + step * 0x94D049BB133111EB + salt * 0x2545F4914F6CDD1D)
    return h & 0x7FFFFFFFFFFFFFFF


def _gen(device: torch.device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def random_orthonormal(n: int, r: int, seed: int) -> np.ndarray:
    """A dense n x r matrix with orthonormal columns, drawn without any QR.

    Columns are r distinct frequencies of the orthonormal DCT-II basis
    (entries sqrt(2/n) cos(pi (i + 1/2) k / n), and sqrt(1/n) for k = 0),
    with the rows randomly permuted and each column given a random sign.
    Permuting rows and flipping signs keeps the columns orthonormal.  Returned
    in float64; orthonormal to rounding (about 1e-15).
    """
    if not (1 <= r <= n):
        raise ValueError("need 1 <= r <= n")
    rng = np.random.Generator(np.random.PCG64(seed))
    freqs = rng.choice(n, size=r, replace=False)
    i = np.arange(n, dtype=np.float64)[:, None] + 0.5
    k = freqs.astype(np.float64)[None, :]
    C = np.cos(np.pi * i * k / n) * math.sqrt(2.0 / n)
    C[:, freqs == 0] = math.sqrt(1.0 / n)
    perm = rng.permutation(n)
    signs = rng.choice(np.array([-1.0, 1.0]), size=r)
    return C[perm] * signs[None, :]


def initial_state(w: Workload, layer: int, device="cpu", r: Optional[int] = None):
    """M0, X0 ~ N(0, init_std^2) in fp32 and Q0 (n x r, fp32, orthonormal)."""
    m, n = w.shapes[layer]
    r = w.r if r is None else r
    device = torch.device(device)
    g = _gen(device, seed_for(w.stream_id, layer, 0, salt=1))
    M0 = torch.randn((m, n), generator=g, device=device, dtype=torch.float32) * w.init_std
    X0 = torch.randn((m, n), generator=g, device=device, dtype=torch.float32) * w.init_std
    Q0 = torch.from_numpy(random_orthonormal(n, r, seed_for(w.stream_id, layer, 0, salt=2)))
    Q0 = Q0.to(torch.float32).to(device)
    return M0, X0, Q0


class GradientStream:
    """Per-layer gradient stream G_1, G_2, ... for one workload.

    ``next()`` returns the next gradient as a tensor of the workload's gradient
    dtype (fp32 or bf16; bf16 values are the round-to-nearest-even cast of the
    fp32 draw).  Steps are numbered from 1 as in the paper's Algorithm 2.
    """

    def __init__(self, w: Workload, layer: int, device="cpu"):
        self.w = w
        self.layer = layer
        self.device = torch.device(device)
        self.m, self.n = w.shapes[layer]
        self.step = 0
        self._U = None
        self._V = None

    def _randn(self, g, *shape):
        return torch.randn(shape, generator=g, device=self.device, dtype=torch.float32)

    def next(self) -> torch.Tensor:
        self.step += 1
        w, t = self.w, self.step
        m, n, k = self.m, self.n, w.k
        g = _gen(self.device, seed_for(w.stream_id, self.layer, t))
        sigma, scale = w.sigma, 1.0
        if w.kind == "lowrank":
            U, V = self._randn(g, m, k), self._randn(g, n, k)
        elif w.kind == "spikes":
            if t in w.spike_steps:
                g2 = _gen(self.device, seed_for(w.stream_id + 1000, self.layer, t))
                U, V = self._randn(g2, m, k), self._randn(g2, n, k)
                scale = w.spike_scale
            else:
                U, V = self._randn(g, m, k), self._randn(g, n, k)
        elif w.kind == "mixed":
            phase = (t - 1) // w.phase_len
            if phase % 2 == 0:          # flat: slowly drifting fixed subspace
                if self._U is None:
                    self._U, self._V = self._randn(g, m, k), self._randn(g, n, k)
                else:
                    self._U = self._U + w.drift * self._randn(g, m, k)
                    self._V = self._V + w.drift * self._randn(g, n, k)
                U, V = self._U, self._V
                sigma = w.sigma_flat
            else:                       # curved: redrawn subspace, larger magnitude
                U, V = self._randn(g, m, k), self._randn(g, n, k)
                scale = w.curved_scale
                self._U = None
        else:
            raise ValueError(f"unknown gradient kind {w.kind!r}")
        G = (U @ V.T) * scale + sigma * self._randn(g, m, n)
        if w.grad_dtype == "bf16":
            return G.to(torch.bfloat16)
        return G


def small_workload(m: int, n: int, r: int, *, steps: int = 6, k: int = 4,
                   grad_dtype: str = "f32", tau: float = 0.5, stream_id: int = 77,
                   layers: int = 1, **kw) -> Workload:
    """A one-shape workload of arbitrary size for tests (same recipe)."""
    return Workload(f"small{m}x{n}r{r}", ((m, n),) * layers, r=r, grad_dtype=grad_dtype,
                    steps=steps, k=k, tau=tau, stream_id=stream_id, **kw)
