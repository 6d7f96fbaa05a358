"""The torch.optim front end on the GPU: one step of a two-matrix model
against the float64 oracle (same gradients, same initial Q), and a short
training run on synthetic data whose loss must fall."""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

import oracle as O  # noqa: E402
from gpu_util import f32, rel  # noqa: E402
from paper_2512_13728_amd.optim import CurvaDion, orthonormal_start  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield


def _model(seed):
    torch.manual_seed(seed)
    return torch.nn.Sequential(torch.nn.Linear(64, 96, bias=False), torch.nn.Tanh(),
                               torch.nn.Linear(96, 32, bias=False)).to(DEV)


def test_step_matches_oracle():
    net = _model(0)
    mats = [net[0].weight, net[2].weight]
    opt = CurvaDion(mats, lr=0.02, momentum=0.95, rank=8, tau=0.5, seed=5)
    x = torch.randn(256, 64, device=DEV)
    y = torch.randn(256, 32, device=DEV)
    states = [O.OracleLayer.from_arrays(np.zeros(tuple(p.shape)), p.detach().cpu().double().numpy(),
                                        orthonormal_start(p.shape[1], 8, "cpu", seed=5 + k).double().numpy())
              for k, p in enumerate(mats)]
    for t in range(3):
        opt.zero_grad()
        loss = torch.nn.functional.mse_loss(net(x), y)
        loss.backward()
        grads = [p.grad.detach().cpu().double().numpy() for p in mats]
        res = O.group_step(states, grads, f32(0.95), f32(0.02), 0.5)
        opt.step()
        torch.cuda.synchronize()
        rm, flag = opt.last[torch.float32]
        print(f"step {t + 1}: rmmc {rm:.4g} (oracle {res['g']:.4g}) sync {flag}", flush=True)
        assert abs(res["g"] - 0.5) / 0.5 > 1e-4, "decision too close to tau"
        assert flag == res["flag"], (t, rm, res["g"])
        for p, L in zip(mats, states):
            assert rel(p.detach().cpu().double().numpy(), L.X) <= 1e-5
            assert rel(opt.state[p]["M"].cpu().double().numpy(), L.M) <= 1e-5
            # continue from the GPU state (teacher forcing)
            L.X = p.detach().cpu().double().numpy()
            L.M = opt.state[p]["M"].cpu().double().numpy()
            L.Q = opt.state[p]["Q"].cpu().double().numpy()


def test_training_reduces_loss():
    """A two-layer tanh network fit to a fixed random teacher on synthetic
    inputs: 150 steps of CurvaDion (rank 16, tau = 0.5) lower the loss by more
    than a quarter (most steps take the skip branch, SGD on the local
    gradient); the gate syncs on some steps and skips the others."""
    torch.manual_seed(1)
    teacher = _model(2)
    net = _model(3)
    opt = CurvaDion([net[0].weight, net[2].weight], lr=0.05, momentum=0.9, rank=16, tau=0.5)
    sched = torch.optim.lr_scheduler.LambdaLR(opt, lambda s: 1.0 if s < 100 else 0.5)
    losses, syncs = [], 0
    for t in range(150):
        x = torch.randn(512, 64, device=DEV)
        with torch.no_grad():
            y = teacher(x)
        opt.zero_grad()
        loss = torch.nn.functional.mse_loss(net(x), y)
        loss.backward()
        opt.step()
        sched.step()
        losses.append(loss.item())
        syncs += int(opt.last[torch.float32][1])
    first, last = np.mean(losses[:10]), np.mean(losses[-10:])
    print(f"loss {first:.4g} -> {last:.4g}, {syncs} syncs in 150 steps", flush=True)
    assert last < 0.75 * first
    assert 1 <= syncs < 150
