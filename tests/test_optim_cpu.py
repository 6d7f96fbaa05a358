"""CPU checks of the torch.optim front end (argument handling only; the
steps themselves run on the GPU, see test_gpu_optim.py)."""
import math

import pytest
import torch

from paper_2512_13728_amd.optim import CurvaDion, orthonormal_start


def test_rejects_non_matrices_and_unknown_policy():
    with pytest.raises(ValueError):
        CurvaDion([torch.nn.Parameter(torch.zeros(8))])
    with pytest.raises(ValueError):
        CurvaDion([torch.nn.Parameter(torch.zeros(4, 4, dtype=torch.float64))])
    with pytest.raises(ValueError):
        CurvaDion([torch.nn.Parameter(torch.zeros(4, 4))], policy="sometimes")


def test_orthonormal_start_is_orthonormal_without_qr():
    for n, r in ((16, 4), (300, 37), (64, 64)):
        q = orthonormal_start(n, r, "cpu", seed=3).double()
        err = (q.T @ q - torch.eye(r, dtype=torch.float64)).abs().max().item()
        assert err < 1e-6, (n, r, err)
    a, b = orthonormal_start(32, 5, "cpu", seed=1), orthonormal_start(32, 5, "cpu", seed=1)
    assert torch.equal(a, b)


def test_rank_fraction_of_min_dimension():
    opt = CurvaDion([torch.nn.Parameter(torch.zeros(768, 2304))], rank=0.125)
    assert opt._rank(768, 2304) == 96 and opt._rank(3072, 768) == 96
    opt = CurvaDion([torch.nn.Parameter(torch.zeros(8, 8))], rank=3)
    assert opt._rank(8, 8) == 3 and opt._rank(2, 8) == 2
    assert math.isclose(opt.param_groups[0]["lr"], 0.02)
