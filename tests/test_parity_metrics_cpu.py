"""CPU checks of the error measures the GPU parity tests apply: a mistake
confined to one tile of the update must fail them even where a norm over the
whole matrix would not see it.  The mistakes are planted in copies of the
oracle's own outputs (no GPU, no kernel)."""
import os
import sys

import numpy as np

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))

import oracle as O  # noqa: E402
from gpu_util import TILE_F32, TOL_BF16, TOL_F32, rel, sync_errors, tile_rel_max  # noqa: E402


def _case(m=2048, n=1536, r=64, seed=5):
    rng = np.random.default_rng(seed)
    B = rng.standard_normal((m, 16)) @ rng.standard_normal((16, n)) + 0.1 * rng.standard_normal((m, n))
    X0 = 0.02 * rng.standard_normal((m, n))
    Q0 = np.linalg.qr(rng.standard_normal((n, r)))[0]
    out = O.sync_update(B, X0, Q0, 0.95, 0.01)
    return B, X0, out


def test_one_wrong_tile_of_the_momentum_correction_is_caught():
    """Zeroing the correction in one 128 x 64 tile of a 2048 x 1536 layer
    (as a kernel that skipped that tile's epilogue would) moves the global
    relative error of dM by only 1/sqrt(384) = 0.05 and of M by about 2e-3:
    M passes even the bf16 bound.  The tile measure of dM sees 1.0 in that
    tile and fails both bounds."""
    B, X0, out = _case()
    Mg = out["M"].copy()
    Mg[128:256, 640:704] = B[128:256, 640:704]          # correction missing in one tile
    e = sync_errors(out, None, X0, B, Mg, out["X"], out["Q"], out["P"])
    assert e["err_M"] <= TOL_BF16                          # the norm of M alone misses it
    assert abs(e["tile_dM"] - 1.0) < 1e-12
    assert e["tile_dM"] > TOL_BF16 and e["tile_dM"] > TILE_F32
    clean = sync_errors(out, None, X0, B, out["M"], out["X"], out["Q"], out["P"])
    assert clean["tile_dM"] == 0.0 and clean["err_dM"] == 0.0


def test_one_wrong_tile_of_the_weight_update_is_caught():
    """The weight change of one tile taken from the neighbouring tile (a tile
    index mistake): the global dX error is about 0.07 (it would pass a loose
    global bound of 0.1), the tile measure is near 1.4."""
    B, X0, out = _case(seed=6)
    Xg = out["X"].copy()
    dX = out["X"] - X0
    Xg[0:128, 0:64] = X0[0:128, 0:64] + dX[128:256, 0:64]
    e = sync_errors(out, None, X0, B, out["M"], Xg, out["Q"], out["P"])
    assert e["err_dX"] < 0.1
    assert e["tile_dX"] > 1.0


def test_one_wrong_panel_of_P_is_caught():
    """A sign flip of one column inside one 64-row panel of P: tiny in the
    global norm of P at this size, an error of order one in that panel."""
    B, X0, out = _case(seed=7)
    Pg = out["P"].copy()
    Pg[64:128, 3] *= -1.0
    e = sync_errors(out, None, X0, B, out["M"], out["X"], out["Q"], Pg)
    assert e["err_P"] < 0.05
    assert e["tile_P"] > 0.1 and e["tile_P"] > TOL_BF16


def test_tile_measure_of_rounding_is_rounding():
    """fp32 rounding of every output is far inside the fp32 tile bound."""
    B, X0, out = _case(seed=8)
    f = lambda a: a.astype(np.float32).astype(np.float64)  # noqa: E731
    e = sync_errors(out, None, X0, B, f(out["M"]), f(out["X"]), f(out["Q"]), f(out["P"]))
    for k in ("tile_dM", "tile_P", "err_P", "err_Q", "err_M"):
        assert e[k] <= TOL_F32, (k, e[k])
    assert tile_rel_max(np.zeros((5, 5)), np.zeros((5, 5))) == 0.0
    assert rel(np.ones(3), np.ones(3)) == 0.0
