"""Float64 CPU oracle for the CurvaDion step (test infrastructure only).

Imported only by the tests, the smoke check and the benchmark's CPU-baseline
leg.  The library never imports it.
"""
from .curvadion_oracle import *  # noqa: F401,F403
from .curvadion_oracle import (OracleLayer, group_step, buffer_update, frobenius_norm, rmmc,
                               gate, orthogonalize, column_normalize, power_iteration,
                               sync_update, local_update, POLICY_RMMC, POLICY_ALWAYS_SYNC,
                               POLICY_NEVER_SYNC, POLICY_EVERY_H, COLNORM_FLOOR)
