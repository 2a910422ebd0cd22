"""Float64 CPU oracle of MKOR's per-step hot path.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
CPU-baseline leg of the benchmark, never by the product path.
"""
from .mkor_oracle import (  # noqa: F401
    EXACT, PAPER_EQ6, NORM_INF, NORM_MAXABS,
    NONFINITE_L, NONFINITE_R, NONFINITE_SCALE,
    Params, FactorStats, LayerStats,
    factor_norm, stabilize, sm_update, update_factor,
    precondition, rescale, layer_step, oracle_step, rank1_means, layer_step_rows,
)
