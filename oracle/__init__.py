"""float64 CPU oracle of the speculate-reuse-repair decode path.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
bench's CPU-baseline leg, never by the product library or its Python binding.
"""
from .prr_oracle import *  # noqa: F401,F403
from .prr_oracle import (  # noqa: F401
    THETA_GRID, attend, calibrate, calibration_objective, criticality_mean, criticality_minmax,
    decision_keys, ema_init, ema_predict, ema_update, hit_rate, merge_states, merge_two,
    missed_and_wasted, page_metadata_mean, page_metadata_minmax, page_tokens, predicted_set,
    repair_block, representative_query, select_topk, serial_step, speculate_then_repair,
)
