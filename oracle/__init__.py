"""fp64 CPU oracle of the Jorge optimizer step (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
package; the GPU library never imports it.
"""
from .jorge_oracle import (BETA_CLAMPED, BETA_DYNAMIC, BETA_FIXED, SERIES_C1, SERIES_C2,
                           SERIES_C3, JorgeOracle, LayerState, beta_select, binomial_series_coefficient,
                           gram_factors, init_factor, precondition, update_factor,
                           update_weights)

__all__ = ["BETA_CLAMPED", "BETA_DYNAMIC", "BETA_FIXED", "SERIES_C1", "SERIES_C2",
           "SERIES_C3", "JorgeOracle", "LayerState", "beta_select", "binomial_series_coefficient",
           "gram_factors", "init_factor", "precondition", "update_factor", "update_weights"]
