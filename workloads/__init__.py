"""Seeded synthetic inputs for the Shifted Non-Local Search path.

This module is shared by the oracle-side tests and the HIP-side tests and
benchmark.  It only synthesises inputs (videos, flows, upstream gradients) and
describes the search settings; it computes nothing of the method itself
(no search, no top-k, no aggregation).
"""
from .synth import (  # noqa: F401
    CONFIGS, N_MAIN_CONFIGS, config_index, config_params, make_config, make_motion_video, small_params,
)
