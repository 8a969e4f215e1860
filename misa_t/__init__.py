"""CPU replay of MISA-T's routing-layer controller (Sec. 4 of "Scheduling Mixed RL Rollouts Beyond Prefix
Locality"): adaptive session admission, workload-aware class caps and residency-time-weighted quotas,
driving the paged-KV attention library with synthetic mixes of RLVR, RLHF and agentic rollouts.

This is a harness around the library, not part of it: the package ``paper_2608_11152_amd`` never imports
it, and ``bench.py`` does not time it.
"""
from .controller import (CLASSES, ClassEstimator, Controller, base_cap, block_time_demand, drain_times,
                         hit_degradation, hold_preferable, prefill_cost, space_caps, spatial_demand, time_caps)

__all__ = ["CLASSES", "ClassEstimator", "Controller", "base_cap", "block_time_demand", "drain_times",
           "hit_degradation", "hold_preferable", "prefill_cost", "space_caps", "spatial_demand", "time_caps"]
