"""Seeded synthetic inputs shared by the GPU path's tests/bench and the CPU oracle.

This package holds workload descriptions (plain parameter values) and seeded random
input generators only. It contains none of the simulator's, policy's or return
computation's arithmetic: each side derives its own constants from these values.
"""
from .presets import (PRESETS, preset, trace_preset, burst_preset, baseline_preset,  # noqa: F401
                      attn_preset)
from .gen import (seeded_actions, seeded_obs, seeded_rewards_values,  # noqa: F401
                  seeded_weights_f32)
