"""Seeded synthetic inputs for the adaptive-depth MoE step.

This package only draws numbers: a counter-based random generator, the
workload shapes, and the recipe that turns both into model weights, hidden
states, placement masks and calibration scalars. It holds none of the
method's arithmetic (no routing, no substitution, no skip or exit rule, no
expert FFN), so the CPU oracle and the HIP path can both take their inputs
from it without sharing any code of the method.
"""
from .rng import splitmix64_stream, normal_f32, uniform_f64, key_for
from .configs import WORKLOADS, workload
from .inputs import make_inputs, mid_state

__all__ = ["splitmix64_stream", "normal_f32", "uniform_f64", "key_for",
           "WORKLOADS", "workload", "make_inputs", "mid_state"]
