"""CPU oracle of the adaptive-depth MoE step.

TEST INFRASTRUCTURE ONLY. This package is the plain, slow, obviously
correct reference that the HIP path is checked against. Only the test
suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import it; the product path (the C-ABI library and its Python binding)
never does, and shares no code with it.
"""
from .trimmoe_oracle import (round_bf16, q_loss, route, substitutes, substitute_candidates,
                             as_candidates, decide,
                             expert_ffn, exit_confidence, layer_step,
                             stack_forward, init_state, model_from_inputs,
                             window_stats, feedback_update,
                             ACT_INACTIVE, ACT_EXEC, ACT_SKIP,
                             KIND_NONE, KIND_LOCAL, KIND_SUB, KIND_REMOTE)

__all__ = ["round_bf16", "q_loss", "route", "substitutes", "substitute_candidates",
           "as_candidates", "decide",
           "expert_ffn", "exit_confidence", "layer_step", "stack_forward",
           "init_state", "model_from_inputs", "window_stats", "feedback_update",
           "ACT_INACTIVE", "ACT_EXEC",
           "ACT_SKIP", "KIND_NONE", "KIND_LOCAL", "KIND_SUB", "KIND_REMOTE"]
