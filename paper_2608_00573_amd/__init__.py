"""MI355X-native adaptive-depth MoE step (TrimMoE, arXiv 2608.00573).

The compute path is libtrimmoe.so (hand-written HIP kernels for gfx950
behind a C ABI, include/trimmoe.h); ``abi`` is its ctypes binding.
"""
from . import abi
from .abi import (trimmoe_abi_version, trimmoe_status_str, trimmoe_workspace_size,
                  trimmoe_state_reset, trimmoe_layer_step, trimmoe_stack_forward,
                  TrimmoeError)

__all__ = ["abi", "trimmoe_abi_version", "trimmoe_status_str", "trimmoe_workspace_size",
           "trimmoe_state_reset", "trimmoe_layer_step", "trimmoe_stack_forward",
           "TrimmoeError"]
