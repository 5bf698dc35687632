"""Offline stage of Table I on top of the library: a full-depth calibration
pass on the GPU, then the statistics, transition rows and replica placement
(host C++ behind the C ABI).  Argument marshalling and call order only."""
from __future__ import annotations

import numpy as np
import torch

from . import abi

# a confidence requirement no softmax or sigmoid reaches: nothing exits
_NEVER = 2.0


def calibration_pass(model: abi.Model, policy: dict, h0: torch.Tensor, workspace: torch.Tensor):
    """Table I, line 1: run the stack at full depth with exact execution
    (budget 0: no skip or substitution; no exit) over the calibration tokens
    h0 (on the GPU) and return the host record (target [N, Q, k] int16,
    importance [N, Q] float32, xi [N, Q] float32, NaN where not evaluated)."""
    N, k = model.n_layers, model.top_k
    st = abi.StateBuffers(h0.clone())
    tr = abi.TraceBuffers(N, h0.shape[0], k, h0.device)
    cal = dict(policy, budget=0.0, p_exit=_NEVER, horizon=1)
    abi.trimmoe_stack_forward(model, abi.make_policy(**cal), st.state, tr.trace, workspace)
    torch.cuda.synchronize()
    return dict(target=tr.target.cpu().numpy(), importance=tr.importance.cpu().numpy(),
                xi=tr.xi.cpu().numpy())


def offline_tables(record: dict, p_exit: float, theta, n_experts: int, trans_b: int):
    """Exit layers at the confidence requirement p_exit, the Sec. IV-C
    statistics (pi, act, sigma, lambda) and the Eq. (38) transition rows."""
    ex = abi.trimmoe_calib_exit_layers(record["xi"], p_exit)
    pi, act, sigma, lam = abi.trimmoe_calib_stats(record["target"], record["importance"], ex,
                                                  np.asarray(theta, np.float32), n_experts)
    to, pr = abi.trimmoe_calib_transitions(record["target"], ex, n_experts, trans_b)
    return dict(exit_layer=ex, pi=pi, act=act, sigma=sigma, lam=lam, trans_to=to, trans_p=pr)


def place(tables: dict, servers: dict):
    """Table I, lines 9-13 over a server scenario (keys nbytes, capacity,
    bandwidth, latency, rho, z, x0); returns (x [M, N, E], replicas added)."""
    return abi.trimmoe_place_replicas(tables["lam"], servers["rho"], servers["z"],
                                      servers["nbytes"], servers["capacity"],
                                      servers["bandwidth"], servers["latency"], servers["x0"])
