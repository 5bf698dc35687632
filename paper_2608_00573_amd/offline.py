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


def calibration_hidden_states(model: abi.Model, policy: dict, h0: torch.Tensor,
                              workspace: torch.Tensor):
    """Table I, line 1, keeping the representation after every layer: the
    full-depth exact pass one layer at a time; returns [h after layer l] for
    l = 0 .. N - 1 (on the GPU, the model's dtype)."""
    cal = abi.make_policy(**dict(policy, budget=0.0, p_exit=_NEVER, horizon=1))
    st = abi.StateBuffers(h0.clone())
    abi.trimmoe_state_reset(model, st.state)
    hs = []
    for l in range(model.n_layers):
        abi.trimmoe_layer_step(model, l, cal, st.state, None, workspace)
        hs.append(st.h.clone())
    torch.cuda.synchronize()
    return hs


def consistency_labels(hs, w_head: torch.Tensor):
    """Eq. (22) for layers 0 .. N - 2: 1 where the output head's prediction
    of the layer's representation equals its prediction at full depth."""
    final = abi.trimmoe_head_argmax(w_head, hs[-1])
    return [abi.trimmoe_consistency_labels(abi.trimmoe_head_argmax(w_head, h), final)
            for h in hs[:-1]]


def train_sigmoid_heads(hs, labels, epochs: int, lr: float):
    """Table I, lines 3-4: one sigmoid exit head per layer 0 .. N - 2 trained
    on BCE (Eq. (23)) from zero; returns [(w fp32 [d], c fp32 [1], losses)]."""
    out = []
    for h, y in zip(hs, labels):
        w = torch.zeros(h.shape[1], dtype=torch.float32, device=h.device)
        c = torch.zeros(1, dtype=torch.float32, device=h.device)
        loss = torch.zeros(max(epochs, 1), dtype=torch.float32, device=h.device)
        abi.trimmoe_train_exit_head(h, y, epochs, lr, w, c, loss)
        out.append((w, c, loss[:epochs]))
    torch.cuda.synchronize()
    return out
