"""The offline stage of Table I end to end: a calibration pass of the stack on
the GPU, the library's statistics, transition rows and placement from it,
against the oracle's own calibration pass of the same model and tokens; then
a look-ahead stack that runs on the calibrated placement and transitions."""
import numpy as np
import pytest
import torch

import oracle as O
from oracle import placement as P
from paper_2608_00573_amd import abi, offline
from synthgen import make_inputs, workload
from synthgen.servers import make_servers

from gpu_harness import GpuRun, check_invariants_gpu, gpu_state_np, gpu_trace_np, log, policy32

pytestmark = pytest.mark.gpu


def _oracle_record(inp):
    model = O.model_from_inputs(inp)
    pol = policy32(dict(inp["policy"], budget=0.0, p_exit=2.0, horizon=1))
    _, traces = O.stack_forward(model, pol, inp["h0"].double().numpy())
    rec = dict(target=np.stack([tr["target"] for tr in traces]),
               importance=np.stack([tr["importance"] for tr in traces]),
               xi=np.stack([tr["xi"] for tr in traces]))
    band = np.zeros(inp["h0"].shape[0], bool)
    for tr in traces:  # tokens whose routing is too close to call
        band |= tr["margin_logit"] <= 1e-5
    return rec, band


@pytest.mark.parametrize("over", [dict(n_layers=4, n_tokens=256),
                                  dict(n_layers=4, n_tokens=256, top_k=2, normalize_topk=1)],
                         ids=["top1", "top2"])
def test_calibration_tables_match_oracle(over):
    cfg = workload("tiny_fp32", **over)
    inp = make_inputs(cfg)
    g = GpuRun(inp)
    log(f"[offline] calibration pass T={cfg['n_tokens']} k={cfg['top_k']}")
    rec = offline.calibration_pass(g.mh.model, inp["policy"], inp["h0"].to(g.dev), g.ws)
    ref, band = _oracle_record(inp)
    ok = ~band
    assert np.array_equal(rec["target"][:, ok], ref["target"][:, ok])
    assert np.allclose(rec["importance"], ref["importance"], rtol=1e-5, atol=1e-7)
    assert np.array_equal(np.isnan(rec["xi"]), np.isnan(ref["xi"]))
    assert np.allclose(rec["xi"], ref["xi"], rtol=1e-4, atol=1e-7, equal_nan=True)

    p_j = float(np.float32(inp["policy"]["p_exit"]))
    theta = [L["theta"] for L in inp["layers"]]
    tab = offline.offline_tables(rec, p_j, theta, cfg["n_experts"], 4)
    ex_ref = P.calibration_exit_layers(ref["xi"], p_j)
    near = np.any(np.abs(ref["xi"] - p_j) <= 1e-5, axis=0) | band   # gate too close to call
    assert np.array_equal(tab["exit_layer"][~near], ex_ref[~near])
    log(f"[offline] band tokens {int(band.sum())}, near-gate tokens {int(near.sum())}, "
        f"pi {np.round(tab['pi'], 3).tolist()}")
    if not near.any():
        # every decision clear: the statistics are those of the oracle's pass
        want = P.calibration_stats(ref["target"], ref["importance"], ex_ref,
                                   np.asarray(theta, np.float64), cfg["n_experts"])
        imp_close = np.any(np.abs(ref["importance"] - np.asarray(theta)[:, None]) <= 1e-5)
        for key, w in zip(("pi", "act", "sigma", "lam"), want):
            if key in ("pi", "act") or not imp_close:
                assert np.array_equal(tab[key], w), key
        to, pr = P.transition_rows(ref["target"], ex_ref, cfg["n_experts"], 4)
        assert np.array_equal(tab["trans_to"], to)
        assert np.array_equal(tab["trans_p"], pr.astype(np.float32))
    assert tab["pi"][0] == 1.0 and np.all(np.diff(tab["pi"]) <= 0)


def test_stack_runs_on_calibrated_placement_and_transitions():
    # Mixtral-like routing (8 experts top-2) at a small width: calibrate on
    # 512 tokens, place replicas over 10 servers with memory ratio 2, give
    # the device server 0's experts and the calibrated transitions, and run
    # a look-ahead stack on fresh tokens
    cfg = workload("tiny_fp32", n_layers=6, top_k=2, normalize_topk=1, n_tokens=512,
                   horizon=3, t_remote=2.0, omega_t=0.2)
    inp = make_inputs(cfg)
    g = GpuRun(inp)
    rec = offline.calibration_pass(g.mh.model, inp["policy"], inp["h0"].to(g.dev), g.ws)
    theta = [L["theta"] for L in inp["layers"]]
    tab = offline.offline_tables(rec, inp["policy"]["p_exit"], theta, cfg["n_experts"], 4)
    srv = make_servers(cfg, n_servers=10, memory_ratio=2.0)
    x, added = offline.place(tab, srv)
    assert P.check_deployment(x, srv["nbytes"], srv["capacity"]) == []
    assert added > 0 and np.all(x >= srv["x0"])
    home = x[srv["home"]]
    log(f"[offline] {added} replicas; server 0 holds {home.sum(axis=1).tolist()} experts per layer")
    layers = []
    for l, L in enumerate(g.layers):
        L = dict(L)
        L["local_mask"] = torch.from_numpy(home[l].copy()).to(g.dev)
        if l < cfg["n_layers"] - 1:
            L["trans_to"] = torch.from_numpy(tab["trans_to"][l].copy()).to(g.dev)
            L["trans_p"] = torch.from_numpy(tab["trans_p"][l].copy()).to(g.dev)
        layers.append(L)
    g2 = GpuRun(inp, layers_dev=layers)
    from synthgen.inputs import make_tokens
    h = make_tokens(cfg, 4242)
    st, tr = g2.stack(h0=h)
    gst, gtr = gpu_state_np(st), gpu_trace_np(tr)
    check_invariants_gpu(cfg, policy32(inp["policy"]), gst, gtr)
    # the placement decides where slots run: executed slots are local or
    # remote exactly as server 0's row says
    for l in range(cfg["n_layers"]):
        run = gtr["action"][l] == O.ACT_EXEC
        kinds, ex = gtr["kind"][l][run], gtr["exec"][l][run]
        assert np.all(home[l][ex[kinds == O.KIND_LOCAL]] == 1)
        assert np.all(home[l][ex[kinds == O.KIND_SUB]] == 1)
        assert np.all(home[l][ex[kinds == O.KIND_REMOTE]] == 0)
