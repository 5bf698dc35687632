"""GPU parity of the look-ahead decision (Sec. V-E, Eq. (38)-(40), H > 1).

Whole stacks through trimmoe_stack_forward against the oracle, on a recipe
where the look-ahead changes decisions (remote slots cost 2 local ones and
the delay weight is 0.2, so spending budget now competes with saving it for
later layers).  fp32 stacks use a 1e-5 band for importance and cost margins
and 1e-7 for budget comparisons (both sides compute D-hat from the same
stored Sim values); bf16 stacks keep the 1e-3 band and 1e-4 for budgets.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_00573_amd import abi
from synthgen import make_inputs, workload

from gpu_harness import (GpuRun, check_invariants_gpu, compare_stack, gpu_state_np,
                         gpu_trace_np, log, oracle_run, policy32)

pytestmark = pytest.mark.gpu

RECIPE = dict(t_remote=2.0, omega_t=0.2)


def _stack(cfg, band, band_budget, budget_tok=None, p_exit_tok=None):
    inp = make_inputs(cfg)
    log(f"[lookahead] {cfg['dtype']} T={cfg['n_tokens']} N={cfg['n_layers']} "
        f"k={cfg['top_k']} B={cfg['trans_support']} H={cfg['horizon']}")
    g = GpuRun(inp)
    st, tr = g.stack(budget_tok=budget_tok, p_exit_tok=p_exit_tok)
    gst, gtr = gpu_state_np(st), gpu_trace_np(tr)
    ref_state, ref_traces = oracle_run(inp, token_budget=budget_tok, token_p_exit=p_exit_tok)
    stats = compare_stack(cfg, ref_state, ref_traces, gst, gtr, band=band,
                          band_budget=band_budget)
    check_invariants_gpu(cfg, policy32(inp["policy"]), gst, gtr, budget_tok, p_exit_tok)
    log(f"[lookahead] ok {stats}")
    return inp, g, gtr, stats


def _decisions_differ(g, gtr, inp):
    """(token, layer) decisions of the GPU at H = 1 that differ from gtr's."""
    st1, tr1 = g.stack(pol=dict(inp["policy"], horizon=1))
    t1 = gpu_trace_np(tr1)
    return int(((t1["action"] != gtr["action"]) | np.any(t1["exec"] != gtr["exec"], axis=2)).sum())


def test_top1_horizon3():
    cfg = workload("tiny_fp32", n_layers=4, horizon=3, **RECIPE)
    inp, g, gtr, stats = _stack(cfg, 1e-5, 1e-7)
    assert stats["excluded_tokens"] <= 4
    assert _decisions_differ(g, gtr, inp) >= 5


def test_top2_horizon3():
    cfg = workload("tiny_fp32", n_layers=4, top_k=2, normalize_topk=1, horizon=3, **RECIPE)
    inp, g, gtr, stats = _stack(cfg, 1e-5, 1e-7)
    assert stats["excluded_tokens"] <= 6
    assert _decisions_differ(g, gtr, inp) >= 5


def test_horizon4_full_transition_rows():
    # H = 4 (three later layers) and 8-entry rows over 8 experts
    cfg = workload("tiny_fp32", n_layers=5, horizon=4, trans_support=8, **RECIPE)
    _, _, _, stats = _stack(cfg, 1e-5, 1e-7)
    assert stats["excluded_tokens"] <= 4 and stats["compared"] > 150


def test_ragged_tokens_horizon2():
    # 333 tokens: eleven route blocks, the last one ragged
    cfg = workload("tiny_fp32", n_layers=3, n_tokens=333, top_k=2, normalize_topk=1, horizon=2,
                   **RECIPE)
    _, _, _, stats = _stack(cfg, 1e-5, 1e-7)
    assert stats["compared"] > 600


@pytest.mark.parametrize("H", [2, 3])
def test_bf16_swiglu_top2_shared(H):
    cfg = workload("tiny_fp32", dtype="bf16", act="swiglu", top_k=2, normalize_topk=1,
                   n_layers=4, n_tokens=512, d_model=128, d_ff=256, d_ff_shared=128,
                   horizon=H, **RECIPE)
    _, _, _, stats = _stack(cfg, 1e-3, 1e-4)
    assert stats["compared"] >= 0.8 * 512


def test_top4_sixty_experts_two_entry_rows():
    # Qwen-like routing: 60 experts top-4 (one candidate per remote slot: 17
    # candidate actions, 16 tuples per level with 2-entry rows), horizon 2
    cfg = workload("tiny_fp32", n_layers=3, n_experts=60, n_local=20, top_k=4, horizon=2,
                   trans_support=2, n_tokens=128, la_subs=1, **RECIPE)
    _, _, _, stats = _stack(cfg, 1e-5, 1e-7)
    assert stats["compared"] > 200


def test_validation_of_look_ahead_limits():
    cfg = workload("tiny_fp32", n_layers=3, horizon=2)
    inp = make_inputs(cfg)
    g = GpuRun(inp)
    st = abi.StateBuffers(inp["h0"].to(g.dev).clone())
    for pol, err in ((dict(inp["policy"], horizon=5), abi.TrimmoeError),
                     (dict(inp["policy"], horizon=0), abi.TrimmoeError),
                     (dict(inp["policy"], la_subs=0), abi.TrimmoeError),
                     (dict(inp["policy"], la_subs=5), abi.TrimmoeError)):
        with pytest.raises(err):
            abi.trimmoe_stack_forward(g.mh.model, g.policy(pol), st.state, None, g.ws)
    # transitions missing on a layer the decision reads
    layers = [dict(L) for L in g.layers]
    layers[0]["trans_to"] = None
    mh = abi.model_handle(cfg, layers)
    with pytest.raises(abi.TrimmoeError):
        abi.trimmoe_stack_forward(mh.model, g.policy(), st.state, None, g.ws)
    # ...but layer 1 alone at H = 2 reads only P_1
    abi.trimmoe_layer_step(mh.model, 1, g.policy(), st.state, None, g.ws)
    torch.cuda.synchronize()


def test_256_experts_look_ahead_tables_beyond_64k_lds():
    # 256 experts top-2 with 8-entry rows, two local candidates per remote
    # slot and two later layers: the route block's look-ahead tables and
    # logits need more than 64 KB of LDS (the launch raises the kernel's
    # dynamic-LDS limit)
    cfg = workload("tiny_fp32", n_layers=3, n_experts=256, n_local=128, top_k=2,
                   normalize_topk=1, horizon=3, trans_support=8, n_tokens=32, la_subs=2,
                   **RECIPE)
    _, _, _, stats = _stack(cfg, 1e-5, 1e-7)
    assert stats["compared"] >= 40


def test_per_token_budgets_and_requirements_horizon3():
    # the recursion spends each token's own budget: zero for every third
    # token (exact execution only), generous for others
    cfg = workload("tiny_fp32", n_layers=4, top_k=2, normalize_topk=1, horizon=3, **RECIPE)
    T = cfg["n_tokens"]
    budget_tok = np.choose(np.arange(T) % 3, [0.0, 0.02, 0.05]).astype(np.float32)
    p_exit_tok = np.where(np.arange(T) % 4 == 0, 2.0, 0.5).astype(np.float32)
    _, _, gtr, stats = _stack(cfg, 1e-5, 1e-7, budget_tok, p_exit_tok)
    assert stats["excluded_tokens"] <= 6
    assert np.all(gtr["kind"][:, np.arange(T) % 3 == 0] != O.KIND_SUB)


@pytest.mark.parametrize("k,H", [(1, 3), (2, 2), (2, 3)])
def test_every_local_candidate_weighed(k, H):
    # a budget that admits most local substitutes (Q up to ~0.5 fits within
    # 0.9): each remote slot weighs all four local candidates at every level
    cfg = workload("tiny_fp32", n_layers=4, top_k=k, normalize_topk=int(k > 1), horizon=H,
                   budget=0.9, la_subs=4, **RECIPE)
    _, _, gtr, stats = _stack(cfg, 1e-5, 1e-7)
    assert stats["compared"] >= 100
    assert (gtr["kind"] == O.KIND_SUB).sum() >= 50


def test_look_ahead_takes_a_higher_loss_substitute():
    # planted on every layer: remote experts 4 and 5 have two local
    # candidates, 0 (Q 0.001) and 1 (Q 0.002); expert 0 moves on to remote
    # expert 6, which has no candidate and cannot be skipped (theta 0),
    # expert 1 to local expert 2.  At H = 2 a slot routed to 4 or 5 runs
    # expert 1 (0.5 + 0.05 + 0.5 = 1.05 against 0.525 + 50 for expert 0);
    # at H = 1, or with one candidate, expert 0
    cfg = workload("tiny_fp32", n_layers=3, horizon=2, la_subs=4, sim_min=-0.5,
                   trans_support=2, n_local=4)
    inp = make_inputs(cfg)
    E, B = cfg["n_experts"], 2
    sim = -np.ones((E, E), np.float32)
    np.fill_diagonal(sim, 1.0)
    for e in (4, 5):
        sim[e][0], sim[e][1] = 1.0 - 2 * 0.001, 1.0 - 2 * 0.002
    nxt = {0: 6, 1: 2, 2: 2, 3: 3, 4: 6, 5: 6, 6: 6, 7: 7}
    to = np.full((E, B), -1, np.int16)
    pr = np.zeros((E, B), np.float32)
    for e, t in nxt.items():
        to[e][0], pr[e][0] = t, 1.0
    for L in inp["layers"]:
        L["sim"] = torch.from_numpy(sim.copy())
        L["local_mask"] = torch.tensor([1, 1, 1, 1, 0, 0, 0, 0], dtype=torch.uint8)
        L["theta"] = 0.0
        if L.get("trans_to") is not None:
            L["trans_to"] = torch.from_numpy(to.copy())
            L["trans_p"] = torch.from_numpy(pr.copy())
    g = GpuRun(inp)
    st, tr = g.stack()
    gst, gtr = gpu_state_np(st), gpu_trace_np(tr)
    ref_state, ref_traces = oracle_run(inp)
    compare_stack(cfg, ref_state, ref_traces, gst, gtr, band=1e-5, band_budget=1e-7)
    l0 = gtr["target"][0][:, 0]
    routed = (l0 == 4) | (l0 == 5)
    assert routed.sum() >= 4
    assert np.all(gtr["exec"][0][routed, 0] == 1)  # the higher-loss candidate
    _, tr1 = g.stack(pol=dict(inp["policy"], la_subs=1))
    assert np.all(gpu_trace_np(tr1)["exec"][0][routed, 0] == 0)
