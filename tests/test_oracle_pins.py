"""Pins of the CPU oracle against what the paper and mathematics fix.

None of these retypes the oracle's own formulas: each checks it against a
library routine, a brute-force search over the definition, a closed form,
a hand-derived example, or an invariant the paper proves.
"""
import itertools
import json
import math
import os
import random

import numpy as np
import pytest
import torch

import oracle as O
from synthgen import make_inputs, workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- rounding --
def test_round_bf16_matches_torch_on_fp32_values():
    g = torch.Generator().manual_seed(0)
    x = (torch.randn(200000, generator=g) * torch.exp(torch.randn(200000, generator=g) * 4))
    x = x.to(torch.float32)
    want = x.to(torch.bfloat16).to(torch.float64).numpy()
    got = O.round_bf16(x.to(torch.float64).numpy())
    assert np.array_equal(got, want)


def test_round_bf16_ties_to_even_by_hand():
    # 1 + 2^-8 lies exactly between 1 and 1 + 2^-7: ties to even -> 1
    assert O.round_bf16(np.array([1.0 + 2.0 ** -8]))[0] == 1.0
    # 1 + 3*2^-8 lies between 1+2^-7 (odd) and 1+2^-6 (even) -> 1 + 2^-6
    assert O.round_bf16(np.array([1.0 + 3 * 2.0 ** -8]))[0] == 1.0 + 2.0 ** -6
    # just above the tie rounds up
    assert O.round_bf16(np.array([1.0 + 2.0 ** -8 + 2.0 ** -40]))[0] == 1.0 + 2.0 ** -7
    assert O.round_bf16(np.array([-3.0]))[0] == -3.0
    assert O.round_bf16(np.array([0.0]))[0] == 0.0


def test_round_bf16_below_the_normal_range():
    # bf16 subnormals are the multiples of 2^-133 below 2^-126; IEEE rounding
    # to nearest, ties to even, reaches them and zero
    u = 2.0 ** -133
    cases = [(8 * u, 8 * u), (2.5 * u, 2 * u), (3.5 * u, 4 * u), (-2.5 * u, -2 * u),
             (0.5 * u, 0.0), (0.5 * u * (1 + 2.0 ** -20), u), (2.0 ** -140, 0.0),
             (1e-300, 0.0), (127.75 * u, 128 * u), (2.0 ** -126 * (1 - 2.0 ** -30), 2.0 ** -126)]
    got = O.round_bf16(np.array([c for c, _ in cases]))
    assert np.array_equal(got, np.array([w for _, w in cases]))
    assert np.signbit(O.round_bf16(np.array([-0.25 * u]))[0])  # -0
    # fp32 subnormal inputs against torch's float -> bfloat16 conversion
    g = torch.Generator().manual_seed(1)
    bits = torch.randint(1, 1 << 23, (50000,), generator=g, dtype=torch.int32)
    x = bits.view(torch.float32) * torch.where(torch.rand(50000, generator=g) < 0.5, -1.0, 1.0)
    want = x.to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(O.round_bf16(x.to(torch.float64).numpy()), want)
    with pytest.raises(ValueError):
        O.round_bf16(np.array([np.inf]))


# -------------------------------------------------------------- Eq. (3) -----
def test_q_loss_closed_forms():
    assert O.q_loss(1.0, 1.0) == 0.0            # identical experts
    assert O.q_loss(-1.0, 1.0) == 1.0           # opposite experts: (1+1)/2
    assert O.q_loss(0.0, 1.0) == 0.5
    assert O.q_loss(0.0, 4.0) == 1.0            # phi clipped to 1
    assert O.q_loss(0.96, 1.0) == pytest.approx(0.02)


# -------------------------------------------------------------- Eq. (4) -----
@pytest.mark.parametrize("seed", range(20))
def test_route_brute_force(seed):
    rs = np.random.RandomState(seed)
    E = rs.randint(2, 9)
    k = rs.randint(1, E + 1)
    z = rs.randn(E)
    if seed % 3 == 0:  # force ties
        z = np.round(z * 2) / 2
    S, w, I, p, margin = O.route(z, k, normalize=False)
    # brute force: the k-subset with the largest logit sum; among equal
    # sums the lexicographically smallest sorted id tuple (ties to lower id)
    best = max(itertools.combinations(range(E), k),
               key=lambda c: (sum(z[list(c)]), [-e for e in c]))
    assert sorted(S) == sorted(best)
    # rank order: logits non-increasing, equal logits by increasing id
    for a, b in zip(S, S[1:]):
        assert z[a] > z[b] or (z[a] == z[b] and a < b)
    soft = torch.softmax(torch.tensor(z), 0).numpy()
    assert I == pytest.approx(float(soft[S].sum()), rel=1e-12)
    assert w == pytest.approx([float(soft[e]) for e in S], rel=1e-12)
    S2, w2, I2, _, _ = O.route(z, k, normalize=True)
    assert sum(w2) == pytest.approx(1.0, rel=1e-12)
    assert I2 == pytest.approx(I)
    if k < E:
        srt = np.sort(z)[::-1]
        assert margin <= srt[k - 1] - srt[k] + 1e-15


# ---------------------------------------------- Eq. (31)-(35), (40) brute ---
def _brute_force_decision(S, w, I, local, sim, d_hat, budget, theta, slope, pol):
    """Full Eq. (34) action set at H = 1, searched exhaustively.

    Each routed slot may run its target (wherever it is deployed: local or a
    remote round trip) or ANY local expert that is a feasible substitute
    (Sim >= sim_min, k != target); skip is a further action when admitted
    by Eq. (35) and the importance threshold.  Costs per Eq. (31)/(32).
    Returns (min cost, action, set of optimal assignments).
    """
    wt = pol["omega_t"]
    wd = 1 - wt
    choices = []
    for e in S:
        opts = [(e, 0.0, pol["t_local"] if local[e] else pol["t_remote"])]
        for j in range(len(local)):
            if j != e and local[j] and sim[e][j] >= pol["sim_min"]:
                q = min(1.0, pol["phi_scale"] * (1 - sim[e][j]) / 2)
                opts.append((j, q, pol["t_local"]))
        choices.append(opts)
    best = math.inf
    best_assign = []
    all_local_feasible = False
    for combo in itertools.product(*choices):
        sq = sum(c[1] for c in combo)
        if d_hat + sq > budget:
            continue
        if all(c[2] == pol["t_local"] for c in combo):
            all_local_feasible = True
        f = wt * sum(c[2] for c in combo) + (wd * sq / budget if budget > 0 else 0.0)
        if f < best - 1e-12:
            best, best_assign = f, [combo]
        elif abs(f - best) <= 1e-12:
            best_assign.append(combo)
    lam = min(1.0, slope * I)
    if (not all_local_feasible) and I <= theta and d_hat + lam <= budget:
        fs = wd * lam / budget if budget > 0 else 0.0
        if fs < best:
            return fs, O.ACT_SKIP, []
    return best, O.ACT_EXEC, best_assign


@pytest.mark.parametrize("seed", range(300))
def test_decide_matches_exhaustive_action_set(seed):
    rs = random.Random(seed)
    E = rs.randint(2, 8)
    k = rs.randint(1, min(3, E))
    local = [rs.random() < 0.5 for _ in range(E)]
    sim = np.eye(E)
    for a in range(E):
        for b in range(a + 1, E):
            s = rs.choice([rs.uniform(-1, 1), 1 - 10 ** rs.uniform(-4, -1)])
            sim[a][b] = sim[b][a] = s
    pol = dict(omega_t=rs.choice([0.5, 0.2, 0.9]), t_local=1.0,
               t_remote=rs.choice([100.0, 3.0, 1.5]), phi_scale=1.0,
               sim_min=rs.choice([-1.0, 0.9, 0.99]))
    budget = rs.choice([0.02, 0.05, 0.005])
    d_hat = rs.uniform(0, budget)
    z = np.array([rs.gauss(0, 1) for _ in range(E)])
    S, w, I, _, _ = O.route(z, k, normalize=False)
    theta = rs.uniform(0, 1)
    slope = rs.uniform(0, 0.2)
    c, q, _ = O.substitutes(sim, local, pol["phi_scale"], pol["sim_min"])
    dec = O.decide(S, w, I, local, O.as_candidates(c, q), d_hat, budget, theta, slope, pol)
    f_min, act, assigns = _brute_force_decision(S, w, I, local, sim, d_hat,
                                                budget, theta, slope, pol)
    assert dec["action"] == act
    if act == O.ACT_EXEC:
        chosen = tuple(dec["exec"])
        assert chosen in {tuple(a[0] for a in combo) for combo in assigns}
        assert d_hat + dec["d_inc"] <= budget  # Property 2 step
    else:
        assert dec["d_inc"] == pytest.approx(min(1.0, slope * I))


# ----------------------------------------------------- hand-derived golden --
def _golden_cases():
    with open(os.path.join(GOLDEN, "decisions.json")) as f:
        return json.load(f)["cases"]


@pytest.mark.parametrize("case", _golden_cases(), ids=lambda c: c["name"])
def test_golden_decisions(case):
    local = case["local"]
    sim = np.array(case["sim"], dtype=np.float64)
    pol = case["policy"]
    S, w, I, _, _ = O.route(np.array(case["z"]), case["k"], case["normalize"])
    assert S == case["expect"]["S"]
    assert I == pytest.approx(case["expect"]["I"], abs=5e-5)
    c, q, _ = O.substitutes(sim, local, pol["phi_scale"], pol["sim_min"])
    dec = O.decide(S, w, I, local, O.as_candidates(c, q), case["d_hat"], pol["budget"],
                   case["theta"], case["slope"], pol)
    ex = case["expect"]
    assert dec["action"] == ex["action"]
    assert dec["exec"] == ex["exec"]
    assert dec["kind"] == ex["kind"]
    assert dec["d_inc"] == pytest.approx(ex["d_inc"], abs=5e-6)
    if "rows" in ex:
        assert [r[0] for r in dec["rows"]] == [r[0] for r in ex["rows"]]
        assert [r[1] for r in dec["rows"]] == pytest.approx(
            [r[1] for r in ex["rows"]], abs=5e-5)


# -------------------------------------------------------------- Eq. (7) -----
def test_exit_confidence_closed_forms():
    rs = np.random.RandomState(0)
    H = rs.randn(5, 16)
    W = rs.randn(40, 16) * 0.5
    b = rs.randn(40)
    xi = O.exit_confidence(H, W, b, "softmax")
    ref = torch.softmax(torch.tensor(H @ W.T + b), dim=1).max(dim=1).values.numpy()
    assert np.allclose(xi, ref, rtol=1e-13)
    # uniform logits -> 1/V
    assert O.exit_confidence(np.zeros((1, 16)), np.zeros((40, 16)), None,
                             "softmax")[0] == pytest.approx(1 / 40)
    w1 = rs.randn(1, 16)
    sig = O.exit_confidence(H, w1, np.array([0.3]), "sigmoid")
    assert np.allclose(sig, torch.sigmoid(torch.tensor(H @ w1[0] + 0.3)).numpy())


# ------------------------------------------------------ helpers for stacks --
def _tiny(**over):
    cfg = workload("tiny_fp32", **over)
    inp = make_inputs(cfg)
    return cfg, inp, O.model_from_inputs(inp)


def _torch_topk_moe_stack(inp, fp32_round=True):
    """Independent plain top-k MoE (no skip/exit/substitution) in torch fp64."""
    cfg = inp["cfg"]
    h = inp["h0"].to(torch.float64).clone()
    for L in inp["layers"]:
        Wr = L["w_router"].to(torch.float64)
        z = h @ Wr.T
        if L["b_router"] is not None:
            z = z + L["b_router"].to(torch.float64)
        p = torch.softmax(z, dim=1)
        val, idx = torch.topk(z, cfg["top_k"], dim=1)
        out = torch.zeros_like(h)
        for t in range(h.shape[0]):
            wsum = p[t, idx[t]].sum()
            for r in range(cfg["top_k"]):
                e = int(idx[t, r])
                wgt = p[t, e] / wsum if cfg["normalize_topk"] else p[t, e]
                x = h[t]
                u = L["w_up"][e].to(torch.float64) @ x
                if cfg["act"] == "relu":
                    a = torch.relu(u)
                else:
                    g = L["w_gate"][e].to(torch.float64) @ x
                    a = torch.nn.functional.silu(g) * u
                out[t] += wgt * (L["w_down"][e].to(torch.float64) @ a)
        h = h + out
        if fp32_round:
            h = h.to(torch.float32).to(torch.float64)
    return h


# ------------------------------------------------- P7 textbook reduction ----
def test_textbook_reduction_plain_topk_moe():
    # all experts local, theta = -1 (never skip), p_J = 2 (never exit)
    cfg, inp, model = _tiny(top_k=2, normalize_topk=1)
    for l in model["layers"]:
        model["layers"][l]["local_mask"] = [1] * cfg["n_experts"]
        model["layers"][l]["theta"] = -1.0
    pol = dict(inp["policy"], p_exit=2.0)
    st, trs = O.stack_forward(model, pol, inp["h0"].double().numpy())
    for L in inp["layers"]:
        L["local_mask"][:] = 1
    ref = _torch_topk_moe_stack(inp).numpy()
    assert np.allclose(st["h"], ref, rtol=0, atol=1e-5 * np.abs(ref).max())
    for tr in trs:
        assert np.all(tr["action"] == O.ACT_EXEC)
        assert np.all(tr["kind"] == O.KIND_LOCAL)
    assert np.all(st["d_acc"] == 0)
    assert np.all(st["exit_layer"] == cfg["n_layers"])


# ---------------------------------------------- P6 dense all-experts FFN ----
def test_dense_all_experts_reconstruction():
    cfg, inp, model = _tiny(top_k=2)
    pol = inp["policy"]
    h0 = inp["h0"].double()
    st = O.init_state(h0.numpy(), cfg["n_layers"])
    h_before = torch.tensor(st["h"]).clone()
    tr = O.layer_step(model, 0, pol, st)
    L = inp["layers"][0]
    dense = []  # E_e(h) for every expert e and every token
    for e in range(cfg["n_experts"]):
        u = h_before @ L["w_up"][e].to(torch.float64).T
        dense.append(torch.relu(u) @ L["w_down"][e].to(torch.float64).T)
    dense = torch.stack(dense, 1)  # [T, E, d]
    want = h_before.clone()
    for t in range(h0.shape[0]):
        if tr["action"][t] != O.ACT_EXEC:
            continue
        for r in range(cfg["top_k"]):
            want[t] += tr["gate"][t][r] * dense[t, tr["exec"][t][r]]
    want = want.to(torch.float32).to(torch.float64).numpy()
    assert np.allclose(st["h"], want, rtol=0, atol=1e-6)
    skipped = tr["action"] == O.ACT_SKIP
    assert np.array_equal(st["h"][skipped], h_before.numpy()[skipped])


# ----------------------------------------------------- P8 special cases -----
def test_zero_budget_no_skip_no_substitution():
    cfg, inp, model = _tiny()
    for l in model["layers"]:
        model["layers"][l]["skip_slope"] = 0.5  # set directly, > 0
    pol = dict(inp["policy"], budget=0.0)
    st, trs = O.stack_forward(model, pol, inp["h0"].double().numpy())
    assert np.all(st["d_acc"] == 0)
    for tr in trs:
        assert not np.any(tr["action"] == O.ACT_SKIP)
        assert not np.any(tr["kind"] == O.KIND_SUB)


def test_nonpositive_p_exit_exits_after_first_executed_layer():
    cfg, inp, model = _tiny(n_layers=3)
    pol = dict(inp["policy"], p_exit=0.0)
    st, trs = O.stack_forward(model, pol, inp["h0"].double().numpy())
    for t in range(cfg["n_tokens"]):
        acts = [tr["action"][t] for tr in trs]
        first_exec = acts.index(O.ACT_EXEC) if O.ACT_EXEC in acts else None
        if first_exec is not None and first_exec < cfg["n_layers"] - 1:
            assert st["exit_layer"][t] == first_exec
            assert all(a == O.ACT_INACTIVE for a in acts[first_exec + 1:])


def test_all_remote_ample_budget_everything_skips():
    cfg, inp, model = _tiny()
    for l in model["layers"]:
        model["layers"][l]["local_mask"] = [0] * cfg["n_experts"]
        model["layers"][l]["theta"] = 1.0
    pol = dict(inp["policy"], budget=100.0, t_remote=1000.0)
    st, trs = O.stack_forward(model, pol, inp["h0"].double().numpy())
    for tr in trs:
        assert np.all(tr["action"] == O.ACT_SKIP)
    assert np.array_equal(st["h"], inp["h0"].double().numpy())
    assert np.all(st["exit_layer"] == cfg["n_layers"])
    assert np.all(np.isnan(st["xi"]))


def test_identity_similarity_no_substitution():
    cfg, inp, model = _tiny()
    for l in model["layers"]:
        model["layers"][l]["sim"] = np.eye(cfg["n_experts"])
    st, trs = O.stack_forward(model, inp["policy"], inp["h0"].double().numpy())
    for tr in trs:
        assert not np.any(tr["kind"] == O.KIND_SUB)


# ------------------------------------ P1-P4 invariants (Properties 2, 3) ----
def _check_invariants(cfg, model, pol, st, trs):
    N = cfg["n_layers"]
    T = len(st["exit_layer"])
    budget = pol["budget"]
    for t in range(T):
        acts = [int(tr["action"][t]) for tr in trs]
        # (c.5): active indicator non-increasing; layer 0 always active
        assert acts[0] != O.ACT_INACTIVE
        alive = [a != O.ACT_INACTIVE for a in acts]
        assert all(a >= b for a, b in zip(alive, alive[1:]))
        L_exit = st["exit_layer"][t]
        for l, tr in enumerate(trs):
            a = acts[l]
            if a == O.ACT_INACTIVE:
                continue
            # Property 2: budget never exceeded
            assert tr["d_acc"][t] <= budget + 1e-12
            if a == O.ACT_SKIP:
                # Eq. (9): no exit judgement after a skip
                assert math.isnan(tr["xi"][t])
                assert L_exit != l
            else:
                # (c.8): executed expert is the target or a local one with
                # Sim >= sim_min
                Lm = model["layers"][l]
                for r in range(cfg["top_k"]):
                    e, x = tr["target"][t][r], tr["exec"][t][r]
                    assert x == e or (Lm["local_mask"][x] and Lm["sim"][e][x] >= pol["sim_min"])
        if L_exit < N:
            # Property 3: the exit layer was executed and xi >= p_J there
            tr = trs[L_exit]
            assert acts[L_exit] == O.ACT_EXEC
            assert tr["xi"][t] >= pol["p_exit"]
            assert all(a == O.ACT_INACTIVE for a in acts[L_exit + 1:])


def test_invariants_tiny():
    cfg, inp, model = _tiny()
    st, trs = O.stack_forward(model, inp["policy"], inp["h0"].double().numpy())
    _check_invariants(cfg, model, inp["policy"], st, trs)
    # the synthetic recipe must reach every branch of the rule
    acts = np.concatenate([tr["action"] for tr in trs])
    kinds = np.concatenate([tr["kind"].ravel() for tr in trs])
    assert (acts == O.ACT_SKIP).any() and (acts == O.ACT_EXEC).any()
    assert (kinds == O.KIND_SUB).any() and (kinds == O.KIND_LOCAL).any()
    assert (st["exit_layer"] < cfg["n_layers"]).any()


@pytest.mark.parametrize("name,T", [("switch_base_8e", 64)])
def test_invariants_bf16_subset(name, T):
    cfg = workload(name, n_tokens=T)
    inp = make_inputs(cfg)
    model = O.model_from_inputs(inp)
    st, trs = O.stack_forward(model, inp["policy"], inp["h0"].double().numpy())
    _check_invariants(cfg, model, inp["policy"], st, trs)
    # bf16 storage: every output h is a bf16 value
    assert np.array_equal(O.round_bf16(st["h"]), st["h"])


def test_per_token_budget_and_p_exit():
    cfg, inp, model = _tiny()
    T = cfg["n_tokens"]
    budget_tok = np.where(np.arange(T) % 2 == 0, 0.0, 0.05)
    pexit_tok = np.where(np.arange(T) % 3 == 0, 2.0, 0.5)
    st, trs = O.stack_forward(model, inp["policy"], inp["h0"].double().numpy(),
                              token_budget=budget_tok, token_p_exit=pexit_tok)
    assert np.all(st["d_acc"][budget_tok == 0] == 0)
    assert np.all(st["d_acc"] <= budget_tok + 1e-12)
    assert np.all(st["exit_layer"][pexit_tok > 1] == cfg["n_layers"])


def test_tokens_are_independent():
    # a subset of tokens gives the same per-token results as the full batch
    cfg, inp, model = _tiny()
    h0 = inp["h0"].double().numpy()
    st, trs = O.stack_forward(model, inp["policy"], h0)
    sub = [3, 17, 40, 63]
    st2, trs2 = O.stack_forward(model, inp["policy"], h0[sub])
    assert np.array_equal(st2["h"], st["h"][sub])
    assert np.array_equal(st2["exit_layer"], st["exit_layer"][sub])
    for a, b in zip(trs, trs2):
        assert np.array_equal(a["exec"][sub], b["exec"])


def _bf16_round_to_odd(x64):
    """fp64 -> bf16 without double rounding, via torch's fp32 -> bf16 RNE.

    First fp64 -> fp32 with round-to-odd (truncate toward zero, set the last
    bit when inexact), then fp32 -> bf16 round-to-nearest-even: rounding to
    odd at >= 2 extra bits makes the second rounding correct.
    """
    x64 = np.asarray(x64, dtype=np.float64)
    y = x64.astype(np.float32)
    yb = y.view(np.uint32).copy()
    inexact = y.astype(np.float64) != x64
    over = np.abs(y.astype(np.float64)) > np.abs(x64)
    yb = np.where(inexact & over, yb - np.uint32(1), yb)
    yb = np.where(inexact, yb | np.uint32(1), yb).astype(np.uint32)
    t = torch.from_numpy(yb.view(np.float32).copy())
    return t.to(torch.bfloat16).to(torch.float64).numpy()


def test_dense_all_experts_bf16_rounding_points():
    # SwiGLU, top-2, a shared expert, bf16 storage: pins the rounding points
    # (activation to bf16 before the down projection, h to bf16 once)
    cfg = workload("tiny_fp32", dtype="bf16", act="swiglu", top_k=2,
                   d_ff_shared=128, normalize_topk=1)
    inp = make_inputs(cfg)
    model = O.model_from_inputs(inp)
    pol = inp["policy"]
    h_before = inp["h0"].to(torch.float64)
    st = O.init_state(h_before.numpy(), cfg["n_layers"])
    tr = O.layer_step(model, 0, pol, st)
    L = inp["layers"][0]

    def ffn(x, up, gate, down):
        u = x @ up.to(torch.float64).T
        g = x @ gate.to(torch.float64).T
        a = torch.from_numpy(_bf16_round_to_odd(
            (torch.nn.functional.silu(g) * u).numpy()))
        return a @ down.to(torch.float64).T

    dense = torch.stack([ffn(h_before, L["w_up"][e], L["w_gate"][e], L["w_down"][e])
                         for e in range(cfg["n_experts"])], 1)
    shared = ffn(h_before, L["ws_up"], L["ws_gate"], L["ws_down"])
    want = h_before.clone()
    n_exec = 0
    for t in range(cfg["n_tokens"]):
        if tr["action"][t] != O.ACT_EXEC:
            continue
        n_exec += 1
        upd = torch.zeros(cfg["d_model"], dtype=torch.float64)
        for x, wx in tr["rows"][t]:
            upd += wx * dense[t, x]
        want[t] = h_before[t] + (upd + shared[t])
    ex = tr["action"] == O.ACT_EXEC
    want_np = want.numpy()
    want_np[ex] = _bf16_round_to_odd(want_np[ex])
    assert n_exec > 0
    # merged rows carry the slot weights of the trace
    for t in np.nonzero(ex)[0]:
        tot = sum(wx for _, wx in tr["rows"][t])
        assert tot == pytest.approx(sum(tr["gate"][t]), rel=1e-12)
    mismatch = np.count_nonzero(st["h"] != want_np)
    assert mismatch <= 2, mismatch
