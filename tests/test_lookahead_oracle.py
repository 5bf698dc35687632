"""Pins of the oracle's look-ahead (Sec. V-E, Eq. (38)-(40)) on hand-built
layers: values worked by hand, a decision the look-ahead reverses, and brute
force over action sequences (a formulation independent of the recursion)."""
import itertools
import math

import numpy as np
import pytest

import oracle as O
import oracle.trimmoe_oracle as T

POL = dict(omega_t=0.5, t_local=1.0, t_remote=100.0, budget=0.02, phi_scale=1.0,
           sim_min=-1.0, p_exit=0.9)


def _layer(local, sub, theta=0.5, slope=0.02, trans=None):
    """A hand-built layer: local mask, {remote expert: (substitute, Q)}."""
    E = len(local)
    sim = np.eye(E)
    for e, (c, q) in sub.items():
        # Q = (1 - Sim) / 2 with phi_scale 1; other local experts get Sim -1
        for j in range(E):
            if j != e and local[j]:
                sim[e][j] = -1.0
        sim[e][c] = 1.0 - 2.0 * q
    for e in range(E):
        if not local[e] and e not in sub:
            for j in range(E):
                if j != e:
                    sim[e][j] = -1.0 - 1e-9   # below sim_min: no substitute
    return dict(local_mask=list(local), sim=sim, theta=theta, skip_slope=slope, trans=trans)


def _tables(model, pol, n=1):
    return {l: O.substitute_candidates(L["sim"], [bool(v) for v in L["local_mask"]],
                                       pol["phi_scale"], pol["sim_min"], n)
            for l, L in model["layers"].items()}


def _phi(model, l, h, x, D, I, pol=POL):
    return T.cost_to_go(model, _tables(model, pol), l, h, x, D, I, pol["budget"], pol, [], [],
                        {})


def test_cost_to_go_by_hand():
    # Layer 1: expert 0 local; 1 remote with substitute 0 at Q = 0.01; 2
    # remote without substitute.  From layer 0, expert 0 moves to 1 or 2
    # with probability 1/2 each.  omega 0.5, t (1, 100), budget 0.02, I 0.3,
    # theta 0.5, slope 0.02 (Lambda 0.006).
    #   target 1: remote 0.5 * 100 = 50, substitute 0.5 * 1 + 0.5 * 0.01 /
    #   0.02 = 0.75 -> 0.75 (a local option exists: no skip);
    #   target 2: remote 50, skip 0.5 * 0.006 / 0.02 = 0.15 -> 0.15.
    # Phi = 0.5 * 0.75 + 0.5 * 0.15 = 0.45.
    trans = [[(1, 0.5), (2, 0.5)], [(0, 1.0)], [(0, 1.0)]]
    model = dict(n_layers=2, top_k=1,
                 layers={0: _layer([1, 0, 0], {}, trans=trans),
                         1: _layer([1, 0, 0], {1: (0, 0.01)})})
    assert _phi(model, 0, 1, [0], 0.0, 0.3) == pytest.approx(0.45, abs=1e-12)
    # with 0.011 already spent the substitute no longer fits (0.021 > 0.02),
    # so target 1 has no local option either and its skip (0.017) is
    # admitted: 0.5 * 0.15 + 0.5 * 0.15 = 0.15
    assert _phi(model, 0, 1, [0], 0.011, 0.3) == pytest.approx(0.15, abs=1e-12)
    # with 0.015 spent nothing but exact execution fits: 0.5 * 50 + 0.5 * 50
    assert _phi(model, 0, 1, [0], 0.015, 0.3) == pytest.approx(50.0, abs=1e-12)
    # horizon 1, or nothing after the last layer: zero
    assert _phi(model, 0, 0, [0], 0.0, 0.3) == 0.0
    assert _phi(model, 1, 2, [0], 0.0, 0.3) == 0.0


def test_look_ahead_reverses_a_myopic_substitution():
    # Layer 0: the target (expert 1) is remote; substituting it by expert 0
    # costs Q = 0.012.  Both run experts move to expert 2 of layer 1, which
    # is remote with no substitute but can be skipped at Lambda = 0.015.
    #   myopic: substitute 0.5 + 0.5 * 0.012 / 0.02 = 0.8 < remote 50.
    #   look-ahead: substitute 0.8 + (skip no longer fits: remote 50) = 50.8;
    #   remote 50 + skip 0.5 * 0.015 / 0.02 = 50.375 -> remote exact.
    to2 = [[(2, 1.0)], [(2, 1.0)], [(2, 1.0)]]
    model = dict(n_layers=2, top_k=1,
                 layers={0: _layer([1, 0, 0], {1: (0, 0.012)}, trans=to2),
                         1: _layer([1, 0, 0], {}, theta=0.5, slope=0.05)})
    I = 0.3
    tables = _tables(model, POL)
    cands, _ = tables[0]
    args = ([1], [1.0], I, [True, False, False], cands, 0.0, POL["budget"], 0.4, 0.05, POL)
    myopic = O.decide(*args)
    assert myopic["action"] == O.ACT_EXEC and myopic["kind"] == [O.KIND_SUB]

    def phi(x, d):
        return T.cost_to_go(model, tables, 0, 1, x, d, I, POL["budget"], POL, [], [], {})
    ahead = O.decide(*args, phi=phi)
    assert ahead["action"] == O.ACT_EXEC and ahead["kind"] == [O.KIND_REMOTE]
    assert phi([0], 0.012) == pytest.approx(50.0)
    assert phi([1], 0.0) == pytest.approx(0.375)


# ------------------------------------------------------------ brute force --
def _step_min_brute(L, S, D, I, pol):
    """Least per-step cost of one layer by enumerating, slot by slot, every
    way to serve it (exact, or any local expert with Sim >= sim_min as its
    substitute) and the skip, with the admission rules of Sec. V-B/V-C.
    Returns [(cost, charge, experts run, is skip)] of the feasible actions."""
    E = len(L["local_mask"])
    b, wt = pol["budget"], pol["omega_t"]
    wd = 1.0 - wt
    ways = []
    for e in S:
        opts = [(e, 0.0, bool(L["local_mask"][e]))]
        if not L["local_mask"][e]:
            for j in range(E):
                if j != e and L["local_mask"][j] and L["sim"][e][j] >= pol["sim_min"]:
                    opts.append((j, min(1.0, pol["phi_scale"] * (1 - L["sim"][e][j]) / 2), True))
        ways.append(opts)
    acts = []
    any_local = False
    for combo in itertools.product(*ways):
        q = sum(c[1] for c in combo)
        if D + q > b:
            continue
        delay = sum(pol["t_local"] if c[2] else pol["t_remote"] for c in combo)
        any_local = any_local or all(c[2] for c in combo)
        acts.append((wt * delay + (wd * q / b if b > 0 else 0.0), q, [c[0] for c in combo], False))
    lam = min(1.0, L["skip_slope"] * I)
    if not any_local and I <= L["theta"] and D + lam <= b:
        acts.append((wd * lam / b if b > 0 else 0.0, lam, list(S), True))
    return acts


def _random_model(rng, N, E, k, B, twins=1):
    """Random layers; each remote expert gets up to `twins` local experts
    close enough that their substitution fits the budget."""
    layers = {}
    for l in range(N):
        local = [1] * (E // 2) + [0] * (E - E // 2)
        rng.shuffle(local)
        sim = rng.uniform(-0.2, 0.2, (E, E))
        for e in range(E):
            sim[e][e] = 1.0
            if not local[e] and rng.uniform() < 0.8:
                locs = [j for j in range(E) if local[j]]
                for j in rng.choice(locs, size=min(int(rng.integers(1, twins + 1)), len(locs)),
                                    replace=False):
                    sim[e][j] = 1.0 - 2.0 * rng.uniform(0.001, 0.02)
        trans = None
        if l < N - 1:
            trans = []
            for e in range(E):
                tg = rng.choice(E, size=B, replace=False)
                p = rng.uniform(size=B) ** 2
                trans.append([(int(t), float(v)) for t, v in zip(tg, p / p.sum())])
        layers[l] = dict(local_mask=local, sim=sim, theta=float(rng.uniform(0.2, 0.8)),
                         skip_slope=float(rng.uniform(0.005, 0.05)), trans=trans)
    return dict(n_layers=N, top_k=k, layers=layers)


def _phi_all(model, l, h, x, D, I, pol):
    """Phi with every local candidate offered (reading L8)."""
    E = len(model["layers"][l]["local_mask"])
    return T.cost_to_go(model, _tables(model, pol, n=E), l, h, x, D, I, pol["budget"], pol, [],
                        [], {})


@pytest.mark.parametrize("k,B,twins", [(1, 3, 1), (2, 2, 1), (1, 3, 3), (2, 2, 2)])
def test_two_step_look_ahead_is_expected_best_next_step(k, B, twins):
    """H = 2: Phi = sum over next-layer tuples of P times the least cost of
    that layer, each enumerated by brute force over every local candidate
    (several of which fit the budget when twins > 1)."""
    rng = np.random.default_rng(11 + k + 7 * twins)
    pol = dict(POL, t_remote=3.0, omega_t=0.3)
    for trial in range(30):
        model = _random_model(rng, 3, 5, k, B, twins)
        x = list(rng.choice(5, size=k, replace=False))
        D, I = float(rng.uniform(0, 0.015)), float(rng.uniform(0.1, 0.9))
        want = 0.0
        for combo in itertools.product(*[model["layers"][0]["trans"][e] for e in x]):
            prob = math.prod(pv for _, pv in combo)
            tau = [t for t, _ in combo]
            want += prob * min(a[0] for a in _step_min_brute(model["layers"][1], tau, D, I, pol))
        assert _phi_all(model, 0, 1, x, D, I, pol) == pytest.approx(want, rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("twins", [1, 3])
def test_three_step_look_ahead_with_certain_transitions_is_best_sequence(twins):
    """H = 3 with one-entry transition rows: Phi is the least total cost over
    every two-layer action sequence, found by exhaustive enumeration."""
    rng = np.random.default_rng(5 + twins)
    pol = dict(POL, t_remote=3.0, omega_t=0.3)
    for trial in range(30):
        model = _random_model(rng, 4, 5, 2, 1, twins)
        x = list(rng.choice(5, size=2, replace=False))
        D, I = float(rng.uniform(0, 0.015)), float(rng.uniform(0.1, 0.9))
        nxt = lambda l, xs: [model["layers"][l]["trans"][e][0][0] for e in xs]  # noqa: E731
        best = math.inf
        for c1, q1, x1, _ in _step_min_brute(model["layers"][1], nxt(0, x), D, I, pol):
            for c2, _, _, _ in _step_min_brute(model["layers"][2], nxt(1, x1), D + q1, I, pol):
                best = min(best, c1 + c2)
        assert _phi_all(model, 0, 2, x, D, I, pol) == pytest.approx(best, rel=1e-12, abs=1e-12)


def test_horizon_changes_decisions_on_the_test_recipe():
    """The recipe the GPU look-ahead tests use reaches decisions that differ
    from the myopic rule (so those tests exercise the cost-to-go)."""
    from synthgen import make_inputs, workload
    from tests.gpu_harness import policy32
    cfg = workload("tiny_fp32", n_layers=4, t_remote=2.0, omega_t=0.2)
    inp = make_inputs(cfg)
    model = O.model_from_inputs(inp)
    h0 = inp["h0"].double().numpy()
    runs = {H: O.stack_forward(model, policy32(dict(inp["policy"], horizon=H)), h0.copy())[1]
            for H in (1, 3)}
    diff = sum(int(((runs[3][l]["action"] != runs[1][l]["action"]) |
                    np.any(runs[3][l]["exec"] != runs[1][l]["exec"], axis=1)).sum())
               for l in range(cfg["n_layers"]))
    assert diff >= 5


def test_look_ahead_picks_a_higher_loss_substitute_for_its_next_layer():
    """Eq. (34) admits every feasible local substitute, and Eq. (40) adds the
    cost-to-go, which depends on the expert run: a higher-loss substitute
    whose next expert is local beats the least-loss one whose next expert is
    remote.  Layer 0: target 0 remote, local 1 (Q 0.001) and 2 (Q 0.002);
    expert 1 moves to expert 3 of layer 1 (remote, no substitute, not
    skippable: theta 0), expert 2 to expert 2 (local).  omega 0.5, t (1,
    100), budget 0.02:
      run 1: 0.5 + 0.5 * 0.001 / 0.02 + 0.5 * 100 = 50.525
      run 2: 0.5 + 0.5 * 0.002 / 0.02 + 0.5 * 1   = 1.05
      remote exact 0: 50 + Phi(0), expert 0 moving to 3 as well = 100."""
    sim = np.full((4, 4), -1.0)
    np.fill_diagonal(sim, 1.0)
    sim[0][1], sim[0][2] = 1.0 - 2 * 0.001, 1.0 - 2 * 0.002
    to = [[(3, 1.0)], [(3, 1.0)], [(2, 1.0)], [(3, 1.0)]]
    L0 = dict(local_mask=[0, 1, 1, 0], sim=sim, theta=0.0, skip_slope=0.01, trans=to)
    L1 = dict(local_mask=[0, 1, 1, 0], sim=np.where(np.eye(4) > 0, 1.0, -1.0 - 1e-9), theta=0.0,
              skip_slope=0.01, trans=None)
    model = dict(n_layers=2, top_k=1, layers={0: L0, 1: L1})
    I = 0.3
    for n, want in ((2, 2), (1, 1)):
        tables = _tables(model, POL, n=n)

        def phi(x, d, tables=tables):
            return T.cost_to_go(model, tables, 0, 1, x, d, I, POL["budget"], POL, [], [], {})
        dec = O.decide([0], [1.0], I, [False, True, True, False], tables[0][0], 0.0,
                       POL["budget"], 0.0, 0.01, POL, phi=phi)
        assert dec["action"] == O.ACT_EXEC and dec["kind"] == [O.KIND_SUB]
        assert dec["exec"] == [want]  # n = 1 keeps only the least-loss one
        assert dec["d_inc"] == pytest.approx(0.001 * want)
    tables = _tables(model, POL, n=2)
    assert T.cost_to_go(model, tables, 0, 1, [1], 0.001, I, POL["budget"], POL, [], [], {}) \
        == pytest.approx(50.0)
    assert T.cost_to_go(model, tables, 0, 1, [2], 0.002, I, POL["budget"], POL, [], [], {}) \
        == pytest.approx(0.5)


@pytest.mark.parametrize("k,B", [(1, 3), (2, 2)])
def test_decision_with_look_ahead_is_best_two_layer_plan(k, B):
    """H = 2 decision (Eq. (40)) over every feasible action now, each valued
    by its per-step cost plus the expected least cost of the next layer,
    both enumerated by brute force over every local candidate."""
    rng = np.random.default_rng(31 + k)
    pol = dict(POL, t_remote=3.0, omega_t=0.3)
    n_checked = 0
    for trial in range(60):
        model = _random_model(rng, 2, 5, k, B, twins=3)
        L0 = model["layers"][0]
        E = len(L0["local_mask"])
        S = list(rng.choice(E, size=k, replace=False))
        D, I = float(rng.uniform(0, 0.015)), float(rng.uniform(0.1, 0.9))
        tables = _tables(model, pol, n=E)

        def phi(x, d):
            return T.cost_to_go(model, tables, 0, 1, x, d, I, pol["budget"], pol, [], [], {})
        best, best_x = math.inf, None
        for f, charge, x, skip in _step_min_brute(L0, S, D, I, pol):
            tot = f
            for combo in itertools.product(*[L0["trans"][e] for e in x]):
                prob = math.prod(pv for _, pv in combo)
                tot += prob * min(a[0] for a in _step_min_brute(
                    model["layers"][1], [t for t, _ in combo], D + charge, I, pol))
            if tot < best - 1e-9:
                best, best_x = tot, ("skip" if skip else x)
        dec = O.decide(S, [1.0 / k] * k, I, [bool(v) for v in L0["local_mask"]], tables[0][0], D,
                       pol["budget"], L0["theta"], L0["skip_slope"], pol, phi=phi)
        got = "skip" if dec["action"] == O.ACT_SKIP else dec["exec"]
        if min(dec["margins_logit"], default=1.0) > 1e-9:  # no exact tie between plans
            assert got == best_x
            n_checked += 1
    assert n_checked >= 40
