"""Plain fp64 CPU oracle of TrimMoE's per-layer adaptive-depth MoE step.

TEST INFRASTRUCTURE ONLY: imported by the tests, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py``; never by the product path.

It computes, token by token and layer by layer, what the online algorithm of
TrimMoE (arXiv 2608.00573, Sec. V, Algorithm 2 in Table II) decides and
what the MoE layer then outputs, restricted to one device and to the myopic
horizon H = 1 (Sec. V-E: with H = 1 the look-ahead term vanishes):

* routing, gating weights and layer importance   -- Sec. III-B, Eq. (4)
* skip degradation Lambda = rho(I)                -- Sec. III-B, Eq. (5)
* substitution loss Q                             -- Sec. III-A, Eq. (3)
* per-step execute / skip costs                   -- Sec. V-A, Eq. (31), (32)
* per-token budget and feasible action set        -- Sec. V-B, Eq. (33), (34)
* transmission necessity and importance admission -- Sec. V-C, Eq. (35)
* action choice and state update                  -- Sec. V-E, Eq. (40)-(42)
* exit head confidence and exit gate              -- Sec. III-C, Eq. (7)-(9)
* residual bypass of a skipped layer              -- Sec. III-B

Readings taken where the paper is silent or ambiguous:

A1  exit head: xi = max softmax(W_exit h + b) (a vocabulary head); the
    paper's own linear+sigmoid head (Sec. IV-A) is the "sigmoid" mode.
A2  exit takes effect right after an executed layer l with xi_l >= p_J;
    the token then runs no later layer.  xi is not evaluated after the last
    layer, nor after a skipped layer (Eq. (9)).
A3  at H = 1 an admissible exit is always taken (its cost is 0, every
    remaining layer costs > 0; Sec. V-A).
A4  comparisons are non-strict exactly as printed: xi >= p_J (Eq. (8)),
    I <= theta (Sec. V-C), D + Q <= budget (Eq. (34)).
A5  I = sum of the full-softmax router probabilities of the top-k experts
    (router bias included), before any renormalisation.
A6  slot weight w = p_e, or p_e / I when top-k renormalisation is on; a
    substitute inherits its target's weight.
A7  phi(x) = min(1, phi_scale * x) in Eq. (3).
A8  rho(I) = min(1, s_l * I) with a per-layer slope s_l (an input).
A9  the budget is per token (Eq. (33) already divides by the token count).
A10 one device: the token never moves; "local" experts are the ones this
    device holds, a remote expert is a round trip.
A11 with top-k > 1 every routed slot is resolved on its own under the one
    token budget; Gamma > 0 iff no feasible all-local assignment exists; a
    skip bypasses all slots of the layer.
A12 normalised per-slot delays t_local, t_remote; the execute cost is
    omega_T * sum of slot delays + omega_D * sum Q / budget.
A13 at H = 1 a remote slot's only useful substitute is its minimum-Q local
    expert with Sim >= sim_min (ties to the lower id): any other local
    substitute has the same delay and spends more budget.  Under look-ahead
    that no longer holds (the cost-to-go depends on which expert runs), see
    L8.
A14 ties: lower expert id in top-k; among execute options fewer
    substitutions, then the lower slot bitmask; execute before skip.
A15 slots that end on the same expert are merged into one row whose weight
    is the sum, added in rank order.
A16 the shared expert (if any) is always local, takes no part in I or in
    substitution, and is bypassed together with the routed ones by a skip.
A17 budget = 0: only zero-loss options are feasible and the quality terms
    of the costs are taken as 0.
A18 a skip charges only Lambda; an exit charges nothing (Eq. (17)).
A19 h_{l+1} = h_l + MoE(h_l): no normalisation inside the step.

Precision (bf16 storage): inputs are the stored bf16 values widened to
fp64; products and sums are fp64; the expert activation is rounded to bf16
(round-to-nearest-even) before the down projection; h is rounded to bf16
once per executed layer after the weighted sum.  In fp32 storage mode only
h is rounded, to fp32.

Every deciding margin is recorded so a caller can tell which decisions are
too close to call at fp32 accuracy (the "band"): ``margin_pre`` covers the
decisions taken before the expert FFN (routing, substitution, skip),
``margin_exit`` the exit gate (which reads the layer's rounded output), and
``margin`` is the smaller of the two.
"""
from __future__ import annotations

import math

import numpy as np

ACT_INACTIVE, ACT_EXEC, ACT_SKIP = 0, 1, 2
KIND_NONE, KIND_LOCAL, KIND_SUB, KIND_REMOTE = -1, 0, 1, 2

_INF = float("inf")


# ----------------------------------------------------------------------------
# rounding
# ----------------------------------------------------------------------------
def round_bf16(x):
    """Round fp64 values to the nearest bf16 (ties to even), returned as fp64.

    Normal range: on the fp64 bit pattern directly (52 -> 7 mantissa bits),
    so there is no intermediate fp32 rounding.  Below 2^-126 the bf16 values
    are the multiples of 2^-133 (subnormals), and a value rounds to the
    nearest of them, ties to even (so magnitudes up to 2^-134 become zero).
    Non-finite values raise.
    """
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    if not np.all(np.isfinite(a)):
        raise ValueError("round_bf16: value outside the supported range")
    b = a.view(np.uint64)
    lsb = (b >> np.uint64(45)) & np.uint64(1)
    b = (b + np.uint64((1 << 44) - 1) + lsb) & ~np.uint64((1 << 45) - 1)
    out = b.view(np.float64)
    tiny = np.abs(a) < 2.0 ** -126
    if np.any(tiny):
        out = np.array(out, copy=True)
        # scaling by a power of two is exact; np.round ties to even
        out[tiny] = np.round(a[tiny] * 2.0 ** 133) * 2.0 ** -133
    return out


def round_f32(x):
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


# ----------------------------------------------------------------------------
# Eq. (3): substitution loss, and the per-layer substitute table (A13)
# ----------------------------------------------------------------------------
def q_loss(sim: float, phi_scale: float) -> float:
    """Q_l(r, k) for k != r, Eq. (3) with phi(x) = min(1, phi_scale * x)."""
    return min(1.0, phi_scale * (1.0 - sim) / 2.0)


def substitute_candidates(sim, local, phi_scale: float, sim_min: float, n: int):
    """Local substitute candidates of every expert e of one layer.

    The local experts j != e with Sim[e][j] >= sim_min (the feasible set
    V_{l,e} of Sec. III-A restricted to this device's experts), the n of
    least Q(e, j) in ascending (Q, j) order (ties to the lower j).  Returns
    (cands, margins): cands[e] = [(j, Q), ...]; margins[e] = the smallest
    deciding margin of the list: the Q gap at its cut (between the n-th and
    the (n + 1)-th candidate, which decides which experts are offered at
    all) and any candidate's distance of Sim to sim_min.  The order inside
    the list decides nothing by itself: options differ by their costs,
    whose own gaps are recorded where they are compared.
    """
    E = len(local)
    cands, margins = [], []
    for e in range(E):
        lst = []
        m = _INF
        for j in range(E):
            if j == e or not local[j]:
                continue
            s = float(sim[e][j])
            m = min(m, abs(s - sim_min))
            if s >= sim_min:
                lst.append((q_loss(s, phi_scale), j))
        lst.sort()
        if len(lst) > n:
            m = min(m, lst[n][0] - lst[n - 1][0])
        cands.append([(j, q) for q, j in lst[:n]])
        margins.append(m)
    return cands, margins


def substitutes(sim, local, phi_scale: float, sim_min: float):
    """Best local substitute c(e) for every expert e of one layer (A13).

    Returns (c, q, margins): c[e] = argmin over local j != e with
    Sim[e][j] >= sim_min of Q(e, j) (ties to the lower j), -1 if none;
    q[e] = Q(e, c[e]); margins[e] = the smallest deciding margin of that
    choice (gap to the second-best candidate, distance of any candidate's
    Sim to sim_min).
    """
    cands, margins = substitute_candidates(sim, local, phi_scale, sim_min, 1)
    c = [lst[0][0] if lst else -1 for lst in cands]
    q = [lst[0][1] if lst else math.nan for lst in cands]
    return c, q, margins


def as_candidates(c, q):
    """Candidate lists holding each expert's best substitute only."""
    return [[(int(ce), float(qe))] if ce >= 0 else [] for ce, qe in zip(c, q)]


# ----------------------------------------------------------------------------
# Eq. (4): routing, gating weights, importance
# ----------------------------------------------------------------------------
def route(z, k: int, normalize: bool):
    """Top-k of the router logits z (ties to the lower id).

    Returns (S, w, I, p, margin): S in rank order, slot weights w, the
    importance I (Eq. (4), reading A5), the full softmax p and the smallest
    gap between consecutive logits among the first k+1 ranks.
    """
    z = np.asarray(z, dtype=np.float64)
    order = np.argsort(-z, kind="stable")
    S = [int(e) for e in order[:k]]
    ex = np.exp(z - z.max())
    p = ex / ex.sum()
    I = float(sum(p[e] for e in S))
    w = [float(p[e] / I) if normalize else float(p[e]) for e in S]
    ranked = z[order[: min(k + 1, len(z))]]
    margin = float(np.min(ranked[:-1] - ranked[1:])) if len(ranked) > 1 else _INF
    return S, w, I, p, margin


# ----------------------------------------------------------------------------
# Algorithm 2 for one token at one layer
# ----------------------------------------------------------------------------
def step_options(S, I, local, cands, d_hat, budget, theta, slope, pol,
                 m_logit, m_budget):
    """The feasible actions of one token at one layer and their per-step costs.

    Eq. (31) execute costs over every way of serving the slots that Eq.
    (34)'s budget filter admits: each remote slot with substitute candidates
    (cands[e], see substitute_candidates) runs its target or one of them,
    local slots run their target (reading A13); Eq. (35) transmission
    necessity, the importance admission of Sec. V-C and the Eq. (32) skip
    cost (readings A8-A18).  Options are numbered in mixed radix over the
    remote slots with candidates, the highest-ranked one the lowest digit
    (digit 0: the target, d: its d-th candidate); with one candidate per
    slot the number is the bitmask of the substituted slots.
    Returns (execs, skip, gamma_pos, lam, kinds0): execs is a list of
    (f, n_sub, mask, option, charge, x) with x the expert each slot would run
    and mask the substituted slots; skip is (f, charge, x) with x the routed
    targets, or None.  Deciding margins are appended to m_logit (importance
    against theta) and m_budget (budget comparisons).
    """
    wt = pol["omega_t"]
    wd = 1.0 - wt
    t_loc, t_rem = pol["t_local"], pol["t_remote"]
    kinds0 = []
    n_local = n_remote = 0
    rsub = []  # ranks of remote slots that have a local substitute
    for r, e in enumerate(S):
        if local[e]:
            kinds0.append(KIND_LOCAL)
            n_local += 1
        else:
            kinds0.append(KIND_REMOTE)
            n_remote += 1
            if cands[e]:
                rsub.append(r)
    radix = [1 + len(cands[S[r]]) for r in rsub]

    def quality(charge):
        return wd * charge / budget if budget > 0 else 0.0

    execs = []
    n_opt = math.prod(radix)
    for o in range(n_opt):
        mask = 0
        sq = 0.0
        x = list(S)
        rest = o
        for r, rad in zip(rsub, radix):
            digit = rest % rad
            rest //= rad
            if digit:
                j, q = cands[S[r]][digit - 1]
                mask |= 1 << r
                sq += q
                x[r] = j
        n_sub = bin(mask).count("1")
        if mask:
            m_budget.append(abs(budget - d_hat - sq))
        if d_hat + sq <= budget:
            f = wt * ((n_local + n_sub) * t_loc + (n_remote - n_sub) * t_rem) + quality(sq)
            execs.append((f, n_sub, mask, o, sq, x))

    # Eq. (35): Gamma > 0 iff no feasible assignment leaves no remote slot
    gamma_pos = not any(e[1] == n_remote for e in execs)
    lam = min(1.0, slope * I)  # Eq. (5), reading A8
    skip = None
    if gamma_pos:
        m_logit.append(abs(I - theta))
        m_budget.append(abs(budget - d_hat - lam))
        if I <= theta and d_hat + lam <= budget:
            skip = (quality(lam), lam, list(S))  # Eq. (32)
    return execs, skip, gamma_pos, lam, kinds0


def decide(S, w, I, local, cands, d_hat, budget, theta, slope, pol, phi=None):
    """Execute/skip decision and server-expert selection for one token.

    Eq. (40): the action minimising the per-step cost plus the look-ahead
    cost-to-go phi(x, D-hat after the action) (zero at H = 1, Sec. V-E);
    ties as in A14 (then the lower option number of step_options).  cands:
    each expert's local substitute candidates (as_candidates turns a table
    of best substitutes into them).  Returns a dict with the action, per-slot
    (target, exec, kind, weight), the merged execute rows, the degradation
    charged, and the margins (all, importance/cost ones, budget ones).
    """
    k = len(S)
    m_logit, m_budget = [], []
    execs, skip_opt, gamma_pos, lam, kinds0 = step_options(
        S, I, local, cands, d_hat, budget, theta, slope, pol, m_logit, m_budget)

    def total(f, charge, x):
        return f + (phi(x, d_hat + charge) if phi is not None else 0.0)

    options = sorted((total(f, sq, x), n_sub, mask, o, sq, x)
                     for (f, n_sub, mask, o, sq, x) in execs)
    best_t, _, best_mask, _, best_sq, best_x = options[0]
    if len(options) > 1:
        m_logit.append(options[1][0] - options[0][0])
    skip = False
    if skip_opt is not None:
        t_skip = total(*skip_opt)
        m_logit.append(abs(best_t - t_skip))
        skip = t_skip < best_t  # tie goes to execute (A14)

    margins = m_logit + m_budget
    out = dict(target=list(S), weight=list(w), importance=I, lam=lam,
               gamma_pos=gamma_pos, margins=margins, margins_logit=m_logit,
               margins_budget=m_budget)
    if skip:
        out.update(action=ACT_SKIP, exec=[-1] * k, kind=[KIND_NONE] * k,
                   d_inc=lam, rows=[])
        return out
    exec_ids = list(best_x)
    kinds = [KIND_SUB if best_mask >> r & 1 else kinds0[r] for r in range(k)]
    rows = []  # merged (expert, weight), first-occurrence rank order (A15)
    for x, wx in zip(exec_ids, w):
        for i, (y, wy) in enumerate(rows):
            if y == x:
                rows[i] = (y, wy + wx)
                break
        else:
            rows.append((x, wx))
    out.update(action=ACT_EXEC, exec=exec_ids, kind=kinds, d_inc=best_sq,
               rows=rows)
    return out


# ----------------------------------------------------------------------------
# Look-ahead cost-to-go (Sec. V-E, Eq. (38)-(40)) for H > 1
#
# Readings: L1 one device, the token never moves (A10): the location in
# Eq. (39) is always home, so the cost-to-go depends on an action only
# through the experts it runs and the budget it leaves.  L2 P_l(x -> y) is an
# input per layer (Eq. (38) counts come from a calibration pass), stored as
# rows of at most B (target, probability) pairs.  The source of a slot is
# the expert it runs (the substitute after a substitution, the routed target
# when the slot runs exact or the layer is skipped).  L3 with top-k > 1 the
# slots move independently: a next-layer target tuple has the product of
# its slots' probabilities, and it is decided as a routed tuple (duplicates
# included).  L4 future importance is the token's importance at the current
# layer (skip admission and Lambda at later layers use it with their own
# theta and slope).  L5 exits are not predicted inside the recursion (their
# confidence is unknown; the calibration sets of Eq. (36) are not part of
# the step), so the recursion ranges over execute and skip.  L6 the
# recursion stops at the last layer.  L7 the decision at the current layer
# keeps the tie order of A14 on the totals f + Phi, then the lower option
# number (step_options).  L8 every level of the recursion, and the decision
# itself, offer each remote slot its target and its local substitute
# candidates (Sim >= sim_min; the policy's la_subs of least loss, ties to
# the lower id): Eq. (34) admits every deployed feasible expert, and with a
# cost-to-go a higher-loss substitute whose transition row leads to local
# experts can win.  Substitutes are offered for remote targets only, among
# local experts: on one device a remote substitute costs the same round trip
# as the exact target, and a local target already costs the least delay,
# which is what substitution exists to reach (Sec. III-A).
# ----------------------------------------------------------------------------
def cost_to_go(model, tables, l: int, h: int, x, d_hat: float, I: float, budget: float, pol,
               m_logit, m_budget, memo=None):
    """Phi_l^(h)(x, D-hat): the expected least cost of the next h layers
    (Eq. (39)) for a token leaving layer l having run experts x."""
    N = model["n_layers"]
    if h == 0 or l >= N - 1:
        return 0.0
    key = (l, h, tuple(x), d_hat)
    if memo is not None and key in memo:
        return memo[key]
    rows = model["layers"][l]["trans"]
    nxt = model["layers"][l + 1]
    cands, sub_m = tables[l + 1]
    acc = 0.0
    for combo in _tuples([rows[e] for e in x]):
        prob = 1.0
        for _, pr in combo:
            prob *= pr
        if prob == 0.0:
            continue
        tau = [t for t, _ in combo]
        m_budget.extend(sub_m[e] for e in tau if not nxt["local_mask"][e])
        execs, skip, _, _, _ = step_options(tau, I, nxt["local_mask"], cands, d_hat,
                                            budget, nxt["theta"], nxt["skip_slope"], pol,
                                            m_logit, m_budget)
        acts = [(f, sq, xo) for (f, _, _, _, sq, xo) in execs]
        if skip is not None:
            acts.append(skip)
        best = min(f + cost_to_go(model, tables, l + 1, h - 1, xo, d_hat + charge, I, budget,
                                  pol, m_logit, m_budget, memo)
                   for f, charge, xo in acts)
        acc += prob * best
    if memo is not None:
        memo[key] = acc
    return acc


def _tuples(rows):
    """Every choice of one entry per row, the first row varying slowest."""
    if not rows:
        yield ()
        return
    for head in rows[0]:
        for rest in _tuples(rows[1:]):
            yield (head,) + rest


# ----------------------------------------------------------------------------
# expert FFN and exit head
# ----------------------------------------------------------------------------
def _silu(g):
    return g / (1.0 + np.exp(-g))


def expert_ffn(X, w_up, w_gate, w_down, act: str, bf16: bool):
    """E(x) = W_down act(W_up x) for the rows of X (fp64).

    ReLU: act = relu(W_up x).  SwiGLU: act = silu(W_gate x) * (W_up x).
    With bf16 storage the activation is rounded to bf16 before W_down.
    """
    u = X @ w_up.T
    if act == "relu":
        a = np.maximum(u, 0.0)
    else:
        a = _silu(X @ w_gate.T) * u
    if bf16:
        a = round_bf16(a)
    return a @ w_down.T


def exit_confidence(H, w_exit, b_exit, mode: str):
    """xi for the rows of H, Eq. (7).

    softmax mode (A1): xi = max_v softmax(z)_v = 1 / sum_v exp(z_v - max z)
    with z = W_exit h + b; sigmoid mode: xi = 1 / (1 + exp(-(w . h + b))).
    """
    z = H @ w_exit.T
    if b_exit is not None:
        z = z + b_exit
    if mode == "sigmoid":
        return 1.0 / (1.0 + np.exp(-z[:, 0]))
    m = z.max(axis=1, keepdims=True)
    return 1.0 / np.exp(z - m).sum(axis=1)


# ----------------------------------------------------------------------------
# state, layer, stack
# ----------------------------------------------------------------------------
def init_state(h0, n_layers: int):
    """Algorithm 2 initialisation: D = 0, every token active (Eq. (6))."""
    T = h0.shape[0]
    return dict(h=np.array(h0, dtype=np.float64, copy=True),
                d_acc=np.zeros(T), active=list(range(T)),
                exit_layer=np.full(T, n_layers, dtype=np.int64),
                xi=np.full(T, math.nan))


def layer_step(model, l: int, pol, state, token_budget=None, token_p_exit=None):
    """One MoE layer l (0-based) for every active token; returns the trace.

    ``state`` is updated in place: h, d_acc, the active list (in token
    order), exit_layer and xi.  ``token_budget`` / ``token_p_exit``
    optionally give a per-token budget / confidence requirement.
    """
    L = model["layers"][l]
    N, E, k = model["n_layers"], model["n_experts"], model["top_k"]
    T = state["h"].shape[0]
    bf16 = model["dtype"] == "bf16"
    local = [bool(v) for v in L["local_mask"]]
    # look-ahead over the next H - 1 layers (Eq. (39)); H = 1 is the myopic rule
    H = int(pol.get("horizon", 1))
    # substitute candidates per remote slot: the best one at H = 1 (A13),
    # the la_subs least-loss ones under look-ahead (L8)
    n_cand = int(pol.get("la_subs", 1)) if H > 1 else 1
    cands, sub_m = substitute_candidates(L["sim"], local, pol["phi_scale"], pol["sim_min"],
                                         n_cand)
    tables = {}
    for j in range(l + 1, min(l + H, N)):
        Lj = model["layers"][j]
        tables[j] = substitute_candidates(Lj["sim"], [bool(v) for v in Lj["local_mask"]],
                                          pol["phi_scale"], pol["sim_min"], n_cand)

    tr = dict(action=np.zeros(T, np.int8),
              target=np.full((T, k), -1, np.int16),
              exec=np.full((T, k), -1, np.int16),
              kind=np.full((T, k), KIND_NONE, np.int8),
              gate=np.full((T, k), math.nan),
              importance=np.full(T, math.nan),
              xi=np.full(T, math.nan), d_acc=np.full(T, math.nan),
              margin=np.full(T, _INF), margin_pre=np.full(T, _INF),
              margin_logit=np.full(T, _INF), margin_budget=np.full(T, _INF),
              margin_exit=np.full(T, _INF), rows={})

    act_list = list(state["active"])
    h = state["h"]
    if act_list:
        Z = h[act_list] @ L["w_router"].T
        if L["b_router"] is not None:
            Z = Z + L["b_router"]

    execd = []
    for i, q in enumerate(act_list):
        S, w, I, _, m_route = route(Z[i], k, bool(model["normalize_topk"]))
        budget = pol["budget"] if token_budget is None else float(token_budget[q])
        la_logit, la_budget = [], []
        phi = None
        if H > 1 and l < N - 1:
            memo = {}

            def phi(x, d, I=I, budget=budget, memo=memo):
                return cost_to_go(model, tables, l, H - 1, x, d, I, budget, pol, la_logit,
                                  la_budget, memo)
        dec = decide(S, w, I, local, cands, state["d_acc"][q], budget,
                     L["theta"], L["skip_slope"], pol, phi)
        m_logit = min([m_route] + dec["margins_logit"] + la_logit)
        m_budget = min(dec["margins_budget"] + la_budget
                       + [sub_m[e] for e in S if not local[e]], default=_INF)
        m = min(m_logit, m_budget)
        tr["margin"][q] = m
        tr["margin_pre"][q] = m
        tr["margin_logit"][q] = m_logit
        tr["margin_budget"][q] = m_budget
        tr["action"][q] = dec["action"]
        tr["target"][q] = S
        tr["gate"][q] = w
        tr["importance"][q] = I
        tr["exec"][q] = dec["exec"]
        tr["kind"][q] = dec["kind"]
        state["d_acc"][q] += dec["d_inc"]  # Eq. (41) / (42)
        if dec["action"] == ACT_EXEC:
            execd.append(q)
            tr["rows"][q] = dec["rows"]

    # grouped expert FFN over the executed rows, then the residual update
    if execd:
        upd = np.zeros((len(execd), h.shape[1]))
        pos = {q: i for i, q in enumerate(execd)}
        by_expert = {}
        for q in execd:
            for x, wx in tr["rows"][q]:
                by_expert.setdefault(x, []).append((q, wx))
        X_all = h[execd]
        for x, lst in by_expert.items():
            idx = [pos[q] for q, _ in lst]
            Y = expert_ffn(X_all[idx], L["w_up"][x],
                           None if L["w_gate"] is None else L["w_gate"][x],
                           L["w_down"][x], model["act"], bf16)
            for j, (q, wx) in enumerate(lst):
                upd[pos[q]] += wx * Y[j]
        if L.get("ws_up") is not None:
            upd += expert_ffn(X_all, L["ws_up"], L["ws_gate"], L["ws_down"],
                              "swiglu", bf16)
        new = X_all + upd
        h[execd] = round_bf16(new) if bf16 else round_f32(new)

        # exit gate after an executed layer, never after the last (A2, A3)
        if l < N - 1:
            xi = exit_confidence(h[execd], L["w_exit"], L["b_exit"],
                                 model.get("conf_mode", "softmax"))
            for i, q in enumerate(execd):
                pj = pol["p_exit"] if token_p_exit is None else float(token_p_exit[q])
                tr["xi"][q] = xi[i]
                state["xi"][q] = xi[i]
                tr["margin_exit"][q] = abs(xi[i] - pj)
                tr["margin"][q] = min(tr["margin"][q], abs(xi[i] - pj))
                if xi[i] >= pj:  # Eq. (8)
                    state["exit_layer"][q] = l

    for q in act_list:
        tr["d_acc"][q] = state["d_acc"][q]
    state["active"] = [q for q in act_list if state["exit_layer"][q] == N]
    return tr


def stack_forward(model, pol, h0, token_budget=None, token_p_exit=None):
    """Algorithm 2 over all N layers; returns (final state, per-layer traces)."""
    state = init_state(h0, model["n_layers"])
    traces = []
    for l in range(model["n_layers"]):
        traces.append(layer_step(model, l, pol, state, token_budget, token_p_exit))
    return state, traces


# ----------------------------------------------------------------------------
# conversion of generated inputs (torch tensors) to the oracle's fp64 model
# ----------------------------------------------------------------------------
def _f64(t):
    if t is None:
        return None
    import torch
    return t.detach().to("cpu").to(torch.float64).numpy()


def model_from_inputs(inputs, layers=None, decision_layers=()):
    """fp64 numpy copy of generated inputs (exact widening of stored values).

    ``decision_layers``: further layers of which only what a look-ahead
    reads is copied (placement, similarity, theta, slope, transitions)."""
    cfg = inputs["cfg"]
    sel = range(cfg["n_layers"]) if layers is None else layers
    out = dict(n_layers=cfg["n_layers"], n_experts=cfg["n_experts"],
               top_k=cfg["top_k"], dtype=cfg["dtype"], act=cfg["act"],
               normalize_topk=cfg["normalize_topk"],
               conf_mode=cfg.get("conf_mode", "softmax"), layers={})
    for l in sel:
        L = inputs["layers"][l]
        out["layers"][l] = dict(
            w_router=_f64(L["w_router"]), b_router=_f64(L["b_router"]),
            w_up=_f64(L["w_up"]), w_gate=_f64(L["w_gate"]), w_down=_f64(L["w_down"]),
            ws_up=_f64(L["ws_up"]), ws_gate=_f64(L["ws_gate"]),
            ws_down=_f64(L["ws_down"]), w_exit=_f64(L["w_exit"]),
            b_exit=_f64(L["b_exit"]),
            local_mask=[int(v) for v in L["local_mask"].cpu()],
            sim=_f64(L["sim"]), theta=float(L["theta"]),
            skip_slope=float(L["skip_slope"]), trans=_trans_rows(L))
    for l in decision_layers:
        L = inputs["layers"][l]
        out["layers"][l] = dict(local_mask=[int(v) for v in L["local_mask"].cpu()],
                                sim=_f64(L["sim"]), theta=float(L["theta"]),
                                skip_slope=float(L["skip_slope"]), trans=_trans_rows(L))
    return out


def _trans_rows(L):
    """Rows of P_l (reading L2): per source expert, its (target, probability)
    entries in stored order, padding (target -1) dropped; None if absent."""
    to, pr = L.get("trans_to"), L.get("trans_p")
    if to is None:
        return None
    to = to.cpu().numpy()
    pr = _f64(pr)
    return [[(int(t), float(v)) for t, v in zip(to[e], pr[e]) if t >= 0]
            for e in range(to.shape[0])]


# ----------------------------------------------------------------------------
# runtime feedback over an observation window (Sec. V-D Eq. (37), Sec. V-F
# Eq. (43))
#
# Readings: F1 a window is a run of stack passes; its statistics are sums
# over them.  F2 xi_exit-bar is the mean confidence at which the window's
# tokens exited; without exits p_J is left unchanged.  F3 the budget
# utilisation D-bar is the mean over the window's tokens of D-hat / budget
# at the end of the pass (a zero budget counts as zero utilisation).  F4 the
# normalised delay T-bar is the total per-slot delay of the executed slots
# (t_local for local exact and substitute slots, t_remote for remote exact
# ones) over T_ref, which Eq. (21) defines as the delay of full-depth exact
# execution on the same placement.  That strategy is not run: T_ref is
# estimated from the pass itself, each layer counting T k slots at the mean
# delay of the routed targets of the tokens active there (skipped tokens
# included), and a layer that no token reached at the mean over all routed
# slots of the pass.  With no exit this is exact for the routes observed.
# A zero T_ref (an empty window, or t_local = t_remote = 0) leaves the
# weights unchanged.
# ----------------------------------------------------------------------------
def window_stats(model, pol, state, traces, token_budget=None):
    """Sums of one stack pass's observations (add the dicts of a window)."""
    N, k = model["n_layers"], model["top_k"]
    T = state["h"].shape[0]
    exited = state["exit_layer"] < N
    budget = np.full(T, float(pol["budget"])) if token_budget is None \
        else np.asarray(token_budget, dtype=np.float64)
    util = np.where(budget > 0, state["d_acc"] / np.where(budget > 0, budget, 1.0), 0.0)
    def slot_delay(local):
        return pol["t_local"] if local else pol["t_remote"]

    delay = 0.0
    layer_mean = []      # mean routed-target delay per layer (None: nobody active)
    routed = []          # every routed slot's delay in the pass
    for l, tr in enumerate(traces):
        for q in np.nonzero(tr["action"] == ACT_EXEC)[0]:
            for kind in tr["kind"][q]:
                delay += slot_delay(kind != KIND_REMOTE)
        local = model["layers"][l]["local_mask"]
        here = [slot_delay(local[e]) for q in np.nonzero(tr["action"] != ACT_INACTIVE)[0]
                for e in tr["target"][q]]
        routed += here
        layer_mean.append(sum(here) / len(here) if here else None)
    ref = 0.0
    if routed:
        pooled = sum(routed) / len(routed)
        ref = sum(T * k * (pooled if m is None else m) for m in layer_mean)
    return dict(tokens=float(T), exits=float(exited.sum()),
                xi_exit=float(state["xi"][exited].sum()), util=float(util.sum()),
                delay=delay, delay_ref=ref)


def feedback_update(pol, stats, eta: float, kappa: float, p_floor: float):
    """New (p_exit, omega_t) after one window.

    Eq. (37): p_J <- clip(p_J + eta (xi_exit-bar - p_J), [p_floor, 1]).
    Eq. (43): omega_D <- clip(omega_D + kappa (D-bar - T-bar), [0, 1]),
              omega_T <- 1 - omega_D.
    """
    p = pol["p_exit"]
    if stats["exits"] > 0:
        xi_bar = stats["xi_exit"] / stats["exits"]
        p = min(1.0, max(p_floor, p + eta * (xi_bar - p)))
    omega_d = 1.0 - pol["omega_t"]
    if stats["tokens"] > 0 and stats["delay_ref"] > 0:
        d_bar = stats["util"] / stats["tokens"]
        t_bar = stats["delay"] / stats["delay_ref"]
        omega_d = min(1.0, max(0.0, omega_d + kappa * (d_bar - t_bar)))
    return p, 1.0 - omega_d
