"""Plain CPU oracle of TrimMoE's offline statistics and replica placement.

TEST INFRASTRUCTURE ONLY: imported by the tests (and nothing on the product
path), like the rest of this package.

From a full-depth calibration record (Table I, line 1: routed experts,
importances and per-layer exit confidences of every calibration token) it
computes:

* active probabilities pi_l                        -- Sec. IV-C, Eq. (26)
* activation frequencies a_l^k                      -- Sec. IV-C (from [37])
* execution probabilities sigma_l^k                 -- Sec. IV-C, Eq. (27)
* expected execution frequencies lambda_l^k          -- Sec. IV-C
* expert transition statistics P_l                  -- Sec. V-E, Eq. (38)

and the communication-aware greedy replication of Table I, lines 9-13, with
the redundancy benefit of Eq. (28); Property 1 (Sec. VI) states what its
output satisfies.

Readings:

P1  the calibration exit layer of a token is the first layer (0-based, not
    the last) whose exit confidence meets p_J, else N (A2); a token is
    active entering layer l iff its exit layer is >= l, which is Eq. (26)'s
    L_q >= l with L_q counted from 1.
P2  a_l^k is the fraction of calibration tokens active at layer l whose
    routed set contains expert k; sigma_l^k (Eq. (27)) the fraction of
    those whose importance exceeds theta_l (0 when no token routes to k);
    lambda = pi * sigma * a.
P3  Eq. (38) with top-k: every pair (k in the routed set at l, k' in the
    routed set at l + 1) of a token active at both layers counts once.
    Rows keep the B most frequent next experts (ties to the lower id) and
    are renormalised over them; a source expert with no count has an empty
    row (padding only).
P4  Eq. (28): B-bar_m and tau-bar_m are the arithmetic means of the
    bandwidth and latency from S_m to the servers hosting e_l^k in the
    current deployment; z_l is the per-token payload of layer l.
P5  Table I, lines 10-13: a pair (m, l, k) is a candidate when e_l^k is not
    yet on S_m and fits S_m's residual memory; the candidate of largest
    benefit is placed (ties: lower l, then k, then m), benefits are
    re-evaluated, and the loop ends when no candidate has a positive
    benefit.
"""
from __future__ import annotations

import math

import numpy as np


def calibration_exit_layers(xi, p_exit: float):
    """P1: per token, the first layer l < N - 1 with xi[l, q] >= p_exit, else N.
    xi is [N, Q] with NaN where no confidence was evaluated."""
    xi = np.asarray(xi, dtype=np.float64)
    N, Q = xi.shape
    out = np.full(Q, N, dtype=np.int64)
    for q in range(Q):
        for l in range(N - 1):
            if not math.isnan(xi[l, q]) and xi[l, q] >= p_exit:
                out[q] = l
                break
    return out


def calibration_stats(target, importance, exit_layer, theta, n_experts: int):
    """pi [N] (Eq. (26)), a [N, E], sigma [N, E] (Eq. (27)), lambda [N, E].

    target [N, Q, k] routed experts of the full-depth pass, importance
    [N, Q], exit_layer [Q] (P1), theta [N]."""
    target = np.asarray(target)
    N, Q, k = target.shape
    E = n_experts
    pi = np.zeros(N)
    act = np.zeros((N, E))
    sigma = np.zeros((N, E))
    for l in range(N):
        active = [q for q in range(Q) if exit_layer[q] >= l]
        pi[l] = len(active) / Q if Q else 0.0
        routed = np.zeros(E)
        above = np.zeros(E)
        for q in active:
            for e in set(int(v) for v in target[l, q]):
                routed[e] += 1
                if float(importance[l, q]) > float(theta[l]):
                    above[e] += 1
        for e in range(E):
            act[l, e] = routed[e] / len(active) if active else 0.0
            sigma[l, e] = above[e] / routed[e] if routed[e] else 0.0
    lam = pi[:, None] * sigma * act
    return pi, act, sigma, lam


def transition_rows(target, exit_layer, n_experts: int, B: int):
    """Eq. (38) with P3: per layer l < N - 1, rows [E] of at most B
    (target, probability) pairs; returns (to [N-1, E, B] int, p [N-1, E, B])
    padded with (-1, 0)."""
    target = np.asarray(target)
    N, Q, k = target.shape
    E = n_experts
    to = np.full((max(N - 1, 0), E, B), -1, dtype=np.int64)
    pr = np.zeros((max(N - 1, 0), E, B))
    for l in range(N - 1):
        counts = np.zeros((E, E), dtype=np.int64)
        for q in range(Q):
            if exit_layer[q] >= l + 1:
                for e in target[l, q]:
                    for f in target[l + 1, q]:
                        counts[int(e), int(f)] += 1
        for e in range(E):
            order = sorted(range(E), key=lambda f: (-counts[e, f], f))
            keep = [f for f in order[:B] if counts[e, f] > 0]
            total = sum(counts[e, f] for f in keep)
            for j, f in enumerate(keep):
                to[l, e, j] = f
                pr[l, e, j] = counts[e, f] / total
    return to, pr


def redundancy_benefit(lam, rho, z, bandwidth, latency, x, m, l, k):
    """Eq. (28) with P4 for one (server, layer, expert)."""
    hosts = [n for n in range(x.shape[0]) if x[n, l, k]]
    b_bar = sum(bandwidth[m][n] for n in hosts) / len(hosts)
    t_bar = sum(latency[m][n] for n in hosts) / len(hosts)
    return lam[l][k] * rho[m][l] * (z[l] / b_bar + t_bar)


def check_deployment(x, nbytes, capacity):
    """(c.1)-(c.3): memory per server within capacity, every expert placed at
    least once, binary entries.  Returns the list of violations."""
    x = np.asarray(x)
    bad = []
    if not np.isin(x, (0, 1)).all():
        bad.append("c.3")
    M = x.shape[0]
    for m in range(M):
        used = float((x[m] * np.asarray(nbytes)).sum())
        if used > capacity[m]:
            bad.append(f"c.1 server {m}")
    if (x.sum(axis=0) < 1).any():
        bad.append("c.2")
    return bad


def place_replicas(lam, rho, z, nbytes, capacity, bandwidth, latency, x0):
    """Table I, lines 9-13 (P5), by re-evaluating every candidate each round.

    Returns (x [M, N, E] uint8, placements in order [(m, l, k, benefit)])."""
    x = np.array(x0, dtype=np.uint8, copy=True)
    M, N, E = x.shape
    used = [float(sum(x[m, l, k] * nbytes[l][k] for l in range(N) for k in range(E)))
            for m in range(M)]
    placed = []
    while True:
        best = None
        for l in range(N):
            for k in range(E):
                for m in range(M):
                    if x[m, l, k] or used[m] + nbytes[l][k] > capacity[m]:
                        continue
                    b = redundancy_benefit(lam, rho, z, bandwidth, latency, x, m, l, k)
                    if b > 0 and (best is None or b > best[0]):
                        best = (b, m, l, k)
        if best is None:
            return x, placed
        b, m, l, k = best
        x[m, l, k] = 1
        used[m] += nbytes[l][k]
        placed.append((m, l, k, b))
