"""Pins of the oracle's offline statistics and replica placement (Sec. IV-C
Eq. (26)-(28), Sec. V-E Eq. (38), Table I, Property 1) against values worked
by hand, closed forms, invariants and brute force."""
import itertools

import numpy as np
import pytest

from oracle import placement as P


def test_exit_layers_by_hand():
    nan = float("nan")
    # 3 layers, 4 tokens, p_J 0.8: token 0 exits after layer 0, token 1
    # after layer 1, token 2 never (0.9 at the last layer does not count),
    # token 3 never (NaN: no confidence evaluated)
    xi = [[0.85, 0.1, 0.2, nan],
          [0.9, 0.8, 0.79, nan],
          [0.95, 0.99, 0.9, nan]]
    assert P.calibration_exit_layers(xi, 0.8).tolist() == [0, 1, 3, 3]


def test_stats_by_hand():
    # 2 layers, 4 tokens, 3 experts, top-1; exit layers 0, 1, 2, 2 (N = 2):
    # pi_0 = 1, pi_1 = 3/4 (tokens 1, 2, 3 active entering layer 1).
    # Layer 0 routes 0, 0, 1, 2 with importances .2 .6 .7 .1, theta .5:
    # a = (2/4, 1/4, 1/4), sigma = (1/2, 1, 0).  Layer 1 (tokens 1-3)
    # routes 2, 2, 0 with importances .9 .1 .6, theta .5:
    # a = (1/3, 0, 2/3), sigma = (1, 0, 1/2).
    target = np.array([[[0], [0], [1], [2]], [[1], [2], [2], [0]]])
    imp = np.array([[.2, .6, .7, .1], [.3, .9, .1, .6]])
    pi, a, s, lam = P.calibration_stats(target, imp, [0, 1, 2, 2], [.5, .5], 3)
    assert pi.tolist() == [1.0, 0.75]
    assert a[0].tolist() == [0.5, 0.25, 0.25] and s[0].tolist() == [0.5, 1.0, 0.0]
    assert a[1] == pytest.approx([1 / 3, 0, 2 / 3]) and s[1].tolist() == [1.0, 0.0, 0.5]
    assert lam[1] == pytest.approx([0.75 * 1 / 3, 0, 0.75 * 2 / 3 * 0.5])


def test_stats_invariants():
    rng = np.random.default_rng(3)
    N, Q, E, k = 5, 300, 7, 2
    target = np.stack([np.stack([rng.choice(E, k, replace=False) for _ in range(Q)])
                       for _ in range(N)])
    imp = rng.uniform(size=(N, Q))
    ex = rng.integers(0, N + 1, size=Q)
    pi, a, s, lam = P.calibration_stats(target, imp, ex, rng.uniform(size=N), E)
    assert pi[0] == 1.0                              # every token enters layer 0
    assert np.all(np.diff(pi) <= 0)                  # non-increasing (Eq. (6))
    assert np.allclose(a.sum(axis=1), k)             # k distinct experts per token
    assert np.all((s >= 0) & (s <= 1)) and np.all(lam <= pi[:, None] + 1e-15)


def test_transition_rows_by_hand():
    # 2 layers, top-2, 4 experts, 3 tokens all active at layer 1:
    # (0,1)->(2,3), (0,2)->(2,0), (1,3)->(3,1).  Pairs from expert 0:
    # 2, 3, 2, 0 -> counts {2: 2, 0: 1, 3: 1}; with B = 2: 2 (2/3) and the
    # tie between 0 and 3 goes to 0 (1/3).  Expert 3: 3, 1 -> 1 (1/2), 3 (1/2).
    target = np.array([[[0, 1], [0, 2], [1, 3]], [[2, 3], [2, 0], [3, 1]]])
    to, pr = P.transition_rows(target, [2, 2, 2], 4, 2)
    assert to[0, 0].tolist() == [2, 0] and pr[0, 0] == pytest.approx([2 / 3, 1 / 3])
    assert to[0, 3].tolist() == [1, 3] and pr[0, 3].tolist() == [0.5, 0.5]
    # a token that exited after layer 0 does not count
    to, pr = P.transition_rows(target, [0, 2, 2], 4, 4)
    assert to[0, 0].tolist() == [0, 2, -1, -1] and pr[0, 0].tolist() == [0.5, 0.5, 0, 0]
    assert to[0, 1].tolist() == [1, 3, -1, -1]


def _instance(rng, M, N, E, ratio=1.6):
    nbytes = rng.uniform(1.0, 3.0, size=(N, E))
    x0 = np.zeros((M, N, E), dtype=np.uint8)
    for l in range(N):
        for k in range(E):
            x0[(k + l) % M, l, k] = 1
    base = (x0 * nbytes).sum(axis=(1, 2))
    capacity = base + rng.uniform(0, 1) * (ratio - 1) * nbytes.sum() / M
    bw = rng.uniform(1, 10, size=(M, M))
    bw = (bw + bw.T) / 2
    lat = rng.uniform(0.01, 0.1, size=(M, M))
    lat = (lat + lat.T) / 2
    rho = rng.dirichlet(np.ones(M), size=1)[0][:, None] * np.ones((1, N))
    lam = rng.uniform(size=(N, E)) * (rng.uniform(size=(N, E)) > 0.2)
    z = rng.uniform(0.5, 2.0, size=N)
    return lam, rho, z, nbytes, capacity, bw, lat, x0


def test_benefit_and_first_replica_by_hand():
    # 2 servers, 1 layer, 2 experts, both on server 0.  lambda (0.5, 0.2),
    # rho (0.3, 0.7), z 2, B(1,0) 4, tau(1,0) 0.5:
    # B(1,0,0) = 0.5 * 0.7 * (2/4 + 0.5) = 0.35, B(1,0,1) = 0.14.
    # Server 1 fits one expert: expert 0 is replicated, then nothing fits.
    lam = [[0.5, 0.2]]
    rho = [[0.3], [0.7]]
    bw = [[100.0, 4.0], [4.0, 100.0]]
    lat = [[0.0, 0.5], [0.5, 0.0]]
    x0 = np.zeros((2, 1, 2), dtype=np.uint8)
    x0[0, 0, :] = 1
    nbytes = [[1.0, 1.0]]
    x, placed = P.place_replicas(lam, rho, [2.0], nbytes, [2.0, 1.0], bw, lat, x0)
    assert [(m, l, k) for m, l, k, _ in placed] == [(1, 0, 0)]
    assert placed[0][3] == pytest.approx(0.35)
    assert x[1, 0].tolist() == [1, 0]
    # with room for both, expert 1 follows
    x, placed = P.place_replicas(lam, rho, [2.0], nbytes, [2.0, 2.0], bw, lat, x0)
    assert [(m, l, k) for m, l, k, _ in placed] == [(1, 0, 0), (1, 0, 1)]
    # zero execution frequency: no benefit, nothing placed
    x, placed = P.place_replicas([[0.0, 0.0]], rho, [2.0], nbytes, [2.0, 2.0], bw, lat, x0)
    assert placed == []


@pytest.mark.parametrize("seed", range(6))
def test_property1_feasibility(seed):
    rng = np.random.default_rng(seed)
    lam, rho, z, nbytes, cap, bw, lat, x0 = _instance(rng, 4, 3, 5)
    assert P.check_deployment(x0, nbytes, cap) == []
    x, placed = P.place_replicas(lam, rho, z, nbytes, cap, bw, lat, x0)
    assert P.check_deployment(x, nbytes, cap) == []       # (c.1)-(c.3)
    assert np.all(x >= x0)                                  # only adds copies
    # the loop stops only when no positive-benefit replica fits
    used = (x * nbytes).sum(axis=(1, 2))
    for m, l, k in itertools.product(range(4), range(3), range(5)):
        if not x[m, l, k] and used[m] + nbytes[l, k] <= cap[m]:
            assert P.redundancy_benefit(lam, rho, z, bw, lat, x, m, l, k) <= 0
    # the first placement is the best candidate of the baseline deployment
    if placed:
        best = max(P.redundancy_benefit(lam, rho, z, bw, lat, x0, m, l, k)
                   for m, l, k in itertools.product(range(4), range(3), range(5))
                   if not x0[m, l, k] and (x0[m] * nbytes).sum() + nbytes[l, k] <= cap[m])
        assert placed[0][3] == best


def test_greedy_matches_exhaustive_on_single_slot_instances():
    """One server holds everything and a second has room for exactly one
    replica: greedy placement must pick the candidate of largest benefit,
    found here by enumerating the candidates."""
    rng = np.random.default_rng(9)
    M, N, E = 2, 4, 1
    for _ in range(20):
        lam, rho, z, _, _, bw, lat, _ = _instance(rng, M, N, E)
        lam = rng.uniform(0.1, 1, size=(N, E))
        nbytes = np.ones((N, E))
        x0 = np.zeros((M, N, E), dtype=np.uint8)
        x0[0] = 1                                           # everything on server 0
        cap = np.array([N, 1.0])
        x, placed = P.place_replicas(lam, rho, z, nbytes, cap, bw, lat, x0)
        for m in (1,):
            want = max(range(N), key=lambda l: (lam[l][0] * rho[m][l] *
                                                (z[l] / bw[m][0] + lat[m][0]), -l))
            assert x[m, :, 0].tolist() == [int(l == want) for l in range(N)]
