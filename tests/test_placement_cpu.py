"""The library's offline statistics and replica placement (host C++ behind
the C ABI) against the oracle, on seeded random calibration records and
deployments.  Host-only functions: these run without a GPU."""
import numpy as np
import pytest

from oracle import placement as P
from paper_2608_00573_amd import abi


def _record(rng, N, Q, E, k):
    target = np.stack([np.stack([rng.choice(E, k, replace=False) for _ in range(Q)])
                       for _ in range(N)]).astype(np.int16)
    importance = rng.uniform(size=(N, Q)).astype(np.float32)
    xi = rng.uniform(size=(N, Q)).astype(np.float32)
    xi[rng.uniform(size=(N, Q)) < 0.1] = np.nan
    theta = rng.uniform(0.2, 0.8, size=N).astype(np.float32)
    return target, importance, xi, theta


@pytest.mark.parametrize("seed,N,Q,E,k", [(0, 4, 200, 8, 1), (1, 6, 333, 8, 2),
                                          (2, 3, 150, 60, 4), (3, 2, 1, 5, 3)])
def test_calibration_statistics_match_oracle(seed, N, Q, E, k):
    rng = np.random.default_rng(seed)
    target, importance, xi, theta = _record(rng, N, Q, E, k)
    p_exit = float(np.float32(0.8))
    ex = abi.trimmoe_calib_exit_layers(xi, p_exit)
    assert ex.tolist() == P.calibration_exit_layers(xi.astype(np.float64), p_exit).tolist()
    got = abi.trimmoe_calib_stats(target, importance, ex, theta, E)
    want = P.calibration_stats(target, importance.astype(np.float64), ex,
                               theta.astype(np.float64), E)
    for g, w in zip(got, want):
        assert np.array_equal(g, w)   # same fp64 operations: bit-identical
    for B in sorted({1, min(3, E), E}):
        to, pr = abi.trimmoe_calib_transitions(target, ex, E, B)
        wto, wpr = P.transition_rows(target, ex, E, B)
        assert np.array_equal(to, wto)
        assert np.array_equal(pr, wpr.astype(np.float32))


def _deployment(rng, M, N, E, ratio, ties=False):
    nbytes = rng.integers(1, 4, size=(N, E)).astype(np.float64)
    x0 = np.zeros((M, N, E), dtype=np.uint8)
    perm = rng.permutation(M)
    for l in range(N):
        for k in range(E):
            x0[perm[(k + l) % M], l, k] = 1
    base = (x0 * nbytes).sum(axis=(1, 2))
    capacity = base + np.floor(rng.uniform(0, 1, size=M) * (ratio - 1) * nbytes.sum() / M)
    if ties:
        bw = np.full((M, M), 4.0)
        lat = np.full((M, M), 0.5)
        lam = rng.choice([0.0, 0.25, 0.5], size=(N, E))
        rho = np.full((M, N), 1.0 / M)
    else:
        bw = rng.uniform(1, 10, size=(M, M))
        lat = rng.uniform(0.0, 0.2, size=(M, M))
        lam = rng.uniform(size=(N, E)) * (rng.uniform(size=(N, E)) > 0.3)
        rho = rng.dirichlet(np.ones(M), size=N).T
    z = rng.uniform(0.5, 2.0, size=N)
    return lam, rho, z, nbytes, capacity, bw, lat, x0


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("ties", [False, True])
def test_placement_matches_oracle(seed, ties):
    rng = np.random.default_rng(100 + seed)
    M, N, E = int(rng.integers(2, 6)), int(rng.integers(1, 5)), int(rng.integers(1, 9))
    inst = _deployment(rng, M, N, E, 2.0, ties)
    x, n = abi.trimmoe_place_replicas(*inst)
    wx, placed = P.place_replicas(*inst)
    assert np.array_equal(x, wx) and n == len(placed)
    assert P.check_deployment(x, inst[3], inst[4]) == []


def test_placement_rejects_infeasible_baselines_and_bad_numbers():
    rng = np.random.default_rng(7)
    lam, rho, z, nbytes, cap, bw, lat, x0 = _deployment(rng, 3, 2, 4, 2.0)
    bad = x0.copy()
    bad[:, 1, 2] = 0                    # an expert placed nowhere: (c.2)
    cases = [((lam, rho, z, nbytes, cap, bw, lat, bad), -2),
             ((lam, rho, z, nbytes, cap * 0.0, bw, lat, x0), -2),          # (c.1)
             ((lam, rho, z, nbytes, cap, bw, lat, x0 * 2), -2),            # (c.3)
             ((lam * np.nan, rho, z, nbytes, cap, bw, lat, x0), -4),
             ((lam, rho, z, nbytes, cap, bw * 0.0, lat, x0), -4),
             ((lam, -rho, z, nbytes, cap, bw, lat, x0), -4)]
    for args, code in cases:
        with pytest.raises(abi.TrimmoeError) as ei:
            abi.trimmoe_place_replicas(*args)
        assert ei.value.status == code
