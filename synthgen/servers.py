"""Synthetic edge-server scenarios for the offline placement (Table I).

Recipe (all draws from ``synthgen.rng``):

* M servers (10 by default, as in the paper's testbed); server 0 is the one
  this device plays;
* expert sizes: the bytes of an expert's weights in the storage dtype
  (up, gate if SwiGLU, down), the same for every expert of a layer;
* baseline deployment: every expert once, layer by layer, dealt round-robin
  over the servers in a seeded order (a dispersal in the spirit of the
  grouping the placement starts from: neighbours in the order land on
  different servers);
* capacities: each server's baseline usage plus a share of
  (memory_ratio - 1) x the total expert bytes, shares proportional to
  U(0.5, 1.5) draws (heterogeneous memories; total = memory_ratio x the
  expert bytes);
* bandwidth B[m][n] ~ U(10, 100) MB/s and latency tau[m][n] ~ U(5, 50) ms,
  symmetric, B[m][m] = 10 GB/s and tau[m][m] = 0;
* token residency rho[m][l]: a seeded access share per server (U(0.5, 1.5)
  draws normalised), the same at every layer (tokens stay on their access
  server on one device);
* z_l: bytes of one token's hidden state, d x the storage element size.

Plain draws only: nothing of the placement rule is computed here.
"""
from __future__ import annotations

import numpy as np

from .rng import permutation, uniform_f64

_ID_SRV = (1 << 40) + 64


def make_servers(cfg, n_servers: int = 10, memory_ratio: float = 2.0, seed: int | None = None):
    M, N, E = n_servers, cfg["n_layers"], cfg["n_experts"]
    d, F = cfg["d_model"], cfg["d_ff"]
    s = cfg["seed"] if seed is None else seed
    es = 2 if cfg["dtype"] == "bf16" else 4
    mats = 3 if cfg["act"] == "swiglu" else 2
    nbytes = np.full((N, E), float(mats * d * F * es))
    x0 = np.zeros((M, N, E), dtype=np.uint8)
    for l in range(N):
        order = permutation(s, _ID_SRV + l, E).numpy()
        for i, e in enumerate(order):
            x0[(i + l) % M, l, int(e)] = 1
    base = (x0 * nbytes[None]).sum(axis=(1, 2))
    share = 0.5 + uniform_f64(s, _ID_SRV + 1000, M).numpy()
    capacity = base + (memory_ratio - 1.0) * nbytes.sum() * share / share.sum()
    ub = uniform_f64(s, _ID_SRV + 1001, M * M).numpy().reshape(M, M)
    ut = uniform_f64(s, _ID_SRV + 1002, M * M).numpy().reshape(M, M)
    bw = 10e6 + 90e6 * np.triu(ub, 1)
    bw = bw + np.triu(bw, 1).T
    np.fill_diagonal(bw, 10e9)
    lat = 5e-3 + 45e-3 * np.triu(ut, 1)
    lat = np.triu(lat, 1) + np.triu(lat, 1).T
    access = 0.5 + uniform_f64(s, _ID_SRV + 1003, M).numpy()
    rho = np.repeat((access / access.sum())[:, None], N, axis=1)
    z = np.full(N, float(d * es))
    return dict(nbytes=nbytes, capacity=capacity, bandwidth=bw, latency=lat, rho=rho, z=z,
                x0=x0, home=0)
