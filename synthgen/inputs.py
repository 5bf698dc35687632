"""Synthetic model weights, hidden states and calibration inputs.

Recipe (all draws from ``synthgen.rng``; ``sigma`` = 0.02 unless noted):

* router W_r [E,d] ~ N(0, sigma); router bias 0, or, when ``zipf_bias`` = s
  > 0, b_e = -s * ln(rank_e + 1) minus its mean, rank_e a seeded permutation
  (Zipf-skewed expert loads);
* placement: a seeded choice of ``n_local`` of the E experts is local;
* experts: every local expert draws up/gate/down ~ N(0, sigma) (down uses
  sigma / sqrt(2N) when ``down_sigma_scale``).  Each remote expert e gets a
  local twin t(e) (round-robin over the local experts) and is stored as
  W_e = alpha_e * N_t + sqrt(1 - alpha_e^2) * N_e on all three matrices,
  with 1 - alpha_e log-uniform over ``twin_alpha_log10``.  Without planted
  twins independent experts have cosine ~0 and no substitute is ever cheap
  enough for the budget;
* similarity Sim [E,E]: fp64 cosine of the stored weights of each expert,
  flattened and concatenated (up, gate, down), diagonal exactly 1;
* exit heads: W_lm [V,d] ~ N(0, sigma) once per model; layer l stores
  gamma_l * W_lm, gamma_l rising linearly over ``exit_gamma`` with depth;
  bias 0;
* hidden states h0 [T,d] ~ N(0,1), plus for token q a planted component
  c_q * W_lm[v_q] / ||W_lm[v_q]||^2 (v_q uniform over the vocabulary, c_q
  uniform over ``exit_plant``), so that the exit-head max-probability grows
  with depth for a seeded share of tokens.  Without it a random head gives
  max-prob ~1/V and no token ever exits;
* importance thresholds theta_l ~ U(0,1) (sorted ascending over depth when
  ``theta_sorted``); skip-degradation slopes s_l = (budget/2)/max(theta_l,
  0.05), i.e. a linear degradation curve whose tolerance is the budget
  spread over two expected skips;
* expert transitions P_l (l < N-1, used by the look-ahead): for each source
  expert e a support of ``trans_support`` = B distinct next-layer experts
  (the first B of a seeded permutation) with probabilities proportional to
  u^3, u ~ U(0,1) per entry (peaked rows, as calibration counts of a
  routing with layer-to-layer correlation would give), stored as fp32 and
  used as stored.

Everything is returned in the storage dtype (bf16 or fp32) on ``device``.
"""
from __future__ import annotations

import math

import torch

from .rng import normal_f32, uniform_f64, permutation, splitmix64_stream

SIGMA = 0.02

# tensor ids: per-layer ids are (layer + 1) << 16 | kind << 10 | expert
_K_UP, _K_GATE, _K_DOWN, _K_SUP, _K_SGATE, _K_SDOWN = 1, 2, 3, 4, 5, 6
_K_ROUTER, _K_ZIPF_PERM, _K_LOCAL_PERM, _K_ALPHA = 7, 8, 9, 10
_K_TRANS_PERM, _K_TRANS_P = 11, 12
_ID_WLM = 1 << 40
_ID_THETA = (1 << 40) + 1
_ID_H0 = (1 << 40) + 16
_ID_PLANT_V = (1 << 40) + 17
_ID_PLANT_C = (1 << 40) + 18


def _lid(layer: int, kind: int, e: int = 0) -> int:
    return ((layer + 1) << 16) | (kind << 10) | e


def storage_dtype(cfg) -> torch.dtype:
    return {"bf16": torch.bfloat16, "f32": torch.float32}[cfg["dtype"]]


def placement(cfg, layer: int) -> torch.Tensor:
    """u8 [E]: 1 where the expert is resident on this GPU ("local")."""
    E = cfg["n_experts"]
    perm = permutation(cfg["seed"], _lid(layer, _K_LOCAL_PERM), E)
    mask = torch.zeros(E, dtype=torch.uint8)
    mask[perm[: cfg["n_local"]]] = 1
    return mask


def twins(cfg, layer: int, mask: torch.Tensor):
    """(twin[e] or -1, alpha[e] as fp32) for each expert of a layer."""
    E = cfg["n_experts"]
    local = [e for e in range(E) if mask[e]]
    remote = [e for e in range(E) if not mask[e]]
    lo, hi = cfg["twin_alpha_log10"]
    u = uniform_f64(cfg["seed"], _lid(layer, _K_ALPHA), E)
    twin = [-1] * E
    alpha = [1.0] * E
    for i, e in enumerate(remote):
        if not local:
            break
        twin[e] = local[i % len(local)]
        one_minus = 10.0 ** (lo + (hi - lo) * float(u[e]))
        alpha[e] = 1.0 - one_minus
    return twin, torch.tensor(alpha, dtype=torch.float32)


def _expert_matrix(cfg, layer, kind, shape, sigma, twin, alpha, device, dt):
    E = cfg["n_experts"]
    out = torch.empty((E,) + tuple(shape), dtype=dt, device=device)
    base = {}
    for e in range(E):
        own = normal_f32(cfg["seed"], _lid(layer, kind, e), shape, sigma, device)
        t = twin[e]
        if t < 0:
            out[e] = own.to(dt)
        else:
            if t not in base:
                base[t] = normal_f32(cfg["seed"], _lid(layer, kind, t), shape,
                                     sigma, device)
            a = alpha[e].item()
            b = torch.tensor(math.sqrt(max(0.0, 1.0 - a * a)),
                             dtype=torch.float32).item()
            mixed = torch.add(torch.mul(base[t], a), torch.mul(own, b))
            out[e] = mixed.to(dt)
        del own
    return out


def _cosine_sim(mats, E: int) -> torch.Tensor:
    """fp64 cosine between experts of the flattened, concatenated weights."""
    gram = None
    for m in mats:
        if m is None:
            continue
        flat = m.reshape(E, -1)
        g = torch.zeros(E, E, dtype=torch.float64, device=m.device)
        step = 1 << 22
        for j in range(0, flat.shape[1], step):
            blk = flat[:, j:j + step].to(torch.float64)
            g += blk @ blk.T
        gram = g if gram is None else gram + g
    n = torch.sqrt(torch.diagonal(gram))
    sim = gram / (n[:, None] * n[None, :])
    sim.fill_diagonal_(1.0)
    return sim.to(torch.float32)


def make_layer(cfg, layer: int, w_lm: torch.Tensor, device="cpu") -> dict:
    E, d, F, Fs = cfg["n_experts"], cfg["d_model"], cfg["d_ff"], cfg["d_ff_shared"]
    N = cfg["n_layers"]
    dt = storage_dtype(cfg)
    seed = cfg["seed"]
    mask = placement(cfg, layer)
    twin, alpha = twins(cfg, layer, mask)
    down_sigma = SIGMA / math.sqrt(2 * N) if cfg["down_sigma_scale"] else SIGMA

    w_router = normal_f32(seed, _lid(layer, _K_ROUTER), (E, d), SIGMA, device).to(dt)
    b_router = None
    if cfg["zipf_bias"] > 0:
        rank = permutation(seed, _lid(layer, _K_ZIPF_PERM), E).to(torch.float64)
        b = -cfg["zipf_bias"] * torch.log(rank + 1.0)
        b_router = (b - b.mean()).to(torch.float32).to(device)

    w_up = _expert_matrix(cfg, layer, _K_UP, (F, d), SIGMA, twin, alpha, device, dt)
    w_gate = None
    if cfg["act"] == "swiglu":
        w_gate = _expert_matrix(cfg, layer, _K_GATE, (F, d), SIGMA, twin, alpha,
                                device, dt)
    w_down = _expert_matrix(cfg, layer, _K_DOWN, (d, F), down_sigma, twin, alpha,
                            device, dt)
    sim = _cosine_sim([w_up, w_gate, w_down], E)

    ws_up = ws_gate = ws_down = None
    if Fs > 0:
        ws_up = normal_f32(seed, _lid(layer, _K_SUP), (Fs, d), SIGMA, device).to(dt)
        ws_gate = normal_f32(seed, _lid(layer, _K_SGATE), (Fs, d), SIGMA, device).to(dt)
        ws_down = normal_f32(seed, _lid(layer, _K_SDOWN), (d, Fs), down_sigma,
                             device).to(dt)

    g_lo, g_hi = cfg["exit_gamma"]
    gamma = g_lo + (g_hi - g_lo) * (layer / (N - 1) if N > 1 else 1.0)
    g32 = torch.tensor(gamma, dtype=torch.float32).item()
    w_exit = torch.mul(w_lm, g32).to(dt)

    theta_all = uniform_f64(seed, _ID_THETA, N)
    if cfg["theta_sorted"]:
        theta_all, _ = torch.sort(theta_all)
    theta = float(torch.tensor(theta_all[layer].item(), dtype=torch.float32))
    slope = float(torch.tensor((cfg["budget"] / 2.0) / max(theta, 0.05),
                               dtype=torch.float32))
    trans_to, trans_p = transitions(cfg, layer)
    return dict(w_router=w_router, b_router=b_router, w_up=w_up, w_gate=w_gate,
                w_down=w_down, ws_up=ws_up, ws_gate=ws_gate, ws_down=ws_down,
                w_exit=w_exit, b_exit=None, local_mask=mask.to(device),
                sim=sim.to(device), theta=theta, skip_slope=slope,
                trans_to=None if trans_to is None else trans_to.to(device),
                trans_p=None if trans_p is None else trans_p.to(device),
                twin=twin, alpha=alpha, gamma=g32)


def transitions(cfg, layer: int):
    """P_layer as (targets int16 [E, B], probabilities fp32 [E, B]); (None,
    None) for the last layer."""
    E, N = cfg["n_experts"], cfg["n_layers"]
    if layer >= N - 1:
        return None, None
    B = min(int(cfg.get("trans_support", 4)), E)
    to = torch.empty(E, B, dtype=torch.int16)
    pr = torch.empty(E, B, dtype=torch.float32)
    for e in range(E):
        perm = permutation(cfg["seed"], _lid(layer, _K_TRANS_PERM, e), E)
        u = uniform_f64(cfg["seed"], _lid(layer, _K_TRANS_P, e), B) ** 3
        to[e] = perm[:B].to(torch.int16)
        pr[e] = (u / u.sum()).to(torch.float32)
    return to, pr


def exit_lm(cfg, device="cpu") -> torch.Tensor:
    return normal_f32(cfg["seed"], _ID_WLM, (cfg["vocab_exit"], cfg["d_model"]),
                      SIGMA, device)


def make_tokens(cfg, token_seed: int | None = None, device="cpu") -> torch.Tensor:
    """h0 [T,d] in the storage dtype, with planted exit directions."""
    T, d, V = cfg["n_tokens"], cfg["d_model"], cfg["vocab_exit"]
    s = cfg["seed"] if token_seed is None else token_seed
    z = normal_f32(s, _ID_H0, (T, d), 1.0, "cpu")
    uv = uniform_f64(s, _ID_PLANT_V, T)
    uc = uniform_f64(s, _ID_PLANT_C, T)
    c_lo, c_hi = cfg["exit_plant"]
    scale = torch.tensor(SIGMA * math.sqrt(3.0) / 65536.0, dtype=torch.float32).item()
    off = torch.empty(T, d, dtype=torch.float64)
    for q in range(T):
        v = min(int(uv[q].item() * V), V - 1)
        # row v of W_lm, drawn by index (same bits as exit_lm on any device)
        raw = splitmix64_stream(cfg["seed"], _ID_WLM, v * d, d)
        fields = (raw & 0xFFFF) + ((raw >> 16) & 0xFFFF) + ((raw >> 32) & 0xFFFF) \
            + ((raw >> 48) & 0xFFFF)
        row = ((fields - 131070).to(torch.float32) * scale).to(torch.float64)
        c = c_lo + (c_hi - c_lo) * float(uc[q])
        off[q] = row * (c / float(row @ row))
    h = torch.add(z, off.to(torch.float32))
    return h.to(storage_dtype(cfg)).to(device)


def make_inputs(cfg, device="cpu", token_seed: int | None = None,
                with_layers: bool = True, layers=None) -> dict:
    """All inputs of one workload: {"cfg", "layers", "h0", "policy"}.

    ``layers`` (an iterable of layer indices) generates only those layers;
    the other entries of the returned list are None.  A layer's tensors do
    not depend on which other layers are generated.
    """
    w_lm = exit_lm(cfg, device)
    out_layers = []
    if with_layers:
        want = set(range(cfg["n_layers"])) if layers is None else set(layers)
        for l in range(cfg["n_layers"]):
            out_layers.append(make_layer(cfg, l, w_lm, device) if l in want else None)
    layers = out_layers
    del w_lm
    h0 = make_tokens(cfg, token_seed, device)
    policy = {k: cfg[k] for k in ("budget", "omega_t", "t_local", "t_remote",
                                  "phi_scale", "sim_min")}
    policy["p_exit"] = cfg["p_exit"]
    policy["horizon"] = int(cfg.get("horizon", 1))
    policy["la_subs"] = int(cfg.get("la_subs", 4))
    return dict(cfg=cfg, layers=layers, h0=h0, policy=policy)


_ID_STATE_ACTIVE = (1 << 40) + 32
_ID_STATE_DACC = (1 << 40) + 33


def mid_state(cfg, layer: int, seed: int, active_frac: float = 0.85,
              spent_frac: float = 0.9) -> dict:
    """A seeded stack state as it could stand before layer ``layer`` (> 0):
    a ragged subset of the tokens still active (each with probability
    ``active_frac``, at least one), the others marked as exited at an earlier
    layer; budget already spent per active token uniform over
    [0, spent_frac * budget].  Plain draws: no decision is computed here.
    Returns numpy arrays in the oracle's state layout (h is filled in by the
    caller from the generated tokens)."""
    import numpy as np
    if layer < 1:
        raise ValueError("mid_state: every token is active before layer 0")
    T, N = cfg["n_tokens"], cfg["n_layers"]
    ua = uniform_f64(seed, _ID_STATE_ACTIVE, T).numpy()
    ud = uniform_f64(seed, _ID_STATE_DACC, T).numpy()
    active = ua < active_frac
    if not active.any():
        active[int(np.argmin(ua))] = True
    budget = float(np.float32(cfg["budget"]))
    d_acc = np.where(active, ud * spent_frac * budget, 0.0).astype(np.float32).astype(np.float64)
    exit_layer = np.where(active, N, (np.arange(T) % layer)).astype(np.int64)
    xi = np.full(T, np.nan)
    return dict(d_acc=d_acc, active=np.nonzero(active)[0].tolist(),
                exit_layer=exit_layer, xi=xi)
