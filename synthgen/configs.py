"""Workload shapes for the adaptive-depth MoE step.

Each workload is named by the backbone whose MoE-layer shapes it borrows;
weights and hidden states are always synthetic (seeded).  The dictionaries
carry shapes, storage dtype, the policy scalars of the online rule
(confidence requirement p_J, per-token budget, delay/quality weights,
normalised per-slot delays) and the knobs of the synthetic recipe.
"""
from __future__ import annotations

import copy

_COMMON_POLICY = dict(budget=0.02, omega_t=0.5, t_local=1.0, t_remote=100.0,
                      phi_scale=1.0, sim_min=-1.0,
                      # exit confidence: max softmax of a vocabulary head, or the
                      # sigmoid of a one-row head (vocab_exit = 1)
                      conf_mode="softmax",
                      # look-ahead horizon H (1: the myopic rule), the support of
                      # each row of the expert transition matrices it reads, and the
                      # local substitute candidates per remote slot it weighs
                      horizon=1, trans_support=4, la_subs=4)

WORKLOADS = {
    # 2 layers, d=64, ReLU 64->256->64, 8 experts top-1, 64 tokens, fp32
    "tiny_fp32": dict(
        n_layers=2, d_model=64, n_experts=8, top_k=1, d_ff=256, d_ff_shared=0,
        vocab_exit=512, n_tokens=64, dtype="f32", act="relu",
        normalize_topk=0, n_local=4, seed=1, p_exit=0.5,
        theta_sorted=False, zipf_bias=0.0, down_sigma_scale=False,
        exit_gamma=(1.0, 2.0), exit_plant=(0.0, 10.0), twin_alpha_log10=(-4.0, -1.0),
        **_COMMON_POLICY),
    # Switch-Base-8E MoE layers: d=768, ReLU 768->3072->768, 8 experts top-1
    "switch_base_8e": dict(
        n_layers=6, d_model=768, n_experts=8, top_k=1, d_ff=3072, d_ff_shared=0,
        vocab_exit=32128, n_tokens=4096, dtype="bf16", act="relu",
        normalize_topk=0, n_local=3, seed=2, p_exit=0.9,
        theta_sorted=True, zipf_bias=0.0, down_sigma_scale=False,
        exit_gamma=(1.0, 2.0), exit_plant=(0.0, 16.0), twin_alpha_log10=(-4.0, -1.0),
        **_COMMON_POLICY),
    # Qwen-MoE-A2.7B MoE layers: d=2048, 60 SwiGLU experts 2048->1408 top-4,
    # shared SwiGLU expert 2048->5632
    "qwen_moe_a2_7b": dict(
        n_layers=24, d_model=2048, n_experts=60, top_k=4, d_ff=1408,
        d_ff_shared=5632, vocab_exit=151936, n_tokens=8192, dtype="bf16",
        act="swiglu", normalize_topk=0, n_local=20, seed=3, p_exit=0.9,
        theta_sorted=True, zipf_bias=0.0, down_sigma_scale=True,
        exit_gamma=(1.0, 2.0), exit_plant=(0.0, 18.0), twin_alpha_log10=(-4.0, -1.0),
        **_COMMON_POLICY),
    # Mixtral-8x7B MoE layers, prefill: d=4096, 8 SwiGLU experts 4096->14336
    # top-2, Zipf(1.1)-skewed router bias
    "mixtral_8x7b_prefill": dict(
        n_layers=32, d_model=4096, n_experts=8, top_k=2, d_ff=14336,
        d_ff_shared=0, vocab_exit=32000, n_tokens=8192, dtype="bf16",
        act="swiglu", normalize_topk=1, n_local=4, seed=4, p_exit=0.9,
        theta_sorted=True, zipf_bias=1.1, down_sigma_scale=True,
        exit_gamma=(1.0, 2.0), exit_plant=(0.0, 16.0), twin_alpha_log10=(-4.0, -1.0),
        **_COMMON_POLICY),
    # Mixtral-8x7B shapes at decode: 32 tokens per step, 128 steps, p_J=0.3
    "mixtral_8x7b_decode": dict(
        n_layers=32, d_model=4096, n_experts=8, top_k=2, d_ff=14336,
        d_ff_shared=0, vocab_exit=32000, n_tokens=32, dtype="bf16",
        act="swiglu", normalize_topk=1, n_local=4, seed=4, p_exit=0.3,
        theta_sorted=True, zipf_bias=1.1, down_sigma_scale=True,
        exit_gamma=(1.0, 2.0), exit_plant=(0.0, 16.0), twin_alpha_log10=(-4.0, -1.0),
        decode_steps=128, token_seed_base=5000,
        **_COMMON_POLICY),
}


def workload(name: str, **overrides) -> dict:
    """A copy of a named workload with fields overridden (e.g. n_tokens)."""
    if name not in WORKLOADS:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(WORKLOADS)}")
    cfg = copy.deepcopy(WORKLOADS[name])
    cfg["name"] = name
    for k, v in overrides.items():
        if k not in cfg and k not in ("token_seed",):
            raise KeyError(f"unknown workload field {k!r}")
        cfg[k] = v
    return cfg
