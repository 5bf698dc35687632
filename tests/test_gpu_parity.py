"""GPU parity of the HIP path (through the C ABI) against the CPU oracle."""
import numpy as np
import pytest
import torch

import oracle as O
from synthgen import make_inputs, workload

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests.gpu_harness import (GpuRun, check_invariants_gpu, compare_stack, gpu_state_np,
                                   gpu_trace_np, log, oracle_run, policy32, teacher_forced)


def _run_and_compare(cfg, pol=None, edit=None, **kw):
    inp = make_inputs(cfg)
    if edit is not None:
        edit(inp)
    log(f"[parity] {cfg['name']} T={cfg['n_tokens']} N={cfg['n_layers']} {kw}")
    g = GpuRun(inp)
    st, tr = g.stack(pol=pol, **{k: v for k, v in kw.items() if k in ("p_exit_tok", "budget_tok")})
    gst, gtr = gpu_state_np(st), gpu_trace_np(tr)
    ref_state, ref_traces = oracle_run(inp, pol=pol, token_budget=kw.get("budget_tok"),
                                       token_p_exit=kw.get("p_exit_tok"))
    stats = compare_stack(cfg, ref_state, ref_traces, gst, gtr)
    check_invariants_gpu(cfg, policy32(inp["policy"] if pol is None else pol), gst, gtr,
                         kw.get("budget_tok"), kw.get("p_exit_tok"))
    log(f"[parity] ok {stats}")
    return inp, gst, gtr, ref_state, ref_traces, stats


def test_tiny_fp32_stack():
    cfg = workload("tiny_fp32")
    _, gst, gtr, ref, _, stats = _run_and_compare(cfg)
    assert stats["excluded_tokens"] <= 4
    # the recipe reaches every branch of the rule on this case
    assert (gtr["action"] == O.ACT_SKIP).any()
    assert (gtr["kind"] == O.KIND_SUB).any()
    assert (gst["exit_layer"] < cfg["n_layers"]).any()


def test_tiny_bf16_swiglu_top2_shared():
    cfg = workload("tiny_fp32", dtype="bf16", act="swiglu", top_k=2, d_ff_shared=128,
                   normalize_topk=1, n_layers=3)
    _run_and_compare(cfg)


@pytest.mark.parametrize("dtype,act", [("f32", "relu"), ("f32", "swiglu"), ("bf16", "relu")])
def test_shared_expert_with_every_routed_activation(dtype, act):
    # the shared expert (SwiGLU) beside ReLU or SwiGLU routed experts, on the
    # fp32 path and beside ReLU on the bf16 path (the bf16 SwiGLU case is
    # above); 200 tokens leave ragged route, row and token tiles
    cfg = workload("tiny_fp32", dtype=dtype, act=act, top_k=2, normalize_topk=1,
                   d_ff_shared=192, n_tokens=200, n_layers=3)
    _run_and_compare(cfg)


def test_large_batch_swiglu_top2_shared():
    # 6144 tokens: the 256-token exit-head tile; top-2 over 4 experts gives
    # long, ragged expert groups
    cfg = workload("tiny_fp32", dtype="bf16", act="swiglu", top_k=2, normalize_topk=1,
                   n_tokens=6144, d_model=128, d_ff=256, n_experts=4, n_local=2,
                   vocab_exit=2048, n_layers=3, d_ff_shared=256)
    _run_and_compare(cfg)


def test_large_batch_relu_top1():
    cfg = workload("switch_base_8e", n_tokens=6500, n_layers=3, d_model=128, d_ff=384,
                   n_experts=2, n_local=1, vocab_exit=1500)
    _run_and_compare(cfg)


def test_large_expert_groups_skewed_ragged():
    # Mixtral-like routing (top-2 of 8, Zipf-skewed router bias) at 4096
    # tokens: 1024 rows per expert on average, so the expert GEMMs take
    # 256-row tiles; d_ff = 576 and d_model = 320 leave partial column tiles
    # in the up/gate (128-column) and down (256-column) GEMMs
    cfg = workload("mixtral_8x7b_prefill", n_tokens=4096, n_layers=2, d_model=320, d_ff=576,
                   vocab_exit=1000)
    # the library picks 256-row tiles from the batch shape: T k >= 1024 E
    assert cfg["n_tokens"] * cfg["top_k"] >= 1024 * cfg["n_experts"]
    _run_and_compare(cfg)


def test_decode_sized_swiglu_split_down_ragged():
    # a decode-sized batch (29 tokens, a few rows per expert) at bf16:
    # d_model 576 leaves a partial 256-column down tile, d_ff 1152 gives the
    # down GEMM two K splits, and the exit head takes its decode tile
    # (vocabulary 1000: a partial 128-row tile)
    cfg = workload("mixtral_8x7b_decode", n_tokens=29, n_layers=3, d_model=576, d_ff=1152,
                   vocab_exit=1000)
    _run_and_compare(cfg)


def test_decode_sized_relu_top1_ragged_up():
    # ReLU up tiles (256 columns) over d_ff 704 leave a partial tile; 32
    # tokens over 8 experts
    cfg = workload("switch_base_8e", n_tokens=32, n_layers=3, d_model=512, d_ff=704,
                   vocab_exit=1000)
    _run_and_compare(cfg)


def test_wide_model_exit_head_ragged():
    # d_model 2048 at 1100 tokens: the exit head takes 256 x 256 tiles with
    # 4 wavefronts; 1100 tokens and 1000 vocabulary rows leave partial token
    # and vocabulary tiles
    cfg = workload("tiny_fp32", dtype="bf16", n_tokens=1100, d_model=2048, d_ff=256,
                   n_experts=4, n_local=2, vocab_exit=1000, n_layers=2)
    _run_and_compare(cfg)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sigmoid_exit_head(dtype):
    # the paper's own exit head: one logit w . h + b through a sigmoid
    # (p_J = 0.99: the planted logits cross 4.6 at different depths)
    cfg = workload("tiny_fp32", dtype=dtype, vocab_exit=1, conf_mode="sigmoid", n_layers=4,
                   n_tokens=200, p_exit=0.99)
    _, gst, gtr, _, _, _ = _run_and_compare(cfg)
    exits = [(gst["exit_layer"] == l).sum() for l in range(cfg["n_layers"])]
    assert sum(e > 0 for e in exits) >= 2


def test_many_experts_bf16_top4_substitution():
    # 160 SwiGLU experts, top-4, 80 local, in bf16: each lane of the
    # substitute table's wavefront scans two or three candidates (160 =
    # 2 x 64 + 32) and the router's MFMA tiles span 10 expert column tiles
    cfg = workload("qwen_moe_a2_7b", n_tokens=512, n_layers=2, d_model=256, d_ff=128,
                   d_ff_shared=128, n_experts=160, n_local=80, vocab_exit=1000)
    _, _, gtr, _, _, _ = _run_and_compare(cfg)
    assert (gtr["kind"] == O.KIND_SUB).any()
    assert (gtr["action"] == O.ACT_SKIP).any()


def test_max_experts_and_top_k_bf16():
    # the library's maxima together: 256 SwiGLU experts, top-8, 128 of them
    # local, bf16 (a whole wavefront per token in top-k and softmax, every
    # token's Eq. (34) enumeration over 8 slots, up to 256 groups of a few
    # rows in the expert GEMMs), 300 tokens (a ragged route block)
    cfg = workload("qwen_moe_a2_7b", n_tokens=300, n_layers=2, d_model=128, d_ff=128,
                   d_ff_shared=128, n_experts=256, n_local=128, top_k=8, vocab_exit=512)
    _, _, gtr, _, _, _ = _run_and_compare(cfg)
    assert (gtr["kind"] == O.KIND_SUB).any()
    assert (gtr["action"] == O.ACT_SKIP).any()


@pytest.mark.parametrize("E,k", [(8, 2), (60, 4)])
def test_tied_router_logits_rank_lower_id_first(E, k):
    # router rows duplicated in pairs: experts 2j and 2j + 1 get bitwise equal
    # logits, so the rank order takes 2j first and its twin right after it
    # (8 experts: 8-lane groups per token; 60: a whole wavefront per token)
    cfg = workload("tiny_fp32", dtype="bf16", n_experts=E, n_local=E // 2, top_k=k,
                   normalize_topk=1, n_tokens=300, n_layers=2)

    def tie(inp):
        for L in inp["layers"]:
            L["w_router"][1::2] = L["w_router"][0::2]

    _, _, gtr, _, _, _ = _run_and_compare(cfg, edit=tie)
    tgt = gtr["target"].reshape(cfg["n_layers"], cfg["n_tokens"], k)
    live = tgt[..., 0] >= 0
    for r in range(0, k, 2):
        assert np.all(tgt[..., r][live] % 2 == 0)
        assert np.all(tgt[..., r + 1][live] == tgt[..., r][live] + 1)


def test_ragged_tokens_bf16_relu():
    # T not a multiple of any tile (route 32, GEMM 128)
    cfg = workload("switch_base_8e", n_tokens=333, n_layers=3, d_model=256, d_ff=512,
                   vocab_exit=1000)
    _run_and_compare(cfg)


def test_single_token():
    cfg = workload("tiny_fp32", n_tokens=1, n_layers=3)
    _run_and_compare(cfg)


def test_all_tokens_exit_after_first_layer():
    # p_J = 0: every token exits after layer 0, later layers see n_active = 0
    cfg = workload("tiny_fp32", n_layers=4)
    inp = make_inputs(cfg)
    pol = dict(inp["policy"], p_exit=0.0)
    _, gst, gtr, _, _, _ = _run_and_compare(cfg, pol=pol)
    # a token exits right after its first executed layer; a skipped layer
    # never triggers an exit (Eq. (9)), so skippers stay active until then
    act = gtr["action"]
    for t in range(cfg["n_tokens"]):
        first = int(np.argmax(act[:, t] == O.ACT_EXEC)) if (act[:, t] == O.ACT_EXEC).any() else None
        if first is not None and first < cfg["n_layers"] - 1:
            assert gst["exit_layer"][t] == first
            assert np.all(act[first + 1:, t] == O.ACT_INACTIVE)
            assert np.all(act[:first, t] == O.ACT_SKIP)
    assert (act[0] == O.ACT_EXEC).sum() > 0


def test_zero_budget_and_per_token_arrays():
    cfg = workload("tiny_fp32", n_layers=3)
    inp = make_inputs(cfg)
    T = cfg["n_tokens"]
    budget_tok = np.where(np.arange(T) % 2 == 0, 0.0, 0.05).astype(np.float32)
    pexit_tok = np.where(np.arange(T) % 3 == 0, 2.0, 0.5).astype(np.float32)
    _, gst, _, _, _, _ = _run_and_compare(cfg, budget_tok=budget_tok, p_exit_tok=pexit_tok)
    assert np.all(gst["d_acc"][budget_tok == 0] == 0)


def test_switch_base_full_size():
    # the benchmark workload: 6 layers, d=768, 8 experts top-1, 4096 tokens
    cfg = workload("switch_base_8e")
    _, gst, gtr, _, _, stats = _run_and_compare(cfg)
    # a token leaves the comparison at its first decision within 1e-3 of a
    # threshold; over 6 layers that is ~8% of tokens on this recipe
    assert stats["excluded_tokens"] < 0.10 * cfg["n_tokens"]
    c = gtr["counters"]
    log(f"[switch] counters per layer (active, exec, skip, exit, subst, remote, rows, experts):\n{c}")
    assert c[:, 2].sum() > 0 and c[:, 3].sum() > 0 and c[:, 4].sum() > 0


def test_determinism_bitwise():
    cfg = workload("switch_base_8e", n_tokens=1024, n_layers=3)
    inp = make_inputs(cfg)
    g = GpuRun(inp)
    st1, tr1 = g.stack()
    st2, tr2 = g.stack()
    assert torch.equal(st1.h, st2.h)
    for k in ("action", "exec", "gate", "xi", "d_acc", "counters"):
        assert torch.equal(getattr(tr1, k).nan_to_num(0) if getattr(tr1, k).is_floating_point()
                           else getattr(tr1, k),
                           getattr(tr2, k).nan_to_num(0) if getattr(tr2, k).is_floating_point()
                           else getattr(tr2, k)), k


@pytest.mark.parametrize("shape", ["large_groups", "wide_exit"])
def test_determinism_bitwise_large_tiles(shape):
    # the large-group expert GEMMs (256-row tiles, dense shared expert) and the
    # large-tile exit head: fixed K order and no atomics, so repeated passes
    # are bit-identical
    if shape == "large_groups":
        cfg = workload("tiny_fp32", dtype="bf16", act="swiglu", top_k=2, normalize_topk=1,
                       n_tokens=4096, d_model=192, d_ff=320, n_experts=4, n_local=2,
                       vocab_exit=700, n_layers=2, d_ff_shared=256)
    else:
        cfg = workload("tiny_fp32", dtype="bf16", n_tokens=1100, d_model=2048, d_ff=256,
                       n_experts=4, n_local=2, vocab_exit=1000, n_layers=2)
    g = GpuRun(make_inputs(cfg))
    st1, tr1 = g.stack()
    st2, tr2 = g.stack()
    assert torch.equal(st1.h, st2.h)
    for k in ("action", "exec", "gate", "xi", "d_acc", "counters"):
        a, b = getattr(tr1, k), getattr(tr2, k)
        if a.is_floating_point():
            a, b = a.nan_to_num(0), b.nan_to_num(0)
        assert torch.equal(a, b), k


def test_switch_base_teacher_forced_layers():
    # every layer of the benchmark workload on 1024 tokens, fed the oracle's
    # exact state: decisions bit-exact outside a 1e-5 band
    cfg = workload("switch_base_8e", n_tokens=1024)
    stats = teacher_forced(make_inputs(cfg))
    assert sum(s["excluded_tokens"] for s in stats) < 0.01 * 1024 * cfg["n_layers"]


def test_tiny_fp32_teacher_forced():
    teacher_forced(make_inputs(workload("tiny_fp32", n_layers=3)))
