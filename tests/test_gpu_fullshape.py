"""Parity at the full per-layer shapes of the Qwen- and Mixtral-shaped workloads.

The GPU runs one layer (trimmoe_layer_step, the launch configuration of the
stack) over every token of the batch, from a seeded mid-stack state: a
ragged active subset and partly spent budgets.  Tokens are independent in
this step (no attention, per-token decisions and budgets), so the oracle
checks a seeded sample of tokens one by one; properties that hold at any
size (budget, exit gate, untouched inactive and skipped tokens, stable
compaction, trace counters) are checked on every token.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_00573_amd import abi
from synthgen import make_inputs, mid_state, workload
from synthgen.rng import normal_f32, uniform_f64

from gpu_harness import (BAND, compare_stack, gpu_state_np, gpu_trace_np, load_state, log,
                         policy32)

pytestmark = pytest.mark.gpu


def _full_layer(name, layer, n_sample, seed, **over):
    cfg = workload(name, **over)
    N, T, k, H = cfg["n_layers"], cfg["n_tokens"], cfg["top_k"], cfg["horizon"]
    dev = torch.device("cuda:0")
    ahead = list(range(layer + 1, min(layer + H, N)))  # layers the look-ahead reads
    log(f"[fullshape] {name} layer {layer} T={T} H={H}: generating inputs on the GPU")
    inp = make_inputs(cfg, device=dev, layers=[layer] + ahead)
    L = inp["layers"][layer]
    # trimmoe_layer_step reads slot `layer` (and, looking ahead, the
    # decision inputs of the next H - 1 slots); the others repeat it
    mh = abi.model_handle(cfg, [inp["layers"][j] if inp["layers"][j] is not None else L
                                for j in range(N)])
    ws = abi.alloc_workspace(mh.model, T, dev)
    policy = abi.make_policy(**inp["policy"])

    before = mid_state(cfg, layer, seed)
    before["h"] = inp["h0"].double().cpu().numpy()
    h_dev = inp["h0"].to(dev).clone()
    st = abi.StateBuffers(h_dev)
    load_state(st, before, cfg["dtype"])
    tr = abi.TraceBuffers(N, T, k, dev)
    log(f"[fullshape] {name} layer {layer}: trimmoe_layer_step over {len(before['active'])} "
        f"active of {T} tokens")
    abi.trimmoe_layer_step(mh.model, layer, policy, st.state, tr.trace, ws)
    torch.cuda.synchronize()
    gst = gpu_state_np(st)
    gtr = gpu_trace_np(tr)

    _check_all_tokens(cfg, layer, inp["policy"], before, gst, gtr)

    # oracle on a seeded sample: active tokens (first, last and random ones)
    # plus a few inactive ones, which must stay untouched
    rng = np.random.default_rng(seed)
    act = before["active"]
    if n_sample >= T:
        idx = np.arange(T)
    else:
        inactive = sorted(set(range(T)) - set(act))
        pick = set(rng.choice(act, size=min(n_sample, len(act)), replace=False).tolist())
        pick |= {act[0], act[-1]}
        if inactive:
            pick |= set(rng.choice(inactive, size=min(4, len(inactive)), replace=False).tolist())
        idx = np.array(sorted(pick))
    aset = set(act)
    sub = dict(h=before["h"][idx].copy(), d_acc=before["d_acc"][idx].copy(),
               active=[i for i, t in enumerate(idx) if t in aset],
               exit_layer=before["exit_layer"][idx].copy(), xi=before["xi"][idx].copy())
    log(f"[fullshape] {name} layer {layer}: oracle on {len(idx)} sampled tokens")
    model = O.model_from_inputs(inp, layers=[layer], decision_layers=ahead)
    pol = policy32(inp["policy"])
    rtr = O.layer_step(model, layer, pol, sub)
    g_sub = {key: v[:, idx] for key, v in gtr.items() if key != "counters"}
    gst_sub = dict(h=gst["h"][idx], d_acc=gst["d_acc"][idx],
                   exit_layer=gst["exit_layer"][idx], xi=gst["xi"][idx])
    stats = compare_stack(cfg, sub, [rtr], gst_sub, g_sub, band=1e-5, layer0=layer,
                          ftol="forced", band_exit=BAND)
    stats["sampled"] = len(idx)
    log(f"[fullshape] {name} layer {layer}: {stats}")
    return stats, gtr, layer


def _check_all_tokens(cfg, l, pol, before, gst, gtr):
    """What holds for every token of one layer step, at any size."""
    N, T = cfg["n_layers"], cfg["n_tokens"]
    act = gtr["action"][l]
    alive = np.zeros(T, bool)
    alive[before["active"]] = True
    # inactive tokens: untouched state, no trace
    assert np.all(act[~alive] == O.ACT_INACTIVE)
    assert np.array_equal(gst["h"][~alive], before["h"][~alive])
    assert np.array_equal(gst["exit_layer"][~alive], before["exit_layer"][~alive])
    # every active token executes or skips (never empty)
    assert np.all((act[alive] == O.ACT_EXEC) | (act[alive] == O.ACT_SKIP))
    # Property 2: budget never exceeded (fp32 slack)
    budget = np.float32(pol["budget"])
    assert np.all(gst["d_acc"][alive] <= budget * (1 + 1e-6) + 1e-9)
    assert np.all(gst["d_acc"][alive] >= before["d_acc"][alive] - 1e-9)
    # skipped tokens: h unchanged, no confidence evaluated (Eq. (9))
    sk = act == O.ACT_SKIP
    assert np.array_equal(gst["h"][sk], before["h"][sk])
    assert np.all(np.isnan(gtr["xi"][l][sk]))
    # Property 3: exits only after an executed layer with xi >= p_J; none at
    # the last layer
    ex = gst["exit_layer"] == l
    assert np.all(act[ex] == O.ACT_EXEC)
    assert np.all(gtr["xi"][l][ex] >= np.float32(pol["p_exit"]))
    if l == N - 1:
        assert not ex.any()
    # stable compaction of the active list
    assert gst["active"] == [t for t in before["active"] if gst["exit_layer"][t] == N]
    # executed slots are the target or a local expert; the counters agree
    L_exec = gtr["exec"][l]
    rows = 0
    used = set()
    for t in np.nonzero(act == O.ACT_EXEC)[0]:
        ids = {int(x) for x in L_exec[t] if x >= 0}
        rows += len(ids)
        used |= ids
    c = gtr["counters"][l]
    assert c[0] == alive.sum() and c[1] == (act == O.ACT_EXEC).sum()
    assert c[2] == sk.sum() and c[3] == ex.sum()
    assert c[6] == rows and c[7] == len(used)


def test_generator_bits_identical_on_gpu():
    """The GPU-generated inputs these tests use equal the CPU generator's."""
    a = normal_f32(4, 12345, (1 << 20,), 0.02, "cuda:0").cpu()
    b = normal_f32(4, 12345, (1 << 20,), 0.02, "cpu")
    assert torch.equal(a, b)
    u = uniform_f64(4, 777, 4096, "cuda:0").cpu()
    assert torch.equal(u, uniform_f64(4, 777, 4096, "cpu"))
    cfg = workload("tiny_fp32", dtype="bf16", d_model=64, d_ff=128, act="swiglu")
    g = make_inputs(cfg, device="cuda:0", layers=[1])["layers"][1]
    c = make_inputs(cfg, device="cpu", layers=[1])["layers"][1]
    for key in ("w_router", "w_up", "w_gate", "w_down", "w_exit", "local_mask"):
        assert torch.equal(g[key].cpu(), c[key]), key
    assert torch.allclose(g["sim"].cpu(), c["sim"], rtol=0, atol=1e-6)


def test_mixtral_prefill_full_layer():
    stats, _, _ = _full_layer("mixtral_8x7b_prefill", 16, n_sample=24, seed=31)
    assert stats["compared"] >= 20


def test_mixtral_prefill_last_layer_no_exit():
    stats, gtr, l = _full_layer("mixtral_8x7b_prefill", 31, n_sample=12, seed=32)
    assert np.all(np.isnan(gtr["xi"][l]))


def test_qwen_full_layer_shared_expert():
    stats, _, _ = _full_layer("qwen_moe_a2_7b", 12, n_sample=24, seed=33)
    assert stats["compared"] >= 20


def test_mixtral_decode_full_layer_every_token():
    # 32 tokens: the oracle checks all of them
    stats, _, _ = _full_layer("mixtral_8x7b_decode", 16, n_sample=32, seed=34)
    assert stats["sampled"] == 32


@pytest.mark.parametrize("layer", [16, 30, 31])
def test_mixtral_decode_full_layer_look_ahead(layer):
    # H = 3 over 8 experts top-2 with 4-entry transition rows (16 tuples per
    # level); at layer 30 the horizon is cut to 2, at the last layer to 1
    stats, _, _ = _full_layer("mixtral_8x7b_decode", layer, n_sample=32, seed=35 + layer,
                              horizon=3)
    assert stats["sampled"] == 32 and stats["compared"] >= 16
