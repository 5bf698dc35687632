"""Full stacks at the Qwen- and Mixtral-shaped workloads, every layer checked.

The GPU runs the whole stack over every token of the batch: layer 0 sees the
full batch, so the largest executed-token count goes through every kernel,
the exit head included, and the GPU's own state flows from layer to layer
(it never sees an oracle value).  The stack runs twice: once through
trimmoe_stack_forward (the launch configuration bench.py times), once as
trimmoe_state_reset plus trimmoe_layer_step per layer, with a seeded sample
of tokens read back between layers; the two runs must agree bit for bit.
Tokens are independent in this step (no attention, per-token decisions and
budgets), so the oracle then re-computes each layer for the sampled tokens
from the GPU's state before that layer, and the GPU's state and trace after
it must match: decisions exactly outside a 1e-5 band (1e-3 for the exit
gate, which reads the layer's rounded output), hidden states within 2e-2,
and each token's confidence xi within the exact shift that the difference
of the two rounded outputs makes through the exit head (fp32 slack added).
What holds at any size (Properties 2 and 3, masks, counters) is checked on
every token.  The Mixtral-shaped weights also serve the first decode steps
(32 fresh tokens each, p_J = 0.3), every token checked; those four steps form
one runtime-feedback window (Sec. V-D, V-F) whose GPU sums and host update
must match the oracle's, and a fifth step runs on the updated policy.

A free-running comparison (each side feeding its own output onward) is not
used at these depths: bf16 rounding flips of the two sides' hidden states
accumulate over 24-32 layers and move router logits by more than any fixed
band, so decisions would legitimately part.

The oracle walks the layers one at a time; each layer's stored weights are
widened to fp64 into buffers allocated once (exact: bf16 values are fp64
values), so the host never holds more than one layer in fp64.
"""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2608_00573_amd import abi
from synthgen import make_inputs, workload
from synthgen.inputs import make_tokens

from gpu_harness import (BAND, check_invariants_gpu, compare_stack, gpu_state_np, gpu_trace_np,
                         log, policy32, xi_rtol_from_outputs)

pytestmark = pytest.mark.gpu

_BIG = ("w_router", "w_up", "w_gate", "w_down", "ws_up", "ws_gate", "ws_down", "w_exit")


class _Widen:
    """One layer at a time as the oracle's fp64 model, through buffers
    allocated (and first touched) once per tensor name."""

    def __init__(self, inp):
        self.inp = inp
        self.f64, self.stage = {}, {}
        L0 = inp["layers"][0]
        for key in _BIG:
            t = L0.get(key)
            if t is None:
                continue
            self.stage[key] = torch.empty(t.shape, dtype=t.dtype, pin_memory=True)
            self.f64[key] = torch.zeros(t.shape, dtype=torch.float64)

    def model(self, l):
        L = dict(self.inp["layers"][l])
        for key, buf in self.f64.items():
            self.stage[key].copy_(L[key])
            buf.copy_(self.stage[key])
            L[key] = buf  # a CPU fp64 tensor: the oracle's conversion is then a view
        view = dict(self.inp, layers=[L if j == l else None
                                      for j in range(len(self.inp["layers"]))])
        return O.model_from_inputs(view, layers=[l])


def _sample(T, n, seed):
    rng = np.random.default_rng(seed)
    pick = set(rng.choice(T, size=n - 2, replace=False).tolist()) | {0, T - 1}
    return np.array(sorted(pick))


def _gpu_stack(mh, policy, h0, N, k, dev):
    T = h0.shape[0]
    ws = abi.alloc_workspace(mh.model, T, dev)
    st = abi.StateBuffers(h0.to(dev).clone())
    tr = abi.TraceBuffers(N, T, k, dev)
    abi.trimmoe_stack_forward(mh.model, policy, st.state, tr.trace, ws)
    torch.cuda.synchronize()
    return gpu_state_np(st), gpu_trace_np(tr), st, tr


def _gpu_rows(st, idx):
    """The sampled tokens' part of a GPU state, as the oracle holds a state."""
    n = int(st.n_active.item())
    act = set(st.active_idx[:n].cpu().numpy().tolist())
    ix = torch.as_tensor(idx, device=st.h.device)
    return dict(h=st.h[ix].double().cpu().numpy(), d_acc=st.d_acc[ix].double().cpu().numpy(),
                active=[i for i, t in enumerate(idx) if int(t) in act],
                exit_layer=st.exit_layer[ix].cpu().numpy().astype(np.int64),
                xi=st.xi[ix].double().cpu().numpy())


def _counters_agree(gtr):
    """Per-layer trace counters against the per-token trace, every token."""
    act, c = gtr["action"], gtr["counters"]
    for l in range(act.shape[0]):
        alive = act[l] != O.ACT_INACTIVE
        assert c[l, 0] == alive.sum() and c[l, 1] == (act[l] == O.ACT_EXEC).sum()
        assert c[l, 2] == (act[l] == O.ACT_SKIP).sum()


class _Run:
    """One batch: the stack pass, then the same stack layer by layer."""

    def __init__(self, label, cfg, mh, pol, h0, idx, dev):
        N, k = cfg["n_layers"], cfg["top_k"]
        self.label, self.cfg, self.pol, self.idx = label, cfg, pol, idx
        policy = abi.make_policy(**pol)
        log(f"[fullstack] {label}: trimmoe_stack_forward over {h0.shape[0]} tokens")
        self.ref_state, self.ref_trace, self.dev_state, self.dev_trace = \
            _gpu_stack(mh, policy, h0, N, k, dev)
        self.policy = policy
        check_invariants_gpu(cfg, pol, self.ref_state, self.ref_trace)
        _counters_agree(self.ref_trace)
        # the same stack, one layer step at a time, the sampled rows read back
        T = h0.shape[0]
        ws = abi.alloc_workspace(mh.model, T, dev)
        st = abi.StateBuffers(h0.to(dev).clone())
        tr = abi.TraceBuffers(N, T, k, dev)
        abi.trimmoe_state_reset(mh.model, st.state)
        self.before = []
        for l in range(N):
            self.before.append(_gpu_rows(st, idx))
            abi.trimmoe_layer_step(mh.model, l, policy, st.state, tr.trace, ws)
        self.after = self.before[1:] + [_gpu_rows(st, idx)]
        torch.cuda.synchronize()
        gst, gtr = gpu_state_np(st), gpu_trace_np(tr)
        # stack pass = reset + layer steps, bit for bit
        assert np.array_equal(gst["h"], self.ref_state["h"])
        assert np.array_equal(gst["exit_layer"], self.ref_state["exit_layer"])
        assert gst["active"] == self.ref_state["active"]
        for key in ("action", "target", "exec", "kind", "counters"):
            assert np.array_equal(gtr[key], self.ref_trace[key]), key
        for key in ("gate", "importance", "xi", "d_acc"):
            assert np.array_equal(np.nan_to_num(gtr[key], nan=-7.0),
                                  np.nan_to_num(self.ref_trace[key], nan=-7.0)), key
        self.trace = {key: v[:, idx] for key, v in gtr.items() if key != "counters"}
        self.stats = dict(compared=0, layers=0)

    def check_layer(self, model, l):
        """Oracle layer l from the GPU's state before it, against the GPU's
        state and trace after it."""
        ost = {key: (list(v) if key == "active" else np.array(v, copy=True))
               for key, v in self.before[l].items()}
        if not ost["active"]:
            return
        rtr = O.layer_step(model, l, policy32(self.pol), ost)
        gst = self.after[l]
        # xi reads the layer's rounded output, which already differs from the
        # oracle's by bf16 rounding flips: each token's xi gets the shift its
        # two outputs imply exactly through the exit head, plus fp32 slack
        xr = xi_rtol_from_outputs(model["layers"][l], model["conf_mode"], ost["h"], gst["h"])
        s = compare_stack(self.cfg, ost, [rtr], gst, self.trace, band=1e-5, layer0=l,
                          ftol="forced", band_exit=BAND, xi_rtol=xr)
        self.stats["xi_rtol_max"] = max(self.stats.get("xi_rtol_max", 0.0),
                                        float(xr[~np.isnan(rtr["xi"])].max(initial=0.0)))
        self.stats["xi_rel_max"] = max(self.stats.get("xi_rel_max", 0.0),
                                       max(s.get("xi_max_rel", [0.0])))
        # the active list after the layer (stable compaction), outside the band
        inb = set(np.nonzero((rtr["margin_pre"] <= 1e-5) | (rtr["margin_exit"] <= BAND))[0])
        assert [t for t in gst["active"] if t not in inb] == \
            [t for t in ost["active"] if t not in inb], f"layer {l}: active list"
        self.stats["compared"] += s["compared"]
        self.stats["layers"] += 1
        self.stats["max_rel_err"] = max(self.stats.get("max_rel_err", 0.0), s["max_rel_err"])


# runtime feedback after the decode window (the decode bench's defaults)
FB_ETA, FB_KAPPA, FB_FLOOR = 0.2, 0.2, 0.1
KEYS = ("tokens", "exits", "xi_exit", "util", "delay", "delay_ref")


def _feedback_window(cfg, inp, mh, runs, dpol):
    """The window's observations (Sec. V-D, V-F) summed on the GPU over the
    decode runs against the oracle's sums of the same passes' states and
    traces, then the library's host update (Eq. (37), Eq. (43)) against the
    oracle's; returns the updated policy."""
    N = cfg["n_layers"]
    stats = torch.zeros(6, dtype=torch.float64, device=runs[0].dev_state.h.device)
    for r in runs:
        abi.trimmoe_window_stats(mh.model, r.policy, r.dev_state.state, r.dev_trace.trace, stats)
    torch.cuda.synchronize()
    got = stats.cpu().numpy()
    model = dict(n_layers=N, top_k=cfg["top_k"],
                 layers={l: dict(local_mask=inp["layers"][l]["local_mask"].cpu().numpy())
                         for l in range(N)})
    ref = np.zeros(6)
    for r in runs:
        tr = [dict(action=r.ref_trace["action"][l], target=r.ref_trace["target"][l],
                   kind=r.ref_trace["kind"][l]) for l in range(N)]
        st = O.window_stats(model, policy32(dpol), r.ref_state, tr)
        ref += np.array([st[key] for key in KEYS])
    log(f"[fullstack] feedback window: gpu {got.tolist()} oracle {ref.tolist()}")
    # counts exactly; the fp64 sums up to their order
    assert got[0] == ref[0] and got[1] == ref[1]
    assert np.allclose(got[2:], ref[2:], rtol=1e-12, atol=1e-12)
    assert got[1] > 0 and got[4] > 0
    policy = abi.make_policy(**dpol)
    abi.trimmoe_feedback_update(policy, got.tolist(), FB_ETA, FB_KAPPA, FB_FLOOR)
    rp, rw = O.feedback_update(policy32(dpol), dict(zip(KEYS, ref.tolist())), FB_ETA, FB_KAPPA,
                               FB_FLOOR)
    assert policy.p_exit == pytest.approx(rp, abs=2e-6)
    assert policy.omega_t == pytest.approx(rw, abs=2e-6)
    assert (policy.p_exit, policy.omega_t) != (policy32(dpol)["p_exit"],
                                               policy32(dpol)["omega_t"])
    return dict(dpol, p_exit=float(policy.p_exit), omega_t=float(policy.omega_t))


def _full_stack(name, n_sample, seed, decode_steps=0):
    cfg = workload(name)
    N, T = cfg["n_layers"], cfg["n_tokens"]
    dev = torch.device("cuda:0")
    log(f"[fullstack] {name}: generating all {N} layers on the GPU")
    inp = make_inputs(cfg, device=dev)
    mh = abi.model_handle(cfg, inp["layers"])
    runs = [_Run("prefill", cfg, mh, inp["policy"], inp["h0"], _sample(T, n_sample, seed), dev)]
    if decode_steps:
        dcfg = workload("mixtral_8x7b_decode")
        assert dcfg["seed"] == cfg["seed"] and dcfg["d_model"] == cfg["d_model"]
        dpol = dict(inp["policy"], p_exit=dcfg["p_exit"])
        for s in range(decode_steps):
            hd = make_tokens(dcfg, dcfg["token_seed_base"] + s, dev)
            runs.append(_Run(f"decode{s}", dcfg, mh, dpol, hd, np.arange(hd.shape[0]), dev))
        # the decode steps form one feedback window; the next step runs on
        # the updated policy
        dpol = _feedback_window(dcfg, inp, mh, runs[1:], dpol)
        hd = make_tokens(dcfg, dcfg["token_seed_base"] + decode_steps, dev)
        runs.append(_Run(f"decode{decode_steps}", dcfg, mh, dpol, hd, np.arange(hd.shape[0]),
                         dev))
    log(f"[fullstack] {name}: oracle over {N} layers, one layer in fp64 at a time")
    wid = _Widen(inp)
    for l in range(N):
        if not any(r.before[l]["active"] for r in runs):
            break  # no sampled token reaches this layer
        model = wid.model(l)
        for r in runs:
            r.check_layer(model, l)
        del model
    out = {}
    for r in runs:
        log(f"[fullstack] {name} {r.label}: {r.stats}")
        out[r.label] = r.stats
    return out, runs[0].ref_trace


def test_qwen_full_stack_sampled_tokens():
    # 24 layers, 60 experts top-4 + shared expert, V = 151936, 8192 tokens
    out, gtr = _full_stack("qwen_moe_a2_7b", n_sample=32, seed=41)
    assert out["prefill"]["compared"] >= 200
    assert gtr["action"][0].min() != O.ACT_INACTIVE  # layer 0: the whole batch


def test_mixtral_full_stack_prefill_and_first_decode_steps():
    # 32 layers, 8 experts top-2, Zipf-skewed groups, 8192 tokens (the large-
    # group core, cut down-GEMM tiles); then 4 decode steps of 32 tokens on
    # the same weights, every token followed; the 4 steps form one feedback
    # window, and a fifth step runs on the updated p_J and omega_T
    out, gtr = _full_stack("mixtral_8x7b_prefill", n_sample=24, seed=42, decode_steps=4)
    assert out["prefill"]["compared"] >= 100
    assert gtr["action"][0].min() != O.ACT_INACTIVE
    for s in range(5):
        assert out[f"decode{s}"]["compared"] >= 32
