"""GPU parity of the exit-head training of Sec. IV-A: the output head's
argmax (the predictions behind the consistency labels of Eq. (22)) and the
BCE gradient descent of Eq. (23), against the oracle on seeded inputs; then
heads trained on a GPU calibration pass drive a sigmoid-mode stack."""
import numpy as np
import pytest
import torch

import oracle as O
from oracle import exit_head as X
from paper_2608_00573_amd import abi, offline
from synthgen import make_inputs, workload
from synthgen.rng import normal_f32

from gpu_harness import GpuRun, check_invariants_gpu, gpu_state_np, gpu_trace_np, log, policy32

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _mat(seed, tid, shape, sigma, dtype):
    t = normal_f32(seed, tid, shape, sigma, "cpu").to(dtype)
    return t, t.double().numpy()


@pytest.mark.parametrize("dtype,V,d,Q", [
    (torch.float32, 1000, 64, 100),
    (torch.bfloat16, 32128, 768, 50),     # decode-sized: 128 x 32 tiles
    (torch.bfloat16, 5000, 128, 700),     # 256 x 128 tiles, ragged vocabulary
    (torch.bfloat16, 3000, 64, 4100),     # 256 x 256 tiles
])
def test_head_argmax_matches_oracle(dtype, V, d, Q):
    log(f"[exit-head] argmax {dtype} V={V} d={d} Q={Q}")
    W, Wn = _mat(11, 1, (V, d), 0.02, dtype)
    H, Hn = _mat(12, 2, (Q, d), 1.0, dtype)
    got = abi.trimmoe_head_argmax(W.to(DEV), H.to(DEV)).cpu().numpy()
    want, margin = X.head_argmax(Wn, Hn)
    clear = margin > 1e-5       # fp32 accumulation of the same stored values
    assert clear.mean() > 0.99
    assert np.array_equal(got[clear], want[clear])


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_training_matches_oracle(dtype):
    Q, d, epochs, lr = 1000, 128, 60, 0.5
    H, Hn = _mat(21, 3, (Q, d), 1.0, dtype)
    u = normal_f32(21, 4, (d,), 1.0, "cpu").double().numpy()
    y = (Hn @ u + 0.5 > 0).astype(np.uint8)                  # a planted linear rule
    w = torch.zeros(d, dtype=torch.float32, device=DEV)
    c = torch.zeros(1, dtype=torch.float32, device=DEV)
    loss = torch.zeros(epochs, dtype=torch.float32, device=DEV)
    Hd, yd = H.to(DEV), torch.from_numpy(y).to(DEV)
    abi.trimmoe_train_exit_head(Hd, yd, epochs, lr, w, c, loss)
    torch.cuda.synchronize()
    ww, cw, lw = X.train_exit_head(Hn, y, epochs, lr)
    log(f"[exit-head] train {dtype}: loss {lw[0]:.4f} -> {lw[-1]:.4f}, "
        f"max |dw| {np.abs(w.cpu().numpy() - ww).max():.2e}")
    assert np.allclose(w.cpu().numpy(), ww, rtol=1e-4, atol=1e-5)
    assert c.item() == pytest.approx(cw, rel=1e-4, abs=1e-5)
    assert np.allclose(loss.cpu().numpy(), lw, rtol=1e-5, atol=1e-6)
    # deterministic: a second run from the same start gives identical weights
    w2 = torch.zeros_like(w)
    c2 = torch.zeros_like(c)
    abi.trimmoe_train_exit_head(Hd, yd, epochs, lr, w2, c2)
    torch.cuda.synchronize()
    assert torch.equal(w, w2) and torch.equal(c, c2)


def test_trained_heads_drive_a_sigmoid_stack():
    # no planted exit direction and wider experts, so that some tokens'
    # predictions still change after layer 0 (labels of both kinds)
    cfg = workload("tiny_fp32", n_layers=4, n_tokens=512, exit_plant=(0.0, 0.0), d_ff=1024)
    inp = make_inputs(cfg)
    g = GpuRun(inp)
    hs = offline.calibration_hidden_states(g.mh.model, inp["policy"], inp["h0"].to(g.dev), g.ws)
    w_head = g.layers[-1]["w_exit"]
    labels = offline.consistency_labels(hs, w_head)

    # the oracle's own full-depth pass and labels (Eq. (22))
    model = O.model_from_inputs(inp)
    pol = policy32(dict(inp["policy"], budget=0.0, p_exit=2.0, horizon=1))
    st = O.init_state(inp["h0"].double().numpy(), cfg["n_layers"])
    ref_h = []
    for l in range(cfg["n_layers"]):
        O.layer_step(model, l, pol, st)
        ref_h.append(st["h"].copy())
    Wn = model["layers"][cfg["n_layers"] - 1]["w_exit"]
    final, mf = X.head_argmax(Wn, ref_h[-1])
    for l in range(cfg["n_layers"] - 1):
        pred, ml = X.head_argmax(Wn, ref_h[l])
        want = X.consistency_labels(pred, final)
        clear = (ml > 1e-5) & (mf > 1e-5)
        got = labels[l].cpu().numpy()
        assert np.array_equal(got[clear], want[clear]), l
        assert 0 < want.sum() < len(want)
        log(f"[exit-head] layer {l}: {int(want.sum())} of {len(want)} consistent")

    trained = offline.train_sigmoid_heads(hs[:-1], labels, 200, 1.0)
    for w, c, loss in trained:
        assert loss[-1].item() < loss[0].item()
    # a sigmoid-mode model whose layers carry the trained heads (the last
    # layer's head is never read)
    cfg2 = dict(cfg, vocab_exit=1, conf_mode="sigmoid")
    layers = []
    for l, L in enumerate(g.layers):
        L = dict(L)
        w, c = trained[min(l, len(trained) - 1)][:2]
        L["w_exit"] = w.reshape(1, -1).contiguous()
        L["b_exit"] = c.clone()
        layers.append(L)
    g2 = GpuRun(dict(inp, cfg=cfg2), layers_dev=layers)
    # a requirement between the trained confidences: some tokens exit early
    st2, tr2 = g2.stack(pol=dict(inp["policy"], p_exit=0.97))
    gst, gtr = gpu_state_np(st2), gpu_trace_np(tr2)
    check_invariants_gpu(cfg2, policy32(dict(inp["policy"], p_exit=0.97)), gst, gtr)
    xi = gtr["xi"][~np.isnan(gtr["xi"])]
    assert xi.size and np.all((xi >= 0) & (xi <= 1))
    log(f"[exit-head] sigmoid stack: exits {int((gst['exit_layer'] < cfg['n_layers']).sum())}")
