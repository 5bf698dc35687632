"""The seeded generator: published splitmix64, device-independent bits."""
import math

import torch

from synthgen import rng, make_inputs, workload
from synthgen.inputs import exit_lm, twins, placement

M64 = (1 << 64) - 1


def _splitmix64_reference(state, n):
    # Vigna's splitmix64, as published: state += golden; mix the state.
    out = []
    for _ in range(n):
        state = (state + 0x9E3779B97F4A7C15) & M64
        z = state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
        out.append(z ^ (z >> 31))
    return out


def test_stream_is_published_splitmix64():
    for seed, tid in [(1, 0), (2, 12345), (99, 1 << 40)]:
        key = rng.key_for(seed, tid)
        ref = _splitmix64_reference(key, 50)
        got = [int(v) & M64 for v in rng.splitmix64_stream(seed, tid, 0, 50)]
        assert got == ref
        # random access: element 37 alone
        one = int(rng.splitmix64_stream(seed, tid, 37, 1)[0]) & M64
        assert one == ref[37]


def test_known_splitmix64_vector():
    # splitmix64 seeded with 0: first output is 0xE220A8397B1DCDAF
    assert _splitmix64_reference(0, 1)[0] == 0xE220A8397B1DCDAF


def test_normal_moments_and_bounds():
    x = rng.normal_f32(7, 3, (1 << 18,), 1.0).double()
    assert abs(x.mean().item()) < 0.01
    assert abs(x.std().item() - 1.0) < 0.01
    assert x.abs().max().item() <= math.sqrt(3.0) * 2 + 1e-6


def test_uniform_range():
    u = rng.uniform_f64(5, 1, 10000)
    assert u.min().item() >= 0.0 and u.max().item() < 1.0
    assert abs(u.mean().item() - 0.5) < 0.01


def test_permutation():
    p = rng.permutation(3, 4, 60)
    assert sorted(p.tolist()) == list(range(60))


def test_tiny_inputs_structure():
    cfg = workload("tiny_fp32")
    inp = make_inputs(cfg)
    for l, L in enumerate(inp["layers"]):
        sim = L["sim"].double()
        assert torch.allclose(sim, sim.T)
        assert torch.all(torch.diagonal(sim) == 1.0)
        assert int(L["local_mask"].sum()) == cfg["n_local"]
        tw, alpha = L["twin"], L["alpha"]
        for e, t in enumerate(tw):
            if t >= 0:
                assert L["local_mask"][t] == 1 and L["local_mask"][e] == 0
                # planted twins: cosine close to alpha
                assert abs(sim[e, t].item() - alpha[e].item()) < 0.05
    assert inp["h0"].shape == (cfg["n_tokens"], cfg["d_model"])


def test_exit_rows_by_index_match_full_draw():
    cfg = workload("tiny_fp32")
    full = exit_lm(cfg)
    d = cfg["d_model"]
    raw = rng.splitmix64_stream(cfg["seed"], 1 << 40, 5 * d, d)
    fields = (raw & 0xFFFF) + ((raw >> 16) & 0xFFFF) + ((raw >> 32) & 0xFFFF) \
        + ((raw >> 48) & 0xFFFF)
    scale = torch.tensor(0.02 * math.sqrt(3.0) / 65536.0, dtype=torch.float32).item()
    row = (fields - 131070).to(torch.float32) * scale
    assert torch.equal(row, full[5])


def test_seeded_reproducible():
    cfg = workload("tiny_fp32")
    a = make_inputs(cfg)
    b = make_inputs(cfg)
    assert torch.equal(a["h0"], b["h0"])
    assert torch.equal(a["layers"][1]["w_down"], b["layers"][1]["w_down"])
    assert placement(cfg, 0).tolist() == placement(cfg, 0).tolist()
    tw0, al0 = twins(cfg, 0, placement(cfg, 0))
    assert tw0 == twins(cfg, 0, placement(cfg, 0))[0]
