"""Engine-clock record of the GEMM kernels (trimmoe_set_clock_record, a
measurement aid): it fills exactly the GEMM classes that ran, with a clock in
a plausible range, leaves every result bit-identical, and stops when
cleared."""
import numpy as np
import pytest
import torch

from paper_2608_00573_amd import abi
from synthgen import make_inputs, workload

from gpu_harness import GpuRun, gpu_state_np, gpu_trace_np, log

pytestmark = pytest.mark.gpu

CASES = {
    # the first core: 128-row expert tiles, the shared expert, 256-token
    # exit tiles
    "first_core": dict(dtype="bf16", act="swiglu", top_k=2, normalize_topk=1, n_layers=3,
                       n_tokens=512, d_model=128, d_ff=256, d_ff_shared=128),
    # the large-group core: 1024 rows per expert on average and d = 2048
    # (k_ffn_big up/gate and down, k_exit_big)
    "large_group_core": dict(dtype="bf16", act="swiglu", n_experts=2, n_local=1, top_k=1,
                             n_layers=2, n_tokens=2048, d_model=2048, d_ff=512,
                             vocab_exit=1024),
}


@pytest.mark.parametrize("case", list(CASES))
def test_clock_record(case):
    cfg = workload("tiny_fp32", **CASES[case])
    inp = make_inputs(cfg)
    g = GpuRun(inp)
    log(f"[clock] {case}: T={cfg['n_tokens']} d={cfg['d_model']} E={cfg['n_experts']}")
    st0, tr0 = g.stack()
    rec = torch.zeros(2 * len(abi.TIMED_CLASSES), dtype=torch.int64, device=g.dev)
    abi.trimmoe_set_clock_record(rec)
    try:
        st1, tr1 = g.stack()
    finally:
        abi.trimmoe_set_clock_record(None)
    got = rec.cpu().numpy().copy()
    g.stack()  # cleared: nothing more is added
    assert np.array_equal(rec.cpu().numpy(), got)
    # the same work, bit for bit
    a, b = gpu_state_np(st0), gpu_state_np(st1)
    for key in ("h", "exit_layer", "xi", "d_acc"):
        assert np.array_equal(a[key], b[key]), key
    assert a["active"] == b["active"]
    ta, tb = gpu_trace_np(tr0), gpu_trace_np(tr1)
    for key in ta:
        assert np.array_equal(np.nan_to_num(ta[key], nan=-7.0),
                              np.nan_to_num(tb[key], nan=-7.0)), key
    # exactly the GEMM classes that ran, each with cycles and ticks
    ran = {"up", "down", "exit"} | ({"shared"} if cfg["d_ff_shared"] else set())
    words = dict(zip(abi.TIMED_CLASSES, got.reshape(-1, 2).tolist()))
    for c, (cycles, ticks) in words.items():
        assert (cycles > 0 and ticks > 0) == (c in ran), (c, cycles, ticks)
    mhz = abi.clock_mhz(rec)
    log(f"[clock] {case}: {mhz}")
    assert set(mhz) == ran
    for c, f in mhz.items():
        assert 100.0 <= f <= 3000.0, (c, f)
