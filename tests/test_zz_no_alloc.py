"""The allocation-free entry point trimmoe_stack_forward_static against
trimmoe_stack_forward (caller workspace) on the same inputs, through the C ABI.

Both run the same kernels; only where the workspace lives differs (the
library's per-device scratch array instead of a caller buffer), so every
output and every trace field must be identical bit for bit.  Two calls in a
row, the second on a smaller batch, check that nothing carries over in the
shared array from one call to the next.
"""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2608_00573_amd import abi
from synthgen import make_inputs, workload

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from tests.gpu_harness import GpuRun, gpu_state_np, gpu_trace_np, log

CASES = {
    # fp32, 8 experts top-1 (every branch of the rule is reached)
    "tiny_fp32": (workload("tiny_fp32"), 64, 37),
    # bf16 SwiGLU top-2 with a shared expert
    "tiny_bf16_swiglu_shared": (workload("tiny_fp32", dtype="bf16", act="swiglu", top_k=2,
                                         d_ff_shared=128, normalize_topk=1, n_layers=3,
                                         n_tokens=300), 300, 129),
    # the Switch-shaped stack at its full batch, then a ragged smaller one
    "switch_base_8e": (workload("switch_base_8e"), 4096, 1333),
}


def _pair(g, h0, static):
    h = h0.to(g.dev).clone()
    st = abi.StateBuffers(h)
    tr = abi.TraceBuffers(g.cfg["n_layers"], h.shape[0], g.cfg["top_k"], g.dev)
    if static:
        abi.trimmoe_stack_forward_static(g.mh.model, g.policy(), st.state, tr.trace)
    else:
        abi.trimmoe_stack_forward(g.mh.model, g.policy(), st.state, tr.trace, g.ws)
    torch.cuda.synchronize()
    return gpu_state_np(st), gpu_trace_np(tr)


def _same(a, b, what):
    for key in a:
        x, y = np.asarray(a[key]), np.asarray(b[key])
        assert x.shape == y.shape and np.array_equal(x, y, equal_nan=x.dtype.kind == "f"), \
            f"{what}: {key} differs"


@pytest.mark.parametrize("name", list(CASES))
def test_static_entry_matches_workspace_entry(name):
    cfg, T1, T2 = CASES[name]
    inp = make_inputs(cfg)
    g = GpuRun(inp)
    # the batch fits the library's array
    assert abi.trimmoe_workspace_size(g.mh.model, T1) <= abi.STATIC_SCRATCH_BYTES
    for T in (T1, T2):  # two calls in a row, the second smaller
        log(f"[no-alloc] {name}: {T} tokens")
        h0 = inp["h0"][:T]
        ref_st, ref_tr = _pair(g, h0, static=False)
        got_st, got_tr = _pair(g, h0, static=True)
        _same(ref_st, got_st, f"{name} T={T} state")
        _same(ref_tr, got_tr, f"{name} T={T} trace")
        assert (ref_tr["action"] != 0).any()


def test_static_entry_rejects_batches_beyond_its_array():
    cfg = workload("switch_base_8e")
    inp = make_inputs(cfg, layers=[0])
    layers = [inp["layers"][0]] * cfg["n_layers"]
    g = GpuRun(dict(inp, layers=layers))
    T = 8192  # needs more than the array holds at the Switch dimensions
    assert abi.trimmoe_workspace_size(g.mh.model, T) > abi.STATIC_SCRATCH_BYTES
    h = torch.zeros(T, cfg["d_model"], dtype=torch.bfloat16, device=g.dev)
    st = abi.StateBuffers(h)
    rc = abi.lib().trimmoe_stack_forward_static(C.byref(g.mh.model), C.byref(g.policy()),
                                                C.byref(st.state), None, None)
    assert rc == -6
    torch.cuda.synchronize()
    assert torch.count_nonzero(h) == 0
