"""Host-side checks of the C ABI: symbols, workspace sizing, validation.

Nothing here launches a kernel: every call either is host-only
(trimmoe_workspace_size, trimmoe_status_str, trimmoe_abi_version) or fails
validation, which happens before any HIP call.
"""
import ctypes as C
import os
import re

import numpy as np
import pytest
import torch

from paper_2608_00573_amd import abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    txt = open(os.path.join(ROOT, "include", "trimmoe.h")).read()
    return sorted(set(re.findall(r"^\w[\w\s\*]*?\b(trimmoe_\w+)\s*\(", txt, re.M)))


def test_header_declares_the_binding_exports():
    assert _declared() == sorted(abi.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = abi.lib()
    for name in _declared():
        assert hasattr(L, name), name
    txt = open(os.path.join(ROOT, "include", "trimmoe.h")).read()
    declared = int(re.search(r"#define TRIMMOE_ABI_VERSION (\d+)", txt).group(1))
    assert abi.trimmoe_abi_version() == declared == abi.ABI_VERSION
    assert abi.trimmoe_status_str(0) == "ok"
    assert "workspace" in abi.trimmoe_status_str(-6)


def _fake_layers(n, E, with_gate=True, shared=False):
    # host tensors used only for their (non-null, aligned) addresses; no call
    # below reaches a kernel
    t = torch.zeros(64, dtype=torch.float32)
    L = dict(w_router=t, b_router=None, w_up=t, w_gate=t if with_gate else None, w_down=t,
             ws_up=t if shared else None, ws_gate=t if shared else None,
             ws_down=t if shared else None, w_exit=t, b_exit=None, local_mask=t, sim=t,
             theta=0.5, skip_slope=0.01)
    return [dict(L) for _ in range(n)]


DIMS = dict(n_layers=2, d_model=64, n_experts=8, top_k=2, d_ff=128, d_ff_shared=0,
            vocab_exit=512, dtype="bf16", act="swiglu", normalize_topk=1)


def _handle(**over):
    dims = dict(DIMS, **over)
    return abi.model_handle(dims, _fake_layers(dims["n_layers"], dims["n_experts"],
                                               dims["act"] == "swiglu", dims["d_ff_shared"] > 0))


def test_workspace_size_grows_with_tokens():
    mh = _handle()
    a = abi.trimmoe_workspace_size(mh.model, 64)
    b = abi.trimmoe_workspace_size(mh.model, 4096)
    assert 0 < a < b
    assert abi.trimmoe_workspace_size(mh.model, 0) > 0


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_workspace_size_covers_every_smaller_batch(dtype):
    # a workspace sized for max_tokens serves any smaller batch, also across
    # the switch to finer exit-head tiles for decode-sized batches
    mh = _handle(dtype=dtype)
    sizes = [abi.trimmoe_workspace_size(mh.model, t) for t in range(1, 200)]
    assert all(x <= y for x, y in zip(sizes, sizes[1:]))


# the full per-layer dimensions of the Switch-, Qwen1.5-MoE- and
# Mixtral-shaped workloads (only the dimensions matter to the sizing)
FULL_DIMS = {
    "switch_base_8e": dict(n_layers=6, d_model=768, n_experts=8, top_k=1, d_ff=3072,
                           d_ff_shared=0, vocab_exit=32128, act="relu", normalize_topk=0),
    "qwen_moe_a2_7b": dict(n_layers=24, d_model=2048, n_experts=60, top_k=4, d_ff=1408,
                           d_ff_shared=5632, vocab_exit=151936, act="swiglu",
                           normalize_topk=0),
    "mixtral_8x7b": dict(n_layers=32, d_model=4096, n_experts=8, top_k=2, d_ff=14336,
                         d_ff_shared=0, vocab_exit=32000, act="swiglu", normalize_topk=1),
}


def _accepts(L, mh, pol, T, bytes_):
    """Whether a stack call on T tokens accepts a workspace of bytes_ bytes.
    The call stops before any HIP work: after the workspace check it rejects
    the wrong event count (TRIMMOE_ERR_SHAPE); a workspace that is too small
    gives TRIMMOE_ERR_WORKSPACE first.  No pointer is dereferenced."""
    st = abi.State(T, 256, 256, 256, 256, 256, 256)
    ev = (C.c_void_p * 1)(C.c_void_p(256))
    rc = L.trimmoe_stack_forward_timed(C.byref(mh.model), C.byref(pol), C.byref(st), None,
                                       C.c_void_p(256), bytes_, None, ev, 1)
    assert rc in (-2, -6), rc
    return rc == -2


@pytest.mark.parametrize("name", sorted(FULL_DIMS))
def test_workspace_for_max_tokens_serves_every_smaller_batch(name):
    # the down GEMM's K split and the exit head's vocabulary tile both change
    # with the batch size; a workspace sized for max_tokens must still be
    # accepted by every batch of at most max_tokens tokens (measured failures
    # of an earlier sizing: 18048 tokens under a size for 18112, 12032 under
    # one for 12992, at the Switch dimensions)
    dims = dict(FULL_DIMS[name], dtype="bf16")
    mh = abi.model_handle(dims, _fake_layers(dims["n_layers"], dims["n_experts"],
                                             dims["act"] == "swiglu", dims["d_ff_shared"] > 0))
    L = abi.lib()
    pol = abi.make_policy(**POL)
    sizes = np.array([abi.trimmoe_workspace_size(mh.model, t) for t in range(0, 40001)])
    assert np.all(np.diff(sizes) >= 0), "workspace size shrinks with more tokens"
    for tmax in (64, 65, 1600, 1665, 12032, 12992, 18048, 18112, 40000):
        ws = int(sizes[tmax])
        for t in sorted({1, 2, 63, 64, 65, 127, 128, 129, tmax // 3, tmax // 2, tmax - 1, tmax}
                        | set(range(max(1, tmax - 300), tmax + 1, 7))):
            if 1 <= t <= tmax:
                assert _accepts(L, mh, pol, t, ws), (tmax, t)
        assert not _accepts(L, mh, pol, tmax, ws - 1)
    # every batch up to 40000 tokens under the size for 40000, and each at its own size
    ws = int(sizes[40000])
    for t in range(1, 40001, 13):
        assert _accepts(L, mh, pol, t, ws), t
        assert _accepts(L, mh, pol, t, int(sizes[t])), t


@pytest.mark.parametrize("over,code", [
    (dict(top_k=9), -2), (dict(n_experts=257, top_k=2), -2), (dict(top_k=9, n_experts=8), -2),
    (dict(d_model=96), -2), (dict(d_ff=100), -2), (dict(n_layers=0), -2),
    (dict(dtype="f32", d_model=66), -2),
])
def test_workspace_size_rejects_bad_shapes(over, code):
    mh = _handle(**over)
    with pytest.raises(abi.TrimmoeError) as ei:
        abi.trimmoe_workspace_size(mh.model, 16)
    assert ei.value.status == code


def test_bad_enums_rejected():
    mh = _handle()
    mh.model.dtype = 7
    with pytest.raises(abi.TrimmoeError) as ei:
        abi.trimmoe_workspace_size(mh.model, 16)
    assert ei.value.status == -3
    mh = _handle()
    mh.model.conf_mode = 1  # sigmoid needs V == 1
    with pytest.raises(abi.TrimmoeError) as ei:
        abi.trimmoe_workspace_size(mh.model, 16)
    assert ei.value.status == -2


def test_missing_gate_and_shared_pointers():
    mh = abi.model_handle(dict(DIMS), _fake_layers(2, 8, with_gate=False))
    with pytest.raises(abi.TrimmoeError) as ei:
        abi.trimmoe_workspace_size(mh.model, 16)
    assert ei.value.status == -1
    mh = abi.model_handle(dict(DIMS, d_ff_shared=128), _fake_layers(2, 8))
    with pytest.raises(abi.TrimmoeError) as ei:
        abi.trimmoe_workspace_size(mh.model, 16)
    assert ei.value.status == -1


def _state_stub(T=16):
    t = torch.zeros(max(T, 1) * 64, dtype=torch.float32)
    return abi.State(T, t.data_ptr(), t.data_ptr(), t.data_ptr(), t.data_ptr(), t.data_ptr(),
                     t.data_ptr()), t


POL = dict(p_exit=0.9, budget=0.02, omega_t=0.5, t_local=1.0, t_remote=100.0, phi_scale=1.0,
           sim_min=-1.0)


@pytest.mark.parametrize("over,code", [
    (dict(omega_t=1.5), -4), (dict(budget=-0.1), -4), (dict(p_exit=float("nan")), -4),
    (dict(t_remote=-1.0), -4), (dict(phi_scale=float("inf")), -4),
])
def test_layer_step_rejects_bad_policy_before_launch(over, code):
    mh = _handle()
    st, keep = _state_stub()
    pol = abi.make_policy(**dict(POL, **over))
    ws = torch.zeros(1 << 20, dtype=torch.uint8)
    with pytest.raises(abi.TrimmoeError) as ei:
        abi.trimmoe_layer_step(mh.model, 0, pol, st, None, ws, stream=torch.cuda.Stream
                               if False else _NullStream())
    assert ei.value.status == code
    assert torch.count_nonzero(keep) == 0  # nothing written


class _NullStream:
    cuda_stream = 0


def test_layer_step_rejects_bad_layer_workspace_and_state():
    mh = _handle()
    st, keep = _state_stub()
    pol = abi.make_policy(**POL)
    L = abi.lib()
    need = abi.trimmoe_workspace_size(mh.model, 16)
    big = torch.zeros(need + 512, dtype=torch.uint8)
    off = (-big.data_ptr()) % 256
    ws = big[off:off + need]
    # layer out of range
    rc = L.trimmoe_layer_step(C.byref(mh.model), 2, C.byref(pol), C.byref(st), None,
                              C.c_void_p(ws.data_ptr()), need, None)
    assert rc == -5
    # workspace too small / misaligned / NULL
    rc = L.trimmoe_layer_step(C.byref(mh.model), 0, C.byref(pol), C.byref(st), None,
                              C.c_void_p(ws.data_ptr()), need - 1, None)
    assert rc == -6
    rc = L.trimmoe_layer_step(C.byref(mh.model), 0, C.byref(pol), C.byref(st), None,
                              C.c_void_p(ws.data_ptr() + 16), need, None)
    assert rc == -6
    rc = L.trimmoe_stack_forward(C.byref(mh.model), C.byref(pol), C.byref(st), None, None,
                                 need, None)
    assert rc == -6
    # NULL state member
    st.xi = None
    rc = L.trimmoe_stack_forward(C.byref(mh.model), C.byref(pol), C.byref(st), None,
                                 C.c_void_p(ws.data_ptr()), need, None)
    assert rc == -1
    # NULL model / policy
    rc = L.trimmoe_stack_forward(None, C.byref(pol), C.byref(st), None,
                                 C.c_void_p(ws.data_ptr()), need, None)
    assert rc == -1
    assert torch.count_nonzero(keep) == 0
    assert torch.count_nonzero(ws) == 0


def _la_layers(n, E, B, with_trans=True):
    layers = _fake_layers(n, E)
    to = torch.zeros(E, B, dtype=torch.int16)
    pr = torch.zeros(E, B, dtype=torch.float32)
    for i, L in enumerate(layers):
        L["trans_to"] = to if with_trans and i < n - 1 else None
        L["trans_p"] = pr if with_trans and i < n - 1 else None
    return layers


@pytest.mark.parametrize("over,B,horizon,subs,code", [
    (dict(), 4, 5, 4, -4),                      # horizon above the maximum
    (dict(), 4, 0, 4, -4),                      # horizon below 1
    (dict(), 4, 2, 0, -4),                      # no substitute candidate weighed
    (dict(), 4, 2, 5, -4),                      # more candidates than the maximum
    (dict(n_experts=16, top_k=5), 2, 2, 1, -2),  # look-ahead needs top-k <= 4
    (dict(), 9, 2, 1, -2),                      # rows of more than 8 entries
    (dict(n_experts=16, top_k=4), 3, 2, 1, -2),  # (2^4 + 1) * 81 first-level branches > 1024
    (dict(n_experts=16, top_k=4), 2, 2, 2, -2),  # (3^4 + 1) * 16 first-level branches > 1024
    (dict(n_layers=4, top_k=2), 8, 4, 1, -2),   # 5^4 * 64^3 evaluations > 2^23
    (dict(n_layers=4, top_k=2), 4, 4, 4, -2),   # 26^4 * 16^3 evaluations > 2^23
])
def test_look_ahead_limits_rejected_before_launch(over, B, horizon, subs, code):
    dims = dict(DIMS, **over)
    mh = abi.model_handle(dims, _la_layers(dims["n_layers"], dims["n_experts"], B))
    st, keep = _state_stub()
    pol = abi.make_policy(**POL, horizon=horizon, la_subs=subs)
    rc = abi.lib().trimmoe_stack_forward(C.byref(mh.model), C.byref(pol), C.byref(st), None,
                                         None, 0, None)
    assert rc == code
    assert torch.count_nonzero(keep) == 0


def test_look_ahead_needs_the_transitions_a_decision_reads():
    dims = dict(DIMS, n_layers=3)
    mh = abi.model_handle(dims, _la_layers(3, 8, 4, with_trans=False))
    st, _ = _state_stub()
    st.xi = None  # a call that passes the look-ahead checks stops at the state
    pol = abi.make_policy(**POL, horizon=2)
    L = abi.lib()
    assert L.trimmoe_stack_forward(C.byref(mh.model), C.byref(pol), C.byref(st), None, None, 0,
                                   None) == -2   # trans_b = 0
    mh = abi.model_handle(dims, _la_layers(3, 8, 4))
    mh.layers[1].trans_to = None
    assert L.trimmoe_stack_forward(C.byref(mh.model), C.byref(pol), C.byref(st), None, None, 0,
                                   None) == -1   # layer 1's decision reads P_1
    # layer 0 at H = 2 reads only P_0; the last layer reads nothing
    for layer in (0, 2):
        assert L.trimmoe_layer_step(C.byref(mh.model), layer, C.byref(pol), C.byref(st), None,
                                    None, 0, None) == -1   # the NULL state member
    assert L.trimmoe_layer_step(C.byref(mh.model), 1, C.byref(pol), C.byref(st), None, None, 0,
                                None) == -1
    pol3 = abi.make_policy(**POL, horizon=3)
    assert L.trimmoe_layer_step(C.byref(mh.model), 0, C.byref(pol3), C.byref(st), None, None, 0,
                                None) == -1


def test_static_entry_validates_before_any_device_call():
    # the allocation-free entry point checks its arguments and its array's
    # size limit before touching the device: a batch larger than the array
    # is rejected with TRIMMOE_ERR_WORKSPACE, bad arguments as usual
    dims = dict(FULL_DIMS["switch_base_8e"], dtype="bf16")
    mh = abi.model_handle(dims, _fake_layers(dims["n_layers"], dims["n_experts"], False))
    L = abi.lib()
    pol = abi.make_policy(**POL)
    T = 8192
    assert abi.trimmoe_workspace_size(mh.model, T) > abi.STATIC_SCRATCH_BYTES
    st = abi.State(T, 256, 256, 256, 256, 256, 256)
    assert L.trimmoe_stack_forward_static(C.byref(mh.model), C.byref(pol), C.byref(st), None,
                                          None) == -6
    bad = abi.make_policy(**dict(POL, omega_t=2.0))
    assert L.trimmoe_stack_forward_static(C.byref(mh.model), C.byref(bad), C.byref(st), None,
                                          None) == -4
    st.xi = None
    assert L.trimmoe_stack_forward_static(C.byref(mh.model), C.byref(pol), C.byref(st), None,
                                          None) == -1


def test_empty_batch_is_a_no_op_without_device_calls():
    # a batch of no tokens: every entry point that runs the path validates
    # its arguments and returns TRIMMOE_OK before any device call, writing
    # nothing (so this runs without a GPU)
    mh = _handle()
    L = abi.lib()
    pol = abi.make_policy(**POL)
    st, keep = _state_stub(T=0)
    need = abi.trimmoe_workspace_size(mh.model, 0)
    assert need > 0
    big = torch.zeros(need + 512, dtype=torch.uint8)
    off = (-big.data_ptr()) % 256
    ws = big[off:off + need]
    assert L.trimmoe_state_reset(C.byref(mh.model), C.byref(st), None) == 0
    assert L.trimmoe_stack_forward(C.byref(mh.model), C.byref(pol), C.byref(st), None,
                                   C.c_void_p(ws.data_ptr()), need, None) == 0
    for layer in range(DIMS["n_layers"]):
        assert L.trimmoe_layer_step(C.byref(mh.model), layer, C.byref(pol), C.byref(st), None,
                                    C.c_void_p(ws.data_ptr()), need, None) == 0
    assert L.trimmoe_stack_forward_static(C.byref(mh.model), C.byref(pol), C.byref(st), None,
                                          None) == 0
    # arguments are still checked first: a bad policy or a missing workspace
    bad = abi.make_policy(**dict(POL, budget=-1.0))
    assert L.trimmoe_stack_forward(C.byref(mh.model), C.byref(bad), C.byref(st), None,
                                   C.c_void_p(ws.data_ptr()), need, None) == -4
    assert L.trimmoe_stack_forward(C.byref(mh.model), C.byref(pol), C.byref(st), None, None,
                                   need, None) == -6
    assert torch.count_nonzero(keep) == 0
    assert torch.count_nonzero(ws) == 0
