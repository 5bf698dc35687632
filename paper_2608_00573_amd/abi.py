"""ctypes binding of libtrimmoe (include/trimmoe.h): marshalling only.

Every step of the adaptive-depth MoE layer runs inside the HIP library;
this module only mirrors the C structs, passes device pointers taken from
torch tensors (torch provides device memory and streams) and turns status
codes into exceptions.  There is no fallback: if the library is missing
the import of ``lib()`` raises.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libtrimmoe.so")

ABI_VERSION = 6   # TRIMMOE_ABI_VERSION this binding is written for
STATIC_SCRATCH_BYTES = 64 << 20  # TRIMMOE_STATIC_SCRATCH_BYTES
N_COUNTERS = 16   # per-layer trace counters (row stride of trimmoe_trace.counters)
TRIMMOE_OK = 0
STATUS = {0: "OK", -1: "ERR_NULL", -2: "ERR_SHAPE", -3: "ERR_DTYPE", -4: "ERR_POLICY",
          -5: "ERR_LAYER", -6: "ERR_WORKSPACE", -7: "ERR_HIP"}
F32, BF16 = 0, 1
ACT_RELU, ACT_SWIGLU = 0, 1
CONF_SOFTMAX, CONF_SIGMOID = 0, 1
MAX_EXPERTS, MAX_TOPK = 256, 8


class Layer(C.Structure):
    _fields_ = [("w_router", C.c_void_p), ("b_router", C.c_void_p),
                ("w_up", C.c_void_p), ("w_gate", C.c_void_p), ("w_down", C.c_void_p),
                ("ws_up", C.c_void_p), ("ws_gate", C.c_void_p), ("ws_down", C.c_void_p),
                ("w_exit", C.c_void_p), ("b_exit", C.c_void_p),
                ("local_mask", C.c_void_p), ("sim", C.c_void_p),
                ("theta", C.c_float), ("skip_slope", C.c_float),
                ("trans_to", C.c_void_p), ("trans_p", C.c_void_p)]


class Model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_experts", C.c_int32),
                ("top_k", C.c_int32), ("d_ff", C.c_int32), ("d_ff_shared", C.c_int32),
                ("vocab_exit", C.c_int32), ("dtype", C.c_int32), ("act", C.c_int32),
                ("conf_mode", C.c_int32), ("normalize_topk", C.c_int32),
                ("layers", C.POINTER(Layer)), ("trans_b", C.c_int32)]


class Policy(C.Structure):
    _fields_ = [("p_exit", C.c_float), ("budget", C.c_float), ("omega_t", C.c_float),
                ("t_local", C.c_float), ("t_remote", C.c_float), ("phi_scale", C.c_float),
                ("sim_min", C.c_float), ("p_exit_tok", C.c_void_p),
                ("budget_tok", C.c_void_p), ("horizon", C.c_int32), ("la_subs", C.c_int32)]


class State(C.Structure):
    _fields_ = [("n_tokens", C.c_int32), ("h", C.c_void_p), ("d_acc", C.c_void_p),
                ("active_idx", C.c_void_p), ("n_active", C.c_void_p),
                ("exit_layer", C.c_void_p), ("xi", C.c_void_p)]


class Trace(C.Structure):
    _fields_ = [("action", C.c_void_p), ("target", C.c_void_p), ("exec", C.c_void_p),
                ("kind", C.c_void_p), ("gate", C.c_void_p), ("importance", C.c_void_p),
                ("xi", C.c_void_p), ("d_acc", C.c_void_p), ("counters", C.c_void_p)]


EXPORTS = ["trimmoe_abi_version", "trimmoe_status_str", "trimmoe_workspace_size",
           "trimmoe_state_reset", "trimmoe_layer_step", "trimmoe_stack_forward",
           "trimmoe_stack_forward_timed", "trimmoe_stack_forward_static",
           "trimmoe_set_clock_record",
           "trimmoe_window_stats", "trimmoe_feedback_update",
           "trimmoe_calib_exit_layers", "trimmoe_calib_stats", "trimmoe_calib_transitions",
           "trimmoe_place_replicas", "trimmoe_head_argmax_workspace_size",
           "trimmoe_head_argmax", "trimmoe_consistency_labels",
           "trimmoe_train_exit_head_workspace_size",
           "trimmoe_train_exit_head"]
TIMED_CLASSES = ["route", "bucket", "up", "down", "shared", "combine", "exit", "gate"]

_lib = None


def lib():
    """The loaded libtrimmoe.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "paper_2608_00573_amd.build.build() (there is no fallback)")
        L = C.CDLL(LIB_PATH)
        L.trimmoe_abi_version.restype = C.c_int
        L.trimmoe_status_str.restype = C.c_char_p
        L.trimmoe_status_str.argtypes = [C.c_int]
        L.trimmoe_workspace_size.restype = C.c_int
        L.trimmoe_workspace_size.argtypes = [C.POINTER(Model), C.c_int32, C.POINTER(C.c_size_t)]
        L.trimmoe_state_reset.restype = C.c_int
        L.trimmoe_state_reset.argtypes = [C.POINTER(Model), C.POINTER(State), C.c_void_p]
        L.trimmoe_layer_step.restype = C.c_int
        L.trimmoe_layer_step.argtypes = [C.POINTER(Model), C.c_int32, C.POINTER(Policy),
                                         C.POINTER(State), C.POINTER(Trace), C.c_void_p,
                                         C.c_size_t, C.c_void_p]
        L.trimmoe_stack_forward.restype = C.c_int
        L.trimmoe_stack_forward.argtypes = [C.POINTER(Model), C.POINTER(Policy),
                                            C.POINTER(State), C.POINTER(Trace), C.c_void_p,
                                            C.c_size_t, C.c_void_p]
        L.trimmoe_stack_forward_timed.restype = C.c_int
        L.trimmoe_stack_forward_timed.argtypes = [C.POINTER(Model), C.POINTER(Policy),
                                                  C.POINTER(State), C.POINTER(Trace),
                                                  C.c_void_p, C.c_size_t, C.c_void_p,
                                                  C.POINTER(C.c_void_p), C.c_int32]
        L.trimmoe_set_clock_record.restype = C.c_int
        L.trimmoe_set_clock_record.argtypes = [C.c_void_p]
        L.trimmoe_stack_forward_static.restype = C.c_int
        L.trimmoe_stack_forward_static.argtypes = [C.POINTER(Model), C.POINTER(Policy),
                                                   C.POINTER(State), C.POINTER(Trace),
                                                   C.c_void_p]
        L.trimmoe_window_stats.restype = C.c_int
        L.trimmoe_window_stats.argtypes = [C.POINTER(Model), C.POINTER(Policy),
                                           C.POINTER(State), C.POINTER(Trace), C.c_void_p,
                                           C.c_void_p]
        L.trimmoe_feedback_update.restype = C.c_int
        L.trimmoe_feedback_update.argtypes = [C.POINTER(Policy), C.POINTER(C.c_double),
                                              C.c_double, C.c_double, C.c_double]
        i32, f32, p = C.c_int32, C.c_float, C.c_void_p
        L.trimmoe_calib_exit_layers.restype = C.c_int
        L.trimmoe_calib_exit_layers.argtypes = [i32, i32, p, f32, p]
        L.trimmoe_calib_stats.restype = C.c_int
        L.trimmoe_calib_stats.argtypes = [i32, i32, i32, i32, p, p, p, p, p, p, p, p]
        L.trimmoe_calib_transitions.restype = C.c_int
        L.trimmoe_calib_transitions.argtypes = [i32, i32, i32, i32, p, p, i32, p, p]
        L.trimmoe_place_replicas.restype = C.c_int
        L.trimmoe_place_replicas.argtypes = [i32, i32, i32, p, p, p, p, p, p, p, p,
                                             C.POINTER(C.c_int32)]
        L.trimmoe_head_argmax_workspace_size.restype = C.c_int
        L.trimmoe_head_argmax_workspace_size.argtypes = [i32, i32, i32, C.POINTER(C.c_size_t)]
        L.trimmoe_head_argmax.restype = C.c_int
        L.trimmoe_head_argmax.argtypes = [i32, i32, i32, i32, p, p, p, p, p, C.c_size_t, p]
        L.trimmoe_consistency_labels.restype = C.c_int
        L.trimmoe_consistency_labels.argtypes = [i32, p, p, p, p]
        L.trimmoe_train_exit_head_workspace_size.restype = C.c_int
        L.trimmoe_train_exit_head_workspace_size.argtypes = [i32, C.POINTER(C.c_size_t)]
        L.trimmoe_train_exit_head.restype = C.c_int
        L.trimmoe_train_exit_head.argtypes = [i32, i32, i32, p, p, i32, f32, p, p, p, p,
                                              C.c_size_t, p]
        if L.trimmoe_abi_version() != ABI_VERSION:
            raise RuntimeError(f"{LIB_PATH} has ABI version {L.trimmoe_abi_version()}, the "
                               f"binding expects {ABI_VERSION}: rebuild it")
        _lib = L
    return _lib


class TrimmoeError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} returned {status} ({STATUS.get(status, '?')})")
        self.status = status


def _check(fn: str, rc: int):
    if rc != TRIMMOE_OK:
        raise TrimmoeError(fn, rc)


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream_handle(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


# ------------------------------------------------------------- wrappers ----
def trimmoe_abi_version() -> int:
    return lib().trimmoe_abi_version()


def trimmoe_status_str(status: int) -> str:
    return lib().trimmoe_status_str(status).decode()


def trimmoe_workspace_size(model: Model, max_tokens: int) -> int:
    out = C.c_size_t(0)
    _check("trimmoe_workspace_size",
           lib().trimmoe_workspace_size(C.byref(model), max_tokens, C.byref(out)))
    return out.value


def trimmoe_state_reset(model: Model, state: State, stream=None):
    _check("trimmoe_state_reset",
           lib().trimmoe_state_reset(C.byref(model), C.byref(state), _stream_handle(stream)))


def trimmoe_layer_step(model: Model, layer: int, policy: Policy, state: State, trace,
                       workspace: torch.Tensor, stream=None):
    tr = C.byref(trace) if trace is not None else None
    _check("trimmoe_layer_step",
           lib().trimmoe_layer_step(C.byref(model), layer, C.byref(policy), C.byref(state), tr,
                                    _ptr(workspace), workspace.numel(), _stream_handle(stream)))


def trimmoe_stack_forward(model: Model, policy: Policy, state: State, trace,
                          workspace: torch.Tensor, stream=None):
    tr = C.byref(trace) if trace is not None else None
    _check("trimmoe_stack_forward",
           lib().trimmoe_stack_forward(C.byref(model), C.byref(policy), C.byref(state), tr,
                                       _ptr(workspace), workspace.numel(),
                                       _stream_handle(stream)))


def trimmoe_stack_forward_static(model: Model, policy: Policy, state: State, trace,
                                 stream=None):
    """trimmoe_stack_forward on the library's per-device scratch array: no
    workspace argument, nothing allocated."""
    tr = C.byref(trace) if trace is not None else None
    _check("trimmoe_stack_forward_static",
           lib().trimmoe_stack_forward_static(C.byref(model), C.byref(policy), C.byref(state),
                                              tr, _stream_handle(stream)))


def trimmoe_stack_forward_timed(model: Model, policy: Policy, state: State, trace,
                                workspace: torch.Tensor, events, stream=None):
    """``events``: list of N * (len(TIMED_CLASSES) + 1) torch.cuda.Event(enable_timing=True)
    already recorded once (so that their HIP events exist)."""
    arr = (C.c_void_p * len(events))(*[e.cuda_event for e in events])
    tr = C.byref(trace) if trace is not None else None
    _check("trimmoe_stack_forward_timed",
           lib().trimmoe_stack_forward_timed(C.byref(model), C.byref(policy), C.byref(state), tr,
                                             _ptr(workspace), workspace.numel(),
                                             _stream_handle(stream), arr, len(events)))


def trimmoe_set_clock_record(rec):
    """``rec``: an int64 device tensor of 2 * len(TIMED_CLASSES) zeros, or None
    to stop recording (the caller keeps the tensor alive while it is set)."""
    if rec is not None:
        assert rec.is_cuda and rec.dtype == torch.int64 and rec.is_contiguous()
        assert rec.numel() == 2 * len(TIMED_CLASSES)
    _check("trimmoe_set_clock_record", lib().trimmoe_set_clock_record(_ptr(rec)))


def clock_mhz(rec) -> dict:
    """Mean engine clock (MHz) per GEMM class from a filled record."""
    r = rec.cpu().tolist()
    return {c: 100.0 * r[2 * i] / r[2 * i + 1]
            for i, c in enumerate(TIMED_CLASSES) if r[2 * i + 1] > 0}


def trimmoe_window_stats(model: Model, policy: Policy, state: State, trace,
                         stats: torch.Tensor, stream=None):
    """Add one stack pass's observations to ``stats`` (float64 [6] on the GPU)."""
    assert stats.dtype == torch.float64 and stats.numel() == 6 and stats.is_contiguous()
    tr = C.byref(trace) if trace is not None else None
    _check("trimmoe_window_stats",
           lib().trimmoe_window_stats(C.byref(model), C.byref(policy), C.byref(state), tr,
                                      _ptr(stats), _stream_handle(stream)))


def trimmoe_feedback_update(policy: Policy, stats, eta: float, kappa: float, p_floor: float):
    """Update policy.p_exit and policy.omega_t in place from a window's stats
    (six numbers on the host)."""
    arr = (C.c_double * 6)(*[float(v) for v in stats])
    _check("trimmoe_feedback_update",
           lib().trimmoe_feedback_update(C.byref(policy), arr, eta, kappa, p_floor))


# ------------------------------------- offline statistics and placement ----
def _host(a, dtype):
    """A C-contiguous numpy copy (or view) of a host array in `dtype`."""
    if isinstance(a, torch.Tensor):
        a = a.detach().cpu().numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=dtype))


def _np_ptr(a: np.ndarray):
    return C.c_void_p(a.ctypes.data)


def trimmoe_calib_exit_layers(xi, p_exit: float) -> np.ndarray:
    """Exit layer of every calibration token from per-layer confidences [N, Q]."""
    xi = _host(xi, np.float32)
    N, Q = xi.shape
    out = np.zeros(Q, dtype=np.int32)
    _check("trimmoe_calib_exit_layers",
           lib().trimmoe_calib_exit_layers(N, Q, _np_ptr(xi), float(p_exit), _np_ptr(out)))
    return out


def trimmoe_calib_stats(target, importance, exit_layer, theta, n_experts: int):
    """(pi [N], act [N, E], sigma [N, E], lambda [N, E]) of a calibration record."""
    target = _host(target, np.int16)
    importance = _host(importance, np.float32)
    exit_layer = _host(exit_layer, np.int32)
    theta = _host(theta, np.float32)
    N, Q, k = target.shape
    E = int(n_experts)
    pi = np.zeros(N)
    act, sigma, lam = np.zeros((N, E)), np.zeros((N, E)), np.zeros((N, E))
    _check("trimmoe_calib_stats",
           lib().trimmoe_calib_stats(N, Q, E, k, _np_ptr(target), _np_ptr(importance),
                                     _np_ptr(exit_layer), _np_ptr(theta), _np_ptr(pi),
                                     _np_ptr(act), _np_ptr(sigma), _np_ptr(lam)))
    return pi, act, sigma, lam


def trimmoe_calib_transitions(target, exit_layer, n_experts: int, trans_b: int):
    """Transition rows (to int16 [N-1, E, B], p float32 [N-1, E, B])."""
    target = _host(target, np.int16)
    exit_layer = _host(exit_layer, np.int32)
    N, Q, k = target.shape
    E, B = int(n_experts), int(trans_b)
    to = np.zeros((max(N - 1, 0), E, B), dtype=np.int16)
    pr = np.zeros((max(N - 1, 0), E, B), dtype=np.float32)
    _check("trimmoe_calib_transitions",
           lib().trimmoe_calib_transitions(N, Q, E, k, _np_ptr(target), _np_ptr(exit_layer), B,
                                           _np_ptr(to), _np_ptr(pr)))
    return to, pr


def trimmoe_place_replicas(lam, rho, z, nbytes, capacity, bandwidth, latency, x0):
    """Greedy replication from a baseline x0 [M, N, E]; returns (x, n_placed)."""
    x = _host(x0, np.uint8).copy()
    M, N, E = x.shape
    args = [_host(v, np.float64) for v in (lam, rho, z, nbytes, capacity, bandwidth, latency)]
    n = C.c_int32(0)
    _check("trimmoe_place_replicas",
           lib().trimmoe_place_replicas(M, N, E, *[_np_ptr(v) for v in args], _np_ptr(x),
                                        C.byref(n)))
    return x, int(n.value)


# ------------------------------------------------- exit-head training ------
def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"hidden states must be bf16 or fp32, not {t.dtype}")


def _aligned_ws(nbytes: int, device) -> torch.Tensor:
    ws = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + nbytes]


def trimmoe_head_argmax(w_head: torch.Tensor, h: torch.Tensor, b_head=None,
                        stream=None) -> torch.Tensor:
    """argmax over the rows of an output head [V, d] for each row of h [Q, d]
    (both on one GPU, same dtype); returns int32 [Q] on the GPU."""
    assert w_head.dtype == h.dtype and w_head.is_contiguous() and h.is_contiguous()
    V, d = w_head.shape
    Q = h.shape[0]
    dt = _dtype_code(h)
    n = C.c_size_t(0)
    _check("trimmoe_head_argmax_workspace_size",
           lib().trimmoe_head_argmax_workspace_size(dt, V, Q, C.byref(n)))
    ws = _aligned_ws(n.value, h.device)
    out = torch.empty(Q, dtype=torch.int32, device=h.device)
    _check("trimmoe_head_argmax",
           lib().trimmoe_head_argmax(dt, V, d, Q, _ptr(w_head), _ptr(b_head), _ptr(h), _ptr(out),
                                     _ptr(ws), ws.numel(), _stream_handle(stream)))
    return out


def trimmoe_consistency_labels(pred: torch.Tensor, ref: torch.Tensor, stream=None):
    """Eq. (22) on the GPU: uint8 [Q], 1 where pred == ref (int32 [Q] each)."""
    assert pred.dtype == torch.int32 and ref.dtype == torch.int32 and pred.shape == ref.shape
    out = torch.empty(pred.shape[0], dtype=torch.uint8, device=pred.device)
    _check("trimmoe_consistency_labels",
           lib().trimmoe_consistency_labels(pred.shape[0], _ptr(pred), _ptr(ref), _ptr(out),
                                            _stream_handle(stream)))
    return out


def trimmoe_train_exit_head(h: torch.Tensor, labels: torch.Tensor, epochs: int, lr: float,
                            w: torch.Tensor, c: torch.Tensor, loss=None, stream=None):
    """Gradient descent of the sigmoid exit head on BCE; w (fp32 [d]) and c
    (fp32 [1]) are updated in place; loss (fp32 [epochs]) if given."""
    assert w.dtype == torch.float32 and c.dtype == torch.float32 and labels.dtype == torch.uint8
    Q, d = h.shape
    n = C.c_size_t(0)
    _check("trimmoe_train_exit_head_workspace_size",
           lib().trimmoe_train_exit_head_workspace_size(Q, C.byref(n)))
    ws = _aligned_ws(n.value, h.device)
    _check("trimmoe_train_exit_head",
           lib().trimmoe_train_exit_head(_dtype_code(h), d, Q, _ptr(h), _ptr(labels), int(epochs),
                                         float(lr), _ptr(w), _ptr(c), _ptr(loss), _ptr(ws),
                                         ws.numel(), _stream_handle(stream)))


# ------------------------------------------------ struct construction ------
class ModelHandle:
    """A Model struct over device tensors; keeps the tensors alive.

    ``layers`` is a list of dicts with the keys of trimmoe_layer (torch
    tensors on one GPU, or None) plus the floats ``theta`` and
    ``skip_slope``.
    """

    def __init__(self, *, n_layers, d_model, n_experts, top_k, d_ff, d_ff_shared, vocab_exit,
                 dtype, act, conf_mode, normalize_topk, layers):
        self._keep = []
        arr = (Layer * n_layers)()
        for i, L in enumerate(layers):
            for key in ("w_router", "b_router", "w_up", "w_gate", "w_down", "ws_up", "ws_gate",
                        "ws_down", "w_exit", "b_exit", "local_mask", "sim", "trans_to",
                        "trans_p"):
                t = L.get(key)
                if t is not None:
                    if not t.is_contiguous():
                        t = t.contiguous()
                    self._keep.append(t)
                setattr(arr[i], key, None if t is None else t.data_ptr())
            arr[i].theta = float(L["theta"])
            arr[i].skip_slope = float(L["skip_slope"])
        self.layers = arr
        trans_b = next((int(L["trans_to"].shape[1]) for L in layers
                        if L.get("trans_to") is not None), 0)
        self.model = Model(n_layers, d_model, n_experts, top_k, d_ff, d_ff_shared, vocab_exit,
                           dtype, act, conf_mode, normalize_topk,
                           C.cast(arr, C.POINTER(Layer)), trans_b)


def make_policy(*, p_exit, budget, omega_t, t_local, t_remote, phi_scale, sim_min,
                p_exit_tok=None, budget_tok=None, horizon=1, la_subs=4) -> Policy:
    return Policy(p_exit, budget, omega_t, t_local, t_remote, phi_scale, sim_min,
                  None if p_exit_tok is None else p_exit_tok.data_ptr(),
                  None if budget_tok is None else budget_tok.data_ptr(), int(horizon),
                  int(la_subs))


class StateBuffers:
    """Caller-owned per-token state on one GPU (h is used in place)."""

    def __init__(self, h: torch.Tensor):
        T = h.shape[0]
        dev = h.device
        self.h = h
        self.d_acc = torch.zeros(T, dtype=torch.float32, device=dev)
        self.active_idx = torch.zeros(max(T, 1), dtype=torch.int32, device=dev)
        self.n_active = torch.zeros(1, dtype=torch.int32, device=dev)
        self.exit_layer = torch.zeros(max(T, 1), dtype=torch.int32, device=dev)
        self.xi = torch.zeros(max(T, 1), dtype=torch.float32, device=dev)
        self.state = State(T, h.data_ptr(), self.d_acc.data_ptr(), self.active_idx.data_ptr(),
                           self.n_active.data_ptr(), self.exit_layer.data_ptr(),
                           self.xi.data_ptr())


class TraceBuffers:
    """Per-layer decision record on one GPU."""

    def __init__(self, n_layers: int, T: int, k: int, device):
        z = dict(device=device)
        self.action = torch.zeros(n_layers, T, dtype=torch.int8, **z)
        self.target = torch.zeros(n_layers, T, k, dtype=torch.int16, **z)
        self.exec = torch.zeros(n_layers, T, k, dtype=torch.int16, **z)
        self.kind = torch.zeros(n_layers, T, k, dtype=torch.int8, **z)
        self.gate = torch.zeros(n_layers, T, k, dtype=torch.float32, **z)
        self.importance = torch.zeros(n_layers, T, dtype=torch.float32, **z)
        self.xi = torch.zeros(n_layers, T, dtype=torch.float32, **z)
        self.d_acc = torch.zeros(n_layers, T, dtype=torch.float32, **z)
        self.counters = torch.zeros(n_layers, N_COUNTERS, dtype=torch.int32, **z)
        self.trace = Trace(*(getattr(self, n).data_ptr() for n in
                             ("action", "target", "exec", "kind", "gate", "importance", "xi",
                              "d_acc", "counters")))


class CounterTrace:
    """A trace that records only the per-layer counters (what the runtime
    feedback observations need)."""

    def __init__(self, n_layers: int, device):
        self.counters = torch.zeros(n_layers, N_COUNTERS, dtype=torch.int32, device=device)
        self.trace = Trace(None, None, None, None, None, None, None, None,
                           self.counters.data_ptr())


def alloc_workspace(model: Model, max_tokens: int, device) -> torch.Tensor:
    """A 256-byte aligned uint8 workspace of the size the library asks for."""
    n = trimmoe_workspace_size(model, max_tokens)
    ws = torch.empty(n + 256, dtype=torch.uint8, device=device)
    off = (-ws.data_ptr()) % 256
    return ws[off:off + n]


def model_handle(dims: dict, layers: list) -> ModelHandle:
    """ModelHandle from a dims dict (n_layers, d_model, n_experts, top_k, d_ff,
    d_ff_shared, vocab_exit, dtype 'bf16'|'f32', act 'relu'|'swiglu',
    normalize_topk, optional conf_mode 'softmax'|'sigmoid') and per-layer
    tensor dicts keyed like trimmoe_layer."""
    return ModelHandle(
        n_layers=dims["n_layers"], d_model=dims["d_model"], n_experts=dims["n_experts"],
        top_k=dims["top_k"], d_ff=dims["d_ff"], d_ff_shared=dims["d_ff_shared"],
        vocab_exit=dims["vocab_exit"], dtype={"f32": F32, "bf16": BF16}[dims["dtype"]],
        act={"relu": ACT_RELU, "swiglu": ACT_SWIGLU}[dims["act"]],
        conf_mode={"softmax": CONF_SOFTMAX, "sigmoid": CONF_SIGMOID}[dims.get("conf_mode", "softmax")],
        normalize_topk=int(dims["normalize_topk"]), layers=layers)
