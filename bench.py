#!/usr/bin/env python3
"""Throughput of the adaptive-depth MoE stack on one MI355X.

A step is one trimmoe_stack_forward over one batch of synthetic tokens (all
layers: route/decide, bucketing, grouped expert FFN, combine, exit head,
exit gate, compaction), inputs already resident in HBM.  For the decode
workload each step takes a fresh batch (32 tokens, its own seed).  Prints
one JSON line:

* value: tokens/s = tokens per batch / median step time.  Every timed step
  is bracketed by its own HIP events on the library's stream; a 512 MiB
  buffer is written between steps, outside those events, so that no step
  finds the previous one's operands in the 256 MB Infinity Cache.  The
  line also gives the p10-p90 spread of the step times, their mean, the
  device's CU count and peak engine clock;
* roofline: the dominant kernel class (by measured time) against its own
  roofline (MFMA or HBM, whichever its algorithmic FLOPs and bytes make
  binding), from HIP events recorded around each kernel class on the
  library's stream (trimmoe_stack_forward_timed) over a second timed pass;
  traffic from the committed rocprofv3 counter summaries when they match;
* cpu_baseline: the CPU oracle (single BLAS thread) on a bounded sample of
  the same tokens (and, for stacks too large to hold in fp64, of the first
  layers), scaled to tokens/s (tokens are independent in this step);
* grouped_gemm_mfma_frac / grouped_gemm_hbm_frac: algorithmic FLOPs and
  weight bytes of the grouped up/gate and down GEMMs over their measured
  time, against the bf16 dense MFMA peak and the HBM bandwidth;
* class_hbm_frac: algorithmic bytes over measured time for every class;
* feedback (decode workload, or --feedback-window > 0): the same batches
  once more, with the runtime feedback rules closing the loop after every
  window of passes (observations on the GPU, Eq. (37) and Eq. (43) on the
  host): the throughput of that loop and the trajectory of p_J and omega_T;
  and the cost of the observations themselves (the same loop with zero step
  sizes, so that the policy and the work stay those of the plain loop).
  Not part of `value`.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "active tokens/s through adaptive-depth MoE stack; grouped-GEMM % MFMA peak"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
PEAK_CLOCK_MHZ = 2400.0     # engine clock the published MFMA peaks assume


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default 20; the decode workload: its step count, 128)")
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mixtral_8x7b_prefill",
                    help="workload (default: the Mixtral-8x7B-shaped prefill batch, the "
                         "largest that fits one GPU)")
    ap.add_argument("--flush-mib", type=int, default=512,
                    help="MiB written between timed steps to evict the Infinity Cache "
                         "(0 = off)")
    ap.add_argument("--horizon", type=int, default=None,
                    help="look-ahead horizon H of the decision (default: the workload's, 1)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--feedback-window", type=int, default=None,
                    help="passes per runtime-feedback window (default: 16 for the decode "
                         "workload, else off; 0 = off)")
    ap.add_argument("--eta", type=float, default=0.2, help="step size of the p_J update")
    ap.add_argument("--kappa", type=float, default=0.2,
                    help="step size of the delay/quality weight update")
    ap.add_argument("--p-floor", type=float, default=0.1, help="lower bound of p_J")
    ap.add_argument("--offline", action="store_true",
                    help="also time the offline stage (calibration pass on the GPU, "
                         "statistics, transition rows, placement over 10 servers)")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain device copy of known size (to scale HBM byte "
                         "counters) and exit")
    return ap.parse_args()


def calibrate_copy():
    """A plain copy of 512 MiB, five times: the known bytes per dispatch that
    FETCH_SIZE / WRITE_SIZE of the same run are divided by."""
    import torch
    n = 512 << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes_read": n, "calibrate_copy_bytes_written": n,
                      "dispatches": 5}), flush=True)


def device_info():
    """CU count and peak engine clock of device 0 (hipDeviceGetAttribute)."""
    import ctypes as C
    hip = C.CDLL("libamdhip64.so")
    out = {}
    for key, attr in (("compute_units", 63), ("peak_engine_clock_mhz", 5)):
        v = C.c_int(0)
        rc = hip.hipDeviceGetAttribute(C.byref(v), attr, 0)
        out[key] = v.value if rc == 0 else None
    if out["peak_engine_clock_mhz"]:
        out["peak_engine_clock_mhz"] //= 1000   # the attribute is in kHz
    return out


def host_cpu():
    """Model name and logical CPU counts of the host."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"model": model, "nproc": os.cpu_count(),
            "usable": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None}


def class_kernel(cls, cfg):
    """The library kernel(s) of a kernel class at the workload's batch size,
    by the library's tile selection: grouped GEMMs with at least 1024 rows
    per expert on average and the shared expert from 2048 tokens run the
    256 x 256 large-group core, the exit head of models with d >= 2048 from
    1024 tokens too; everything else the 8-wavefront streaming core."""
    T, k, E, d = cfg["n_tokens"], cfg["top_k"], cfg["n_experts"], cfg["d_model"]
    bf16 = cfg["dtype"] == "bf16"
    swiglu = cfg["act"] == "swiglu"
    big = bf16 and T * k >= 1024 * E
    if cls == "up":
        name = ("k_ffn_big<0>" if swiglu else "k_ffn_big<1>") if big else \
            ("k_ffn_mma<128x128 dual, up>" if swiglu else "k_ffn_mma<128x256, up>")
        return name + " (grouped up/gate + activation)"
    if cls == "down":
        return ("k_ffn_big<2>" if big else "k_ffn_mma<128x256, down>") + " (grouped down)"
    if cls == "exit":
        return ("k_exit_big" if bf16 and T >= 1024 and d >= 2048 else "k_exit_mma") + \
            " (exit head + softmax partials)"
    return {"route": "k_route (route, substitution, skip)",
            "bucket": "k_scan + k_bucket (bucketing)",
            "shared": "k_ffn_mma / k_ffn_big (shared expert)",
            "combine": "k_combine (weighted combine)",
            "gate": "k_exit_reduce + k_compact (exit gate)"}[cls]


def log(msg):
    """Progress on stderr (the JSON line is the only stdout)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def step_stats(ms):
    """Median, p10, p90 and mean of per-step times (ms)."""
    import numpy as np
    a = np.asarray(ms, dtype=np.float64)
    return dict(median=float(np.median(a)), p10=float(np.percentile(a, 10)),
                p90=float(np.percentile(a, 90)), mean=float(a.mean()), min=float(a.min()),
                max=float(a.max()))


def algorithmic_work(cfg, counters):
    """Per-layer algorithmic FLOPs and bytes, per kernel class, from the
    traced counters.

    counters[l] = (active, executed, skipped, exited, substituted slots,
    remote slots, merged rows, distinct experts).  Only the work the method
    must do: router over active tokens; expert FFN over merged rows; shared
    expert and exit head over executed tokens (exit head not at the last
    layer); every weight matrix touched read once; h read per active token
    and written per executed token; index lists of the bucketing.
    Intermediates (activations, split-K partials, softmax partials) are
    implementation bytes and not counted.
    """
    N, d, E, F, Fs, V = (cfg[k] for k in ("n_layers", "d_model", "n_experts", "d_ff",
                                          "d_ff_shared", "vocab_exit"))
    b = 2 if cfg["dtype"] == "bf16" else 4
    m = 3 if cfg["act"] == "swiglu" else 2
    out = []
    for l in range(N):
        n_a, n_x, rows, distinct = (int(counters[l][i]) for i in (0, 1, 6, 7))
        last = l == N - 1
        flop = dict(route=2 * n_a * d * E, bucket=0,
                    up=2 * rows * d * F * (m - 1), down=2 * rows * d * F,
                    shared=6 * n_x * d * Fs, combine=0,
                    exit=0 if last else 2 * n_x * d * V, gate=0)
        byt = dict(route=(E * d * b if n_a else 0) + n_a * d * b,
                   bucket=8 * (rows + n_a),
                   up=distinct * (m - 1) * d * F * b + rows * d * b,
                   down=distinct * d * F * b,
                   shared=(3 * d * Fs * b + n_x * d * b) if (n_x and Fs) else 0,
                   combine=2 * n_x * d * b,
                   exit=0 if (last or not n_x) else V * d * b + n_x * d * b,
                   gate=0 if last else 8 * n_a)
        out.append(dict(layer=l, n_active=n_a, n_exec=n_x, rows=rows, distinct=distinct,
                        flop=flop, bytes=byt))
    return out


def counter_traffic(cls, workload):
    """Calibrated HBM-side bytes per launch of the kernel class ``cls`` on
    ``workload`` from the committed rocprofv3 counter summaries (FETCH_SIZE and
    WRITE_SIZE passes scaled by a plain copy): (bytes, summary path, kernel
    name), or (None, None, None) when no summary covers it or the kernel's
    source file has changed since the counters were taken."""
    import glob
    import hashlib
    keys = ("class", "kernel", "workload", "traffic_bytes_per_launch", "source", "source_sha256")
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        for block in open(path).read().split("```"):
            fields = {}
            for line in block.splitlines():
                k, sep, v = line.strip().partition(": ")
                if sep and k in keys:
                    fields[k] = v.strip()
            if fields.get("class") != cls or fields.get("workload") != workload:
                continue
            src = os.path.join(ROOT, fields.get("source", ""))
            if not os.path.isfile(src) or \
                    hashlib.sha256(open(src, "rb").read()).hexdigest() != fields.get("source_sha256"):
                return None, None, None
            return (float(fields["traffic_bytes_per_launch"]), os.path.relpath(path, ROOT),
                    fields.get("kernel"))
    return None, None, None


def _f64_layer_bytes(cfg):
    m = 3 if cfg["act"] == "swiglu" else 2
    d, E = cfg["d_model"], cfg["n_experts"]
    return 8 * (E * m * d * cfg["d_ff"] + 3 * d * cfg["d_ff_shared"] +
                cfg["vocab_exit"] * d + E * d + E * E)


def cpu_baseline(inp, target_s, max_f64_bytes=24e9):
    """The oracle as it stands, one BLAS thread, on the first S tokens.

    The oracle works on fp64 copies of the weights.  When the whole stack
    would not fit in ``max_f64_bytes`` it runs the first layers only and the
    time is scaled to all layers (early layers have the most active tokens,
    so this errs towards a slower oracle).  Weight conversion is outside the
    timed part; only the oracle's layer steps are timed."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle as O

    cfg = inp["cfg"]
    N = cfg["n_layers"]
    n_l = min(N, max(1, int(max_f64_bytes // _f64_layer_bytes(cfg))))
    H = int(inp["policy"].get("horizon", 1))
    models = {l: O.model_from_inputs(inp, layers=[l],
                                     decision_layers=range(l + 1, min(l + H, N)))
              for l in range(n_l)}
    pol = {k: float(np.float32(v)) for k, v in inp["policy"].items()}
    h0 = inp["h0"].double().cpu().numpy()
    T = h0.shape[0]
    with threadpool_limits(limits=1):
        # size the sample from a small probe, then refine
        S = min(T, 64 if n_l == N else 8)
        for _ in range(3):
            state = O.init_state(h0[:S], N)
            dt = 0.0
            for l in range(n_l):
                t0 = time.perf_counter()
                O.layer_step(models[l], l, pol, state)
                dt += time.perf_counter() - t0
            if dt >= 0.6 * target_s or S == T:
                break
            S = min(T, max(S + 1, int(S * target_s / max(dt, 1e-3))))
    scale = N / n_l
    layers = f"all {N} layers" if n_l == N else \
        f"layers 0-{n_l - 1} of {N} (fp64 weights of the whole stack exceed " \
        f"{max_f64_bytes / 1e9:.0f} GB; time scaled by {scale:g})"
    extrap = S < T or n_l < N
    cpu = host_cpu()
    return dict(value=S / (dt * scale), unit="tokens/s", cores=1, kind="oracle",
                extrapolated=extrap, host_cpu=cpu["model"], host_nproc=cpu["nproc"],
                host_cpus_usable=cpu["usable"],
                sample=f"first {S} of {T} tokens of the {cfg['name']} batch through "
                       f"{layers}, fp64 numpy oracle, 1 BLAS thread (1 core of "
                       f"{cpu['nproc']}: {cpu['model']}), {dt:.1f} s timed; "
                       + ("extrapolated linearly to the batch and depth (tokens are "
                          "independent in this step)" if extrap else "the whole workload"))


def feedback_loop(abi, cfg, mh, pol0, batches, K, window, ws, eta, kappa, p_floor,
                  observe=True):
    """K passes over the batches with the runtime feedback rules applied after
    every `window` passes; the window's observations accumulate on the GPU and
    one host copy of six numbers per window feeds the host update.  Returns
    (ms, per-window trajectory).  observe=False: the same K passes back to
    back with no observation and no update (the plain loop)."""
    import torch
    dev = batches[0].device
    policy = abi.make_policy(**pol0)
    ct = abi.CounterTrace(cfg["n_layers"], dev)
    stats = torch.zeros(6, dtype=torch.float64, device=dev)
    host = torch.zeros(6, dtype=torch.float64).pin_memory()
    nb = len(batches)
    states = [abi.StateBuffers(batches[i % nb].clone()) for i in range(K)]
    traj = []
    stream = torch.cuda.current_stream()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(K):
        if not observe:
            abi.trimmoe_stack_forward(mh.model, policy, states[i].state, None, ws)
            continue
        abi.trimmoe_stack_forward(mh.model, policy, states[i].state, ct.trace, ws)
        abi.trimmoe_window_stats(mh.model, policy, states[i].state, ct.trace, stats)
        if (i + 1) % window == 0 or i == K - 1:
            host.copy_(stats, non_blocking=True)
            stats.zero_()
            stream.synchronize()
            s = host.tolist()
            abi.trimmoe_feedback_update(policy, s, eta, kappa, p_floor)
            traj.append(dict(after_pass=i + 1, p_exit=policy.p_exit, omega_t=policy.omega_t,
                             exit_frac=s[1] / s[0] if s[0] else 0.0,
                             util=s[3] / s[0] if s[0] else 0.0,
                             delay_norm=s[4] / s[5] if s[5] else 0.0))
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1), traj


def offline_stage(abi, cfg, mh, inp, h0, ws):
    """Table I on this workload: the calibration pass over the batch, the
    Sec. IV-C statistics and Eq. (38) rows (4 entries), and the Eq. (28)
    greedy replication over 10 synthetic servers with memory ratio 2, each
    timed."""
    import torch

    from paper_2608_00573_amd import offline
    from synthgen.servers import make_servers

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    rec = offline.calibration_pass(mh.model, inp["policy"], h0, ws)
    t1 = time.perf_counter()
    theta = [L["theta"] for L in inp["layers"]]
    tab = offline.offline_tables(rec, inp["policy"]["p_exit"], theta, cfg["n_experts"],
                                 min(4, cfg["n_experts"]))
    t2 = time.perf_counter()
    srv = make_servers(cfg, n_servers=10, memory_ratio=2.0)
    x, added = offline.place(tab, srv)
    t3 = time.perf_counter()
    return {"calibration_tokens": int(h0.shape[0]), "servers": 10, "memory_ratio": 2.0,
            "calibration_pass_s": t1 - t0, "statistics_and_transitions_s": t2 - t1,
            "placement_s": t3 - t2, "replicas_added": added,
            "pi": [round(float(v), 4) for v in tab["pi"]],
            "home_experts_per_layer": x[srv["home"]].sum(axis=1).tolist()}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no sharding or collectives "
              "(tokens are independent; shard them across processes yourself); "
              "run it with --gpus 1", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy()
        return

    import numpy as np
    import torch

    from paper_2608_00573_amd import abi
    from synthgen import make_inputs, workload
    from synthgen.inputs import make_tokens

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    cfg = workload(args.workload)
    if args.horizon is not None:
        cfg["horizon"] = args.horizon
    decode = "decode_steps" in cfg
    K = args.steps if args.steps is not None else (cfg["decode_steps"] if decode else 20)
    W = args.warmup
    t_gen = time.perf_counter()
    log(f"{cfg['name']}: generating inputs on the GPU")
    inp = make_inputs(cfg, device=dev)
    T, N = cfg["n_tokens"], cfg["n_layers"]
    # one token batch per step for decode (fresh tokens, seeds base + s), else
    # the one batch every step
    if decode:
        batches = [make_tokens(cfg, cfg["token_seed_base"] + s, dev) for s in range(K)]
    else:
        batches = [inp["h0"].to(dev)]
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t_gen
    log(f"inputs ready in {t_gen:.1f} s; {W} warmup + {K} timed steps")
    mh = abi.model_handle(cfg, inp["layers"])
    policy = abi.make_policy(**inp["policy"])
    ws = abi.alloc_workspace(mh.model, T, dev)
    nb = len(batches)
    states = [abi.StateBuffers(batches[i % nb].clone()) for i in range(K + W)]
    stream = torch.cuda.current_stream()

    # a buffer written between steps (outside the step events) so that no
    # step starts with the previous step's operands in the Infinity Cache
    flush = torch.empty(args.flush_mib << 20, dtype=torch.uint8, device=dev) \
        if args.flush_mib > 0 else None

    def evict(i):
        if flush is not None:
            flush.fill_(i & 0xff)

    # warmup, then the timed region (inputs resident, no host sync inside)
    for i in range(W):
        evict(i)
        abi.trimmoe_stack_forward(mh.model, policy, states[K + i].state, None, ws)
    torch.cuda.synchronize()
    ev0 = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
    ev1 = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
    t0 = time.perf_counter()
    for i in range(K):
        evict(i)
        ev0[i].record(stream)
        abi.trimmoe_stack_forward(mh.model, policy, states[i].state, None, ws)
        ev1[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = [a.elapsed_time(b) for a, b in zip(ev0, ev1)]
    sst = step_stats(step_ms)
    ms_step = sst["median"]
    ms_total = float(sum(step_ms))
    del states

    log(f"timed: median {ms_step:.3f} ms per step; kernel-class pass")
    # per-kernel-class timing: HIP events on the same stream, same work, the
    # same eviction between steps
    classes = list(abi.TIMED_CLASSES)
    per = len(classes) + 1
    events = [torch.cuda.Event(enable_timing=True) for _ in range(N * per)]
    for e in events:
        e.record(stream)
    class_ms = np.zeros((N, per - 1))
    for i in range(K):
        st = abi.StateBuffers(batches[i % nb].clone())
        evict(i)
        abi.trimmoe_stack_forward_timed(mh.model, policy, st.state, None, ws, events)
        torch.cuda.synchronize()
        for l in range(N):
            for c in range(per - 1):
                class_ms[l, c] += events[l * per + c].elapsed_time(events[l * per + c + 1])
    class_ms /= K

    log("traced pass for the algorithmic work")
    # traced passes (one per distinct batch) for the algorithmic work
    work_steps = []
    for bt in batches:
        st = abi.StateBuffers(bt.clone())
        tr = abi.TraceBuffers(N, T, cfg["top_k"], dev)
        abi.trimmoe_stack_forward(mh.model, policy, st.state, tr.trace, ws)
        torch.cuda.synchronize()
        work_steps.append(algorithmic_work(cfg, tr.counters.cpu().numpy()))
    # mean engine clock of each GEMM class: one more pass of the same work
    # with the library's clock record set (bf16 GEMM kernels only)
    clock = {}
    if cfg["dtype"] == "bf16":
        log("engine-clock pass")
        rec = torch.zeros(2 * len(classes), dtype=torch.int64, device=dev)
        st = abi.StateBuffers(batches[0].clone())
        evict(0)
        abi.trimmoe_set_clock_record(rec)
        try:
            abi.trimmoe_stack_forward(mh.model, policy, st.state, None, ws)
            torch.cuda.synchronize()
        finally:
            abi.trimmoe_set_clock_record(None)
        clock = abi.clock_mhz(rec)
    # per-step averages, per class and per layer
    flop = {c: sum(w["flop"][c] for ws_ in work_steps for w in ws_) / nb for c in classes}
    byts = {c: sum(w["bytes"][c] for ws_ in work_steps for w in ws_) / nb for c in classes}

    peak = PEAK_BF16_TFLOPS if cfg["dtype"] == "bf16" else PEAK_FP32_TFLOPS
    dev_info = device_info()
    t_class = class_ms.sum(axis=0)  # ms per step per class
    ci = {n: i for i, n in enumerate(classes)}
    launches = {c: N for c in classes}
    launches["exit"] = N - 1
    launches["gate"] = N - 1
    if not cfg["d_ff_shared"]:
        launches["shared"] = 0
    dom = max((c for c in classes if launches[c]), key=lambda c: t_class[ci[c]])
    dom_s = t_class[ci[dom]] * 1e-3
    mfma_bound = flop[dom] / (peak * 1e12) >= byts[dom] / (PEAK_HBM_GBS * 1e9)
    traffic, traffic_src, traffic_kernel = counter_traffic(dom, cfg["name"])
    if mfma_bound:
        achieved, pk, unit = flop[dom] / dom_s / 1e12, peak, "TFLOP/s"
    else:
        achieved, pk, unit = byts[dom] / dom_s / 1e9, PEAK_HBM_GBS, "GB/s"
    gg_s = (t_class[ci["up"]] + t_class[ci["down"]]) * 1e-3
    gg_frac = (flop["up"] + flop["down"]) / gg_s / 1e12 / peak if gg_s else 0.0
    gg_hbm = (byts["up"] + byts["down"]) / gg_s / 1e9 / PEAK_HBM_GBS if gg_s else 0.0
    stack_bound_s = sum(max(sum(w["flop"].values()) / (peak * 1e12),
                            sum(w["bytes"].values()) / (PEAK_HBM_GBS * 1e9))
                        for ws_ in work_steps for w in ws_) / nb
    active_layers = sum(w["n_active"] for ws_ in work_steps for w in ws_) / nb
    step_bytes = sum(byts.values())

    out = {
        "metric": METRIC,
        "value": T / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg["dtype"],
        "data": "synthetic (seeded generator: planted twin experts, planted exit confidence)",
        "config": {"workload": cfg["name"], "n_layers": N, "d_model": cfg["d_model"],
                   "experts": cfg["n_experts"], "top_k": cfg["top_k"], "d_ff": cfg["d_ff"],
                   "d_ff_shared": cfg["d_ff_shared"], "vocab_exit": cfg["vocab_exit"],
                   "tokens_per_step": T, "fresh_batch_per_step": decode,
                   "horizon": cfg["horizon"], "transition_row_entries": cfg["trans_support"],
                   "parallelism": "single-gpu"},
        "roofline": {
            "kernel": class_kernel(dom, cfg),
            "class": dom,
            "bound": "mfma" if mfma_bound else "hbm",
            "achieved": achieved,
            "peak": pk,
            "unit": unit,
            "frac": achieved / pk,
            "traffic": traffic,
            "traffic_unit": "bytes per launch",
            "traffic_source": traffic_src,
            "traffic_kernel": traffic_kernel,
            "avg_launch_ms": t_class[ci[dom]] / launches[dom],
            "algorithmic_flop_per_launch": flop[dom] / launches[dom],
            "algorithmic_bytes_per_launch": byts[dom] / launches[dom],
            # the same rate against the peak scaled to the engine clock the
            # kernel ran at (the published peak assumes the peak clock)
            "clock_mhz": clock.get(dom),
            "frac_at_clock": (achieved / (pk * clock[dom] / PEAK_CLOCK_MHZ)
                              if mfma_bound and dom in clock else None),
        },
        "grouped_gemm_mfma_frac": gg_frac,
        # against the peak at the engine clock the up and down GEMMs ran at
        # (time-weighted)
        "grouped_gemm_mfma_frac_at_clock": (
            gg_frac * PEAK_CLOCK_MHZ * gg_s * 1e3
            / (t_class[ci["up"]] * clock["up"] + t_class[ci["down"]] * clock["down"])
            if gg_s and "up" in clock and "down" in clock else None),
        "grouped_gemm_hbm_frac": gg_hbm,
        "class_hbm_frac": {c: (byts[c] / (t_class[ci[c]] * 1e-3) / 1e9 / PEAK_HBM_GBS
                               if t_class[ci[c]] > 0 else 0.0) for c in classes},
        "step_algorithmic_gb_per_s": step_bytes / (ms_step * 1e-3) / 1e9,
        "active_token_layers_per_s": active_layers / (ms_step * 1e-3),
        "stack_roofline_frac": stack_bound_s / (ms_step * 1e-3),
        "step_ms": {k: round(v, 4) for k, v in sst.items()},
        "tokens_per_s_p10_p90": [T / (sst["p90"] * 1e-3), T / (sst["p10"] * 1e-3)],
        "tokens_per_s_mean": T * K / (ms_total * 1e-3),
        "timing": f"median of {K} steps, each between its own HIP events; "
                  + (f"{args.flush_mib} MiB written between steps (outside the events)"
                     if flush is not None else "no cache eviction between steps"),
        "device": dev_info,
        "sustained_clock_mhz": clock,
        "kernel_ms_per_step": {n: float(t_class[i]) for i, n in enumerate(classes)},
        "per_layer": [{k: w[k] for k in ("n_active", "n_exec", "rows", "distinct")}
                      for w in work_steps[0]],
        "wall_s_timed_region": wall,
        "input_generation_s": t_gen,
    }
    fw = args.feedback_window if args.feedback_window is not None else (16 if decode else 0)
    if fw > 0:
        ms_plain, _ = feedback_loop(abi, cfg, mh, inp["policy"], batches, K, fw, ws, 0.0, 0.0,
                                    args.p_floor, observe=False)
        ms_obs, _ = feedback_loop(abi, cfg, mh, inp["policy"], batches, K, fw, ws, 0.0, 0.0,
                                  args.p_floor)
        ms_fb, traj = feedback_loop(abi, cfg, mh, inp["policy"], batches, K, fw, ws, args.eta,
                                    args.kappa, args.p_floor)
        out["feedback"] = {
            "window": fw, "eta": args.eta, "kappa": args.kappa, "p_floor": args.p_floor,
            "tokens_per_s": T * K / (ms_fb * 1e-3), "ms_per_step": ms_fb / K,
            "plain_loop_tokens_per_s": T * K / (ms_plain * 1e-3),
            "observation_cost_frac": ms_obs / ms_plain - 1.0,
            "p_exit_start": inp["policy"]["p_exit"], "omega_t_start": inp["policy"]["omega_t"],
            "windows": traj}
    if args.offline:
        out["offline"] = offline_stage(abi, cfg, mh, inp, batches[0], ws)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle on a sample)")
        inp["h0"] = batches[0]
        out["cpu_baseline"] = cpu_baseline(inp, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
