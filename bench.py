#!/usr/bin/env python3
"""Throughput of the adaptive-depth MoE stack on one MI355X.

A step is one trimmoe_stack_forward over one batch of synthetic tokens (all
layers: route/decide, bucketing, grouped expert FFN, combine, exit head,
exit gate, compaction), inputs already resident in HBM.  Prints one JSON
line:

* value: tokens/s = tokens per batch * steps / timed seconds;
* roofline: the dominant kernel class (by measured time) against its
  roofline, from HIP events recorded around each kernel class on the
  library's stream (trimmoe_stack_forward_timed) over a second timed pass;
* cpu_baseline: the CPU oracle (single BLAS thread) on a bounded sample of
  the same tokens, scaled to tokens/s (tokens are independent in this step);
* grouped_gemm_mfma_frac: algorithmic FLOPs of the grouped up/gate and down
  GEMMs over their measured time, against the bf16 dense MFMA peak.
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


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="switch_base_8e")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
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


def algorithmic_work(cfg, counters):
    """Per-layer algorithmic FLOPs and bytes from the traced counters.

    counters[l] = (active, executed, skipped, exited, substituted slots,
    remote slots, merged rows, distinct experts).  Only the work the method
    must do: router over active tokens; expert FFN over merged rows; shared
    expert and exit head over executed tokens (exit head not at the last
    layer); weight bytes of each matrix touched once; h read per active and
    written per executed token.
    """
    N, d, E, F, Fs, V = (cfg[k] for k in ("n_layers", "d_model", "n_experts", "d_ff",
                                          "d_ff_shared", "vocab_exit"))
    b = 2 if cfg["dtype"] == "bf16" else 4
    m = 3 if cfg["act"] == "swiglu" else 2
    out = []
    for l in range(N):
        n_a, n_x, rows, distinct = (int(counters[l][i]) for i in (0, 1, 6, 7))
        last = l == N - 1
        f_route = 2 * n_a * d * E
        f_up = 2 * rows * d * F * (m - 1)
        f_down = 2 * rows * d * F
        f_shared = 6 * n_x * d * Fs
        f_exit = 0 if last else 2 * n_x * d * V
        by_route = (E * d * b if n_a else 0) + n_a * d * b
        by_experts = distinct * m * d * F * b
        by_shared = 3 * d * Fs * b if (n_x and Fs) else 0
        by_exit = 0 if (last or not n_x) else V * d * b
        by_out = n_x * d * b
        out.append(dict(layer=l, n_active=n_a, n_exec=n_x, rows=rows, distinct=distinct,
                        flop_route=f_route, flop_up=f_up, flop_down=f_down,
                        flop_shared=f_shared, flop_exit=f_exit,
                        bytes=by_route + by_experts + by_shared + by_exit + by_out,
                        bytes_exit=by_exit + (0 if last else n_x * d * b)))
    return out


def counter_traffic(kernel, workload):
    """Calibrated HBM-side bytes per launch of ``kernel`` on ``workload`` from
    the committed rocprofv3 counter summaries (FETCH_SIZE and WRITE_SIZE
    passes scaled by a plain copy), or (None, None) when no summary covers it
    or the kernel's source file has changed since the counters were taken."""
    import glob
    import hashlib
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        fields = {}
        for line in open(path):
            k, sep, v = line.strip().partition(": ")
            if sep and k in ("kernel", "workload", "traffic_bytes_per_launch", "source",
                             "source_sha256"):
                fields[k] = v.strip()
        if fields.get("kernel") != kernel or fields.get("workload") != workload:
            continue
        src = os.path.join(ROOT, fields.get("source", ""))
        if not os.path.isfile(src):
            return None, None
        if hashlib.sha256(open(src, "rb").read()).hexdigest() != fields.get("source_sha256"):
            return None, None
        return float(fields["traffic_bytes_per_launch"]), os.path.relpath(path, ROOT)
    return None, None


def cpu_baseline(inp, target_s):
    """The oracle as it stands, one BLAS thread, on the first S tokens."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle as O

    cfg = inp["cfg"]
    model = O.model_from_inputs(inp)
    pol = {k: float(np.float32(v)) for k, v in inp["policy"].items()}
    h0 = inp["h0"].double().cpu().numpy()
    T = h0.shape[0]
    with threadpool_limits(limits=1):
        # size the sample from a small probe, then refine once
        S = min(T, 64)
        for _ in range(3):
            t0 = time.perf_counter()
            O.stack_forward(model, pol, h0[:S])
            dt = time.perf_counter() - t0
            if dt >= 0.6 * target_s or S == T:
                break
            S = min(T, max(S + 1, int(S * target_s / max(dt, 1e-3))))
    return dict(value=S / dt, unit="tokens/s", cores=1, kind="oracle",
                sample=f"first {S} of {T} tokens of the {cfg['name']} batch through all "
                       f"{cfg['n_layers']} layers, fp64 numpy oracle, 1 BLAS thread, "
                       f"{dt:.1f} s; tokens are independent so tokens/s scales to the batch")


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

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    cfg = workload(args.workload)
    t_gen = time.perf_counter()
    inp = make_inputs(cfg, device=dev)
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t_gen
    T, N = cfg["n_tokens"], cfg["n_layers"]
    mh = abi.model_handle(cfg, inp["layers"])
    policy = abi.make_policy(**inp["policy"])
    ws = abi.alloc_workspace(mh.model, T, dev)
    h0 = inp["h0"].to(dev)
    K, W = args.steps, args.warmup
    states = [abi.StateBuffers(h0.clone()) for _ in range(K + W)]
    stream = torch.cuda.current_stream()

    # warmup, then the timed region (inputs resident, no host sync inside)
    for i in range(W):
        abi.trimmoe_stack_forward(mh.model, policy, states[i].state, None, ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record(stream)
    for i in range(W, W + K):
        abi.trimmoe_stack_forward(mh.model, policy, states[i].state, None, ws)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_total = e0.elapsed_time(e1)
    ms_step = ms_total / K

    # per-kernel-class timing: HIP events on the same stream, same work
    per = len(abi.TIMED_CLASSES) + 1
    events = [torch.cuda.Event(enable_timing=True) for _ in range(N * per)]
    for e in events:
        e.record(stream)
    class_ms = np.zeros((N, per - 1))
    for i in range(K):
        st = abi.StateBuffers(h0.clone())
        abi.trimmoe_stack_forward_timed(mh.model, policy, st.state, None, ws, events)
        torch.cuda.synchronize()
        for l in range(N):
            for c in range(per - 1):
                class_ms[l, c] += events[l * per + c].elapsed_time(events[l * per + c + 1])
    class_ms /= K

    # one traced step for the per-layer counts of the algorithmic work
    st = abi.StateBuffers(h0.clone())
    tr = abi.TraceBuffers(N, T, cfg["top_k"], dev)
    abi.trimmoe_stack_forward(mh.model, policy, st.state, tr.trace, ws)
    torch.cuda.synchronize()
    counters = tr.counters.cpu().numpy()
    work = algorithmic_work(cfg, counters)

    peak = PEAK_BF16_TFLOPS if cfg["dtype"] == "bf16" else PEAK_FP32_TFLOPS
    ci = {n: i for i, n in enumerate(abi.TIMED_CLASSES)}
    t_class = class_ms.sum(axis=0)  # ms per step per class
    flops = {"up": sum(w["flop_up"] for w in work), "down": sum(w["flop_down"] for w in work),
             "exit": sum(w["flop_exit"] for w in work),
             "shared": sum(w["flop_shared"] for w in work)}
    launches = {"up": N, "down": N, "exit": N - 1, "shared": N if cfg["d_ff_shared"] else 0}
    dom = max(("up", "down", "exit", "shared"), key=lambda c: t_class[ci[c]])
    dom_ms = t_class[ci[dom]]
    dom_tflops = flops[dom] / (dom_ms * 1e-3) / 1e12 if dom_ms > 0 else 0.0
    gg_ms = t_class[ci["up"]] + t_class[ci["down"]]
    gg_frac = (flops["up"] + flops["down"]) / (gg_ms * 1e-3) / 1e12 / peak if gg_ms else 0.0
    stack_bound_ms = sum(max((w["flop_route"] + w["flop_up"] + w["flop_down"] +
                              w["flop_shared"] + w["flop_exit"]) / (peak * 1e12),
                             w["bytes"] / (PEAK_HBM_GBS * 1e9)) for w in work) * 1e3
    active_layers = sum(w["n_active"] for w in work)
    dom_kernel = {"up": "k_ffn_mma", "down": "k_ffn_mma", "exit": "k_exit_mma",
                  "shared": "k_ffn_mma"}[dom]
    traffic, traffic_src = counter_traffic(dom_kernel, cfg["name"])

    out = {
        "metric": METRIC,
        "value": T * K / (ms_total * 1e-3),
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
                   "tokens_per_step": T, "parallelism": "single-gpu"},
        "roofline": {
            "kernel": {"up": "k_ffn_mma (grouped up/gate + activation)",
                       "down": "k_ffn_mma (grouped down)",
                       "exit": "k_exit_mma (exit head + softmax partials)",
                       "shared": "k_ffn_mma (shared expert)"}[dom],
            "bound": "mfma",
            "achieved": dom_tflops,
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": dom_tflops / peak,
            "traffic": traffic,
            "traffic_unit": "bytes per launch",
            "traffic_source": traffic_src,
            "avg_launch_ms": dom_ms / launches[dom] if launches[dom] else None,
            "algorithmic_flop_per_step": flops[dom],
        },
        "grouped_gemm_mfma_frac": gg_frac,
        "active_token_layers_per_s": active_layers * K / (ms_total * 1e-3),
        "stack_roofline_frac": stack_bound_ms / ms_step,
        "kernel_ms_per_step": {n: float(t_class[i]) for i, n in enumerate(abi.TIMED_CLASSES)},
        "per_layer": [{k: w[k] for k in ("n_active", "n_exec", "rows", "distinct")} for w in work],
        "wall_s_timed_region": wall,
        "input_generation_s": t_gen,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(inp, args.cpu_seconds)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
