#!/usr/bin/env python3
"""Benchmark of the ScaDLES hot path on one MI355X.

One step = the whole hot path over one batch of synthetic input: Eqn 4a
weights (host), Top-k selection + energies + adaptive rule for every device,
Eqn 4b weighted aggregation and the Eqn 4c SGD update, i.e. one
scadles_step_fused call. Default workload: 32 devices x 143,667,240 fp32
gradient elements (VGG-19-sized), ratio 0.01, the weights and learning rates
of 10 consecutive iterations cycled over the steps. Inputs are resident in HBM
before the timed region starts.

Prints one JSON line (metric: gradient elements compressed+aggregated per
second; roofline of the dominant kernel, the main select pass, against the
8 TB/s HBM peak; the CPU oracle's rate on a bounded sample).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
METRIC = "gradient elements/s compressed+aggregated; % of MI355X HBM roofline"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_main_select_c5.json")
SELECT_SRC = os.path.join(ROOT, "paper_2301_08897_amd", "csrc", "select.hip")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(sc, s, it):
    """Bytes the method itself must move in one step (select + compact + aggregate):
    read every gradient once, write the (idx, val) pairs, write the dense aggregate."""
    ks = sum(sc.topk_k(s.n, s.ratios[it, j]) for j in range(s.K))
    return 4 * s.K * s.n + 8 * ks + 4 * s.n


def source_hash(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic_entry(parts):
    """HBM bytes per launch of the main select pass measured by rocprofv3 counters,
    if recorded for the current kernel source and the same number of launches."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("select_hip_sha256_16") != source_hash(SELECT_SRC) or t.get("parts") != parts:
        return None
    return t.get("hbm_bytes_per_launch")


def cpu_baseline(s, threads):
    """The oracle, as it stands, on a bounded sample of the same workload: the full
    step (Top-k by full sort, energies, Eqn 4b, Eqn 4c) for `threads` devices of
    iteration 0, the devices' Top-k run in parallel threads."""
    import oracle
    import workloads
    from concurrent.futures import ThreadPoolExecutor

    S = max(1, min(s.K, threads))
    G = np.empty((S, s.n), dtype=np.float32)
    for j in range(S):
        workloads.gradient(s, 0, j, out=G[j], k=oracle.topk_k(s.n, s.ratios[0, j]))
    rates = s.rates[0, :S]
    t0 = time.perf_counter()
    w, gamma = oracle.stream_weights(rates, base_batch=s.base_batch)
    ks = [oracle.topk_k(s.n, s.ratios[0, j]) for j in range(S)]
    with ThreadPoolExecutor(S) as ex:
        res = list(ex.map(lambda j: oracle.topk(G[j], ks[j]), range(S)))
    dense = oracle.aggregate([(r[0], r[1]) for r in res], w, s.n)
    params = np.zeros(s.n, dtype=np.float32)
    oracle.sgd(params, dense, float(np.float32(s.eta * gamma)))
    dt = time.perf_counter() - t0
    return {"value": S * s.n / dt, "unit": "elements/s", "cores": S, "kind": "oracle",
            "sample": f"{S} of the {s.K} devices (iteration 0, full n={s.n} each): full-sort Top-k "
                      f"in {S} threads, serial double aggregation and SGD; {dt:.1f} s wall"}


def bench_layers(args, s, sc, torch, G, params, weights, lrs):
    """The hot path with the per-layer Top-k (the workload's layer layout):
    per-layer selection of every device, Eqn 4b over the layered sets and
    Eqn 4c, in one library call per step. Timed as whole steps; the roofline
    entry is the step's algorithmic bytes over its time."""
    seg_off = [0] + [int(x) for x in s.seg_end]
    if args.row_max is not None:
        sc.set_option("row_max", args.row_max)
    step = sc.FusedStep(G, s.ratios[0], params=params, seg_off=seg_off)
    for i in range(args.warmup):
        it = i % s.iterations
        step.run(weights[it], lrs[it])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        it = i % s.iterations
        step.run(weights[it], lrs[it])
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms = dt * 1e3 / args.steps
    ks = sum(step.k)
    alg = 4 * s.K * s.n + 8 * ks + 4 * s.n
    gbps = alg / (ms * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": s.K * s.n / (dt / args.steps), "unit": "elements/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": s.name, "K": s.K, "n": s.n, "ratio": float(s.ratios[0, 0]), "delta": "inf",
                   "topk": f"per layer ({len(seg_off) - 1} layers), {ks // s.K} entries kept per device",
                   "optimizer": "SGD (Eqn 4c)"},
        "roofline": {"bound": "hbm", "achieved": gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": gbps / HBM_PEAK_GBPS, "traffic": None,
                     "kernel": "whole step (algorithmic bytes 4Kn + 8*sum(k) + 4n over the step time)"},
    }
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=5, help="workload 1..5 (default 5, the largest)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-threads", type=int, default=16)
    ap.add_argument("--stages", action="store_true", help="also print per-stage milliseconds")
    ap.add_argument("--parts", type=int, default=1,
                    help="device groups whose selections are pipelined (library option 'parts')")
    ap.add_argument("--optimizer", choices=("sgd", "momentum"), default="sgd",
                    help="update after the aggregation: Eqn 4c (default), or momentum SGD 0.9 with weight "
                         "decay 5e-4 (the VGG19 setup of the paper's evaluation)")
    ap.add_argument("--topk", choices=("global", "layers"), default="global",
                    help="Top-k over each flat gradient (default), or per layer of the workload's layer "
                         "layout (each layer keeps its own top fraction; three library calls per step: "
                         "per-layer selection, Eqn 4b aggregation, Eqn 4c SGD)")
    ap.add_argument("--stream", choices=("none", "persistence", "truncation"), default="none",
                    help="take every step's weights and learning rate from the devices' stream buffers "
                         "under this policy (host, inside the timed step): the workload's rates as samples/s, "
                         "iterations of --iter-s seconds, batches bounded to [8, 1024]")
    ap.add_argument("--iter-s", type=float, default=1.6,
                    help="simulated iteration time of --stream (default 1.6 s, the paper's VGG19 iteration)")
    ap.add_argument("--row-max", type=int, default=None,
                    help="with --topk layers: layers of at most this many elements are selected one workgroup "
                         "per (device, layer) (library option 'row_max')")
    ap.add_argument("--ewma", type=float, default=None, metavar="BETA",
                    help="adaptive rule on moving averages of the energies with this factor, and the CNC / "
                         "floats-sent accounting, inside the fused step (delta stays +inf)")
    ap.add_argument("--evict", action="store_true",
                    help="write 1 GiB of scratch before every timed step (not timed) so that no input sits in "
                         "the 256 MB last-level cache; step times then come from events around each step")
    ap.add_argument("--calibrate", action="store_true",
                    help="first run one 1 GiB device-to-device copy (a plain copy kernel of known size "
                         "for scaling HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the hot path keeps all simulated devices in one GPU's HBM "
              "and has no multi-GPU mode; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2301_08897_amd as sc
    import workloads

    dev = torch.device("cuda:0")
    s = workloads.spec(args.config)
    log(f"workload {s.name}")
    t0 = time.perf_counter()
    G = torch.empty((s.K, s.n), dtype=torch.float32, device=dev)
    host = np.empty(s.n, dtype=np.float32)
    for j in range(s.K):
        workloads.gradient(s, 0, j, out=host, k=sc.topk_k(s.n, s.ratios[0, j]))
        G[j].copy_(torch.from_numpy(host))
    params = torch.from_numpy(workloads.params0(s)).to(dev)
    torch.cuda.synchronize()
    log(f"inputs resident in HBM ({4 * s.K * s.n / 1e9:.1f} GB) after {time.perf_counter() - t0:.1f} s")

    if args.calibrate:
        src = torch.empty(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        src.fill_(1.0)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        torch.cuda.empty_cache()

    weights, lrs = [], []
    for it in range(s.iterations):
        w, gamma = sc.stream_weights(s.rates[it], base_batch=s.base_batch)
        weights.append(w)
        lrs.append(float(np.float32(s.eta * gamma)))
    sc.set_option("parts", args.parts)
    parts = min(args.parts, s.K)
    extra = {} if args.ewma is None else {"ewma_beta": args.ewma, "track": True}
    if args.optimizer == "momentum":
        mbuf = torch.zeros_like(params)
        step = sc.FusedStep(G, s.ratios[0], params=params, momentum_buf=mbuf, momentum=0.9, weight_decay=5e-4,
                            **extra)
    else:
        step = sc.FusedStep(G, s.ratios[0], params=params, **extra)
    if args.topk == "layers":
        return bench_layers(args, s, sc, torch, G, params, weights, lrs)
    for i in range(args.warmup):
        it = i % s.iterations
        if any(s.ratios[it] != s.ratios[0]):
            step.set_ratios(s.ratios[it])
        step.run(weights[it], lrs[it])
    torch.cuda.synchronize()

    buffers, host_s = None, 0.0
    if args.stream != "none":
        buffers = sc.StreamBuffers(np.rint(s.rates[0]).astype(np.uint64), b_min=8, b_max=1024, policy=args.stream,
                                   base_batch=s.base_batch)
        iter_us = int(round(args.iter_s * 1e6))

    sc.profile_enable(True)
    # per-step times: an event on the caller's stream after every step (with
    # --evict also one before every step, after the cache-evicting write)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)] if args.evict else None
    scratch = torch.empty(1 << 28, dtype=torch.float32, device=dev) if args.evict else None
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    marks[0].record()
    for i in range(args.steps):
        if scratch is not None:
            scratch.fill_(float(i))
            starts[i].record()
        it = i % s.iterations
        if buffers is not None:
            h0 = time.perf_counter()
            _, w, gamma = buffers.iteration(iter_us)
            lr = float(np.float32(s.eta * gamma))
            host_s += time.perf_counter() - h0
            step.run(w, lr)
        else:
            step.run(weights[it], lrs[it])
        marks[i + 1].record()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    if starts is not None:
        per_step = sorted(starts[i].elapsed_time(marks[i + 1]) for i in range(args.steps))
        dt = sum(per_step) * 1e-3
    else:
        per_step = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps))
    stages, calls = sc.profile_read()
    sc.profile_enable(False)

    ms_per_step = dt * 1e3 / args.steps
    value = s.K * s.n / (dt / args.steps)
    # The main pass runs as `parts` launches (devices split evenly), each reading
    # its devices' gradients once: per launch 4 * (K / parts) * n bytes.
    launch_ms = stages["main_select"] / max(calls, 1) / parts
    launch_bytes = 4 * s.K * s.n / parts
    achieved = launch_bytes / (launch_ms * 1e-3) / 1e9
    alg = np.mean([algorithmic_bytes(sc, s, i % s.iterations) for i in range(args.steps)])
    sel_ms = stages["total"] / max(calls, 1)
    traffic = traffic_entry(parts)

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "elements/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "ms_median": per_step[len(per_step) // 2],
        "ms_min": per_step[0],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": s.name, "K": s.K, "n": s.n, "ratio": float(s.ratios[0, 0]),
                   "delta": "inf", "iterations": s.iterations, "sgd": True, "cache_evicted": bool(args.evict),
                   "adaptive": ("moving average, beta %g, with accounting" % args.ewma if args.ewma is not None
                                else "instantaneous energies"),
                   "optimizer": ("momentum SGD 0.9, weight decay 5e-4" if args.optimizer == "momentum"
                                 else "SGD (Eqn 4c)")},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": traffic,
                     "kernel": "k_main (main select pass: one read of every gradient)",
                     "launch_ms": launch_ms, "launch_bytes": launch_bytes, "launches_per_step": parts},
        "step_roofline": {"algorithmic_bytes": alg, "GBps": alg / (sel_ms * 1e-3) / 1e9,
                          "frac": alg / (sel_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                          "note": "select+compact+aggregate(+SGD) stages, algorithmic bytes "
                                  "4Kn + 8*sum(k) + 4n over their summed event time"},
    }
    if buffers is not None:
        out["config"]["stream"] = {"policy": args.stream, "iteration_s": args.iter_s, "b_min": 8, "b_max": 1024}
        out["stream"] = {"host_us_per_iteration": host_s * 1e6 / args.steps,
                         "queued_samples_after": int(buffers.field("queued").sum()),
                         "dropped_samples": int(buffers.field("dropped").sum())}
        # the buffer simulation alone: all devices over 10^5 iterations (after one untimed run)
        sim = (np.rint(s.rates[0]).astype(np.uint64), [iter_us] * s.K, 8, 1024, args.stream, 100_000)
        sc.stream_simulate(*sim)
        h0 = time.perf_counter()
        sc.stream_simulate(*sim)
        out["stream"]["simulate_ns_per_device_iteration"] = (time.perf_counter() - h0) * 1e9 / (s.K * 100_000)
    if args.stages:
        out["stage_ms"] = {k: v / max(calls, 1) for k, v in stages.items()}
    # Eqn 4c on its own (the fused step folds it into the aggregation): reads
    # params and the aggregate, writes params, 12 n bytes per call
    dense = step.dense
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(3):
        sc.apply_sgd(params, dense, 0.0)
    ev0.record()
    for _ in range(20):
        sc.apply_sgd(params, dense, 0.0)
    ev1.record()
    torch.cuda.synchronize()
    sgd_ms = ev0.elapsed_time(ev1) / 20
    out["sgd_alone"] = {"ms": sgd_ms, "bytes": 12 * s.n, "GBps": 12 * s.n / (sgd_ms * 1e-3) / 1e9,
                        "frac": 12 * s.n / (sgd_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                        "note": "scadles_apply_sgd on n elements (lr 0), HIP events on the stream it runs on"}
    if not args.no_cpu_baseline:
        del G, step
        torch.cuda.empty_cache()
        log("timing the CPU oracle on a bounded sample ...")
        out["cpu_baseline"] = cpu_baseline(s, args.cpu_threads)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
