#!/usr/bin/env python3
"""Benchmark of the ScaDLES hot path on one MI355X.

One step = the whole hot path over one iteration's synthetic input: Eqn 4a
weights (host), Top-k selection + energies + adaptive rule for every device,
Eqn 4b weighted aggregation and the Eqn 4c SGD update, i.e. one
scadles_step_fused call. Default workload: 32 devices x 143,667,240 fp32
gradient elements (VGG-19-sized), ratio 0.01, 10 consecutive iterations, each
with its own gradients, weights and learning rate; the timed steps cycle
through the iterations. Every iteration's gradients are resident in HBM
before the timed region starts (184 GB for the default workload).

Prints one JSON line (metric: gradient elements compressed+aggregated per
second; roofline of the dominant kernel, the main select pass, against the
8 TB/s HBM peak; the whole step's fraction of that peak, the figure the
target is stated in; standalone timings of the three calls of the path; the
CPU oracle's rate on a bounded sample).
"""
from __future__ import annotations

import argparse
import hashlib
import json
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


def host_cpu():
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except AttributeError:
        usable = os.cpu_count()
    return {"model": model, "nproc": os.cpu_count(), "usable": usable}


def cpu_baseline(s, threads):
    """The oracle, as it stands, on a bounded sample of the same workload:
    device 0's Top-k (full sort) on one thread, then the step of `threads`
    devices of iteration 0 -- their Top-k (full sort, energies) on parallel
    threads, Eqn 4b (serial double sums) and Eqn 4c -- each part timed."""
    import oracle
    import workloads
    from concurrent.futures import ThreadPoolExecutor

    S = max(1, min(s.K, threads))
    ks = [oracle.topk_k(s.n, s.ratios[0, j]) for j in range(S)]
    G = np.empty((S, s.n), dtype=np.float32)
    for j in range(S):
        workloads.gradient(s, 0, j, out=G[j], k=ks[j])
    t0 = time.perf_counter()
    oracle.topk(G[0], ks[0])
    t_single = time.perf_counter() - t0
    t0 = time.perf_counter()
    w, gamma = oracle.stream_weights(s.rates[0, :S], base_batch=s.base_batch)
    with ThreadPoolExecutor(S) as ex:
        res = list(ex.map(lambda j: oracle.topk(G[j], ks[j]), range(S)))
    t1 = time.perf_counter()
    dense = oracle.aggregate([(r[0], r[1]) for r in res], w, s.n)
    t2 = time.perf_counter()
    params = np.zeros(s.n, dtype=np.float32)
    oracle.sgd(params, dense, float(np.float32(s.eta * gamma)))
    t3 = time.perf_counter()
    dt = t3 - t0
    return {"value": S * s.n / dt, "unit": "elements/s", "cores": S, "kind": "oracle",
            "sample": f"{S} of the {s.K} devices (iteration 0, full n={s.n} each): full-sort Top-k of the "
                      f"{S} devices on {S} threads, serial double aggregation of their sets, SGD; "
                      f"{dt:.1f} s wall",
            "host": host_cpu(),
            "seconds": {"topk_parallel": t1 - t0, "aggregate": t2 - t1, "sgd": t3 - t2, "step": dt,
                        "topk_device0_single_thread": t_single},
            "single_thread_topk_elements_per_s": s.n / t_single}


def event_ms(torch, fn, reps, stream=None):
    """Average milliseconds of fn() over reps calls, HIP events around them."""
    for _ in range(2):
        fn()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / reps


def roof(nbytes, ms):
    gbps = nbytes / (ms * 1e-3) / 1e9
    return {"ms": ms, "bytes": nbytes, "GBps": gbps, "frac": gbps / HBM_PEAK_GBPS}


def bench_layers(args, s, sc, torch, G, params, weights, lrs):
    """The hot path with the per-layer Top-k (the workload's layer layout):
    per-layer selection of every device, Eqn 4b over the layered sets and
    Eqn 4c, in one library call per step. Timed as whole steps; the roofline
    entry is the step's algorithmic bytes over its time."""
    seg_off = [0] + [int(x) for x in s.seg_end]
    if args.row_max is not None:
        sc.set_option("row_max", args.row_max)
    if args.row_split is not None:
        sc.set_option("row_split", args.row_split)
    step = sc.FusedStep(G[0], s.ratios[0], params=params, seg_off=seg_off)
    R = len(G)
    for i in range(args.warmup):
        it = i % s.iterations
        step.set_grads(G[it % R])
        step.run(weights[it], lrs[it])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        it = i % s.iterations
        step.set_grads(G[it % R])
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
                   "iterations": s.iterations, "resident_gradient_sets": R,
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
    ap.add_argument("--resident", type=int, default=None,
                    help="iterations whose gradients are kept in HBM and cycled (default: every iteration of "
                         "the workload, fewer only if HBM cannot hold them)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-standalone", action="store_true",
                    help="skip the standalone timings of scadles_topk_select, scadles_weighted_aggregate "
                         "and scadles_apply_sgd")
    ap.add_argument("--cpu-threads", type=int, default=16)
    ap.add_argument("--stages", action="store_true", help="also print per-stage milliseconds")
    ap.add_argument("--parts", type=int, default=1,
                    help="device groups whose selections are pipelined (library option 'parts')")
    ap.add_argument("--optimizer", choices=("sgd", "momentum"), default="sgd",
                    help="update after the aggregation: Eqn 4c (default), or momentum SGD 0.9 with weight "
                         "decay 5e-4 (the VGG19 setup of the paper's evaluation)")
    ap.add_argument("--topk", choices=("global", "layers"), default="global",
                    help="Top-k over each flat gradient (default), or per layer of the workload's layer "
                         "layout (each layer keeps its own top fraction), in one fused call per step")
    ap.add_argument("--stream", choices=("none", "persistence", "truncation"), default="none",
                    help="take every step's weights and learning rate from the devices' stream buffers "
                         "under this policy (host, inside the timed step): the workload's rates as samples/s, "
                         "iterations of --iter-s seconds, batches bounded to [8, 1024]")
    ap.add_argument("--iter-s", type=float, default=1.6,
                    help="simulated iteration time of --stream (default 1.6 s, the paper's VGG19 iteration)")
    ap.add_argument("--row-max", type=int, default=None,
                    help="with --topk layers: layers of at most this many elements are selected one workgroup "
                         "per (device, layer) (library option 'row_max')")
    ap.add_argument("--row-split", type=int, default=None,
                    help="--topk layers: rows of more than this many elements are split over several "
                         "workgroups (library option 'row_split')")
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
    # Every iteration's gradients resident at once (as many as HBM holds with
    # room for the workspace and outputs), generated on the host device by
    # device and copied in.
    per_set = 4 * s.K * s.n
    free, _ = torch.cuda.mem_get_info()
    fit = max(1, int((free - 24 * 2**30) // per_set))
    R = min(s.iterations, fit, args.resident or s.iterations)
    G = []
    host = np.empty(s.n, dtype=np.float32)
    for it in range(R):
        g = torch.empty((s.K, s.n), dtype=torch.float32, device=dev)
        for j in range(s.K):
            workloads.gradient(s, it, j, out=host, k=sc.topk_k(s.n, s.ratios[it, j]))
            g[j].copy_(torch.from_numpy(host))
        G.append(g)
    params = torch.from_numpy(workloads.params0(s)).to(dev)
    torch.cuda.synchronize()
    log(f"{R} iteration(s) of gradients resident in HBM ({R * per_set / 1e9:.1f} GB) after "
        f"{time.perf_counter() - t0:.1f} s")

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
    if args.topk == "layers":
        return bench_layers(args, s, sc, torch, G, params, weights, lrs)
    extra = {} if args.ewma is None else {"ewma_beta": args.ewma, "track": True}
    mbuf = torch.zeros_like(params) if args.optimizer == "momentum" else None
    opt = dict(momentum_buf=mbuf, momentum=0.9, weight_decay=5e-4) if mbuf is not None else {}
    # one step object (outputs and workspace) per distinct ratio vector of the
    # workload's iterations, all allocated before the timed region; a step only
    # switches its gradient pointers
    steps = {}
    for it in range(s.iterations):
        key = tuple(float(r) for r in s.ratios[it])
        if key not in steps:
            steps[key] = sc.FusedStep(G[it % R], s.ratios[it], params=params, **opt, **extra)
    plan = [(steps[tuple(float(r) for r in s.ratios[it])], G[it % R]) for it in range(s.iterations)]

    def run_step(i, w=None, lr=None):
        it = i % s.iterations
        step, g = plan[it]
        step.set_grads(g)
        step.run(weights[it] if w is None else w, lrs[it] if lr is None else lr)

    for i in range(args.warmup):
        run_step(i)
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
        if buffers is not None:
            h0 = time.perf_counter()
            _, w, gamma = buffers.iteration(iter_us)
            lr = float(np.float32(s.eta * gamma))
            host_s += time.perf_counter() - h0
            run_step(i, w, lr)
        else:
            run_step(i)
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
        "config": {"workload": s.name, "K": s.K, "n": s.n,
                   "ratios": sorted({float(r) for r in s.ratios.ravel()}),
                   "delta": "inf", "iterations": s.iterations, "resident_gradient_sets": R,
                   "gradients": ("every iteration's own, cycled over the steps" if R == s.iterations else
                                 f"the first {R} iterations' gradients cycled over the steps"),
                   "sgd": True, "cache_evicted": bool(args.evict),
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
                          "note": "the target's figure: the whole fused step (select + compact + aggregate, "
                                  "with the SGD update folded in), algorithmic bytes 4Kn + 8*sum(k) + 4n over "
                                  "its event-timed duration"},
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
    step0, g0 = plan[0]
    dense = step0.dense
    sgd_ms = event_ms(torch, lambda: sc.apply_sgd(params, dense, 0.0), 20)
    out["sgd_alone"] = dict(roof(12 * s.n, sgd_ms),
                            note="scadles_apply_sgd on n elements (lr 0), HIP events on the stream it runs on")
    if not args.no_standalone:
        # Top-k of one gradient (device 0 of iteration 0): one read of n floats
        # and the k kept pairs written
        k0 = sc.topk_k(s.n, s.ratios[0, 0])
        ws = torch.empty(sc.workspace_bytes(1, s.n, [s.ratios[0, 0]]), dtype=torch.uint8, device=dev)
        t_ms = event_ms(torch, lambda: sc.topk_select(g0[0], s.ratios[0, 0], workspace=ws), 10)
        out["topk_select_alone"] = dict(roof(4 * s.n + 8 * k0, t_ms), elements_per_s=s.n / (t_ms * 1e-3),
                                        note="scadles_topk_select on device 0's gradient (n elements), "
                                             "algorithmic bytes 4n + 8k")
        # Eqn 4b of the step's K sparse sets (the last step's outputs): the
        # pairs read and the dense aggregate written
        step0.set_grads(g0)
        o = step0.run(weights[0], lrs[0])
        sets = list(zip(o.idx, o.val))
        agg_out = torch.empty(s.n, dtype=torch.float32, device=dev)
        aws = torch.empty(sc.aggregate_workspace_bytes(s.K, s.n), dtype=torch.uint8, device=dev)
        ks = sum(t.numel() for t in o.idx)
        a_ms = event_ms(torch, lambda: sc.weighted_aggregate(sets, weights[0], s.n, out=agg_out, workspace=aws), 10)
        out["weighted_aggregate_alone"] = dict(roof(8 * ks + 4 * s.n, a_ms),
                                               note="scadles_weighted_aggregate of the K sparse sets of a "
                                                    "step, algorithmic bytes 8*sum(k) + 4n")
        del ws, aws, agg_out, sets, o
    if not args.no_cpu_baseline:
        del G, plan, steps, g0, step0, dense
        torch.cuda.empty_cache()
        log("timing the CPU oracle on a bounded sample ...")
        out["cpu_baseline"] = cpu_baseline(s, args.cpu_threads)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
