"""Benchmark of the placement evaluator on one MI355X.

A step is one pass of the placement path over the large workload (512 workers
with 512 resident requests each, 65536 arriving queries): every (query, worker)
pair is evaluated (KV peak, decode and TTFT checks), each query is resolved by
Algorithm 1 and committed in arrival order, diagnostics included.  Inputs and
worker state are resident in HBM before the timed region.  The same JSON line
reports the roofline position of the pair-evaluation kernel, the tiny, medium
and long workloads (the long one heartbeats, rebuilds and commits), the scaling
sweep (256 cluster configurations x 16384 queries, with its answer), Algorithm
2, the smallest cluster per arrival rate (Eq. 7), and the CPU oracle timed on a
bounded sample on this host.

    python bench.py [--gpus 1] [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import gc
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "query×worker placement evals/sec + scenario sweeps/sec; % of HBM roofline"
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, GB/s
# VALU issue: 256 compute units x 4 SIMDs x 16 lanes per clock x 2.4 GHz, in
# 10^12 32-bit lane operations per second (a wave64 instruction takes 4 clocks)
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
# 32-bit operations the pair evaluator needs per (query, worker) pair, counted
# from its formula: breakpoint slot 2, KV peak with the query 8, capacity test 1,
# decode test 4, TTFT test 1, feasibility 2, smallest-excess bookkeeping 4
OPS_PER_PAIR = 22
TILE_LARGE = 65536


def scan_equivalent_bytes_per_pair(residents_per_worker: int) -> int:
    """Bytes an O(R) scan of the worker's state would read per pair: the two
    int32 columns the breakpoint rule depends on plus five int64 aggregates."""
    return 8 * residents_per_worker + 40


# the translation unit of the pair-evaluation kernel
EVAL_SOURCES = ("ald_kernels.hip", "ald_device.h", "ald_internal.h")


def kernel_source_sha256() -> str:
    h = hashlib.sha256()
    for p in EVAL_SOURCES:
        p = os.path.join("paper_2405_06856_amd", "csrc", p)
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per pair-evaluation launch from the committed counter record,
    or None when the kernel source changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "pair_eval_large_traffic.json")
    try:
        with open(path) as f:
            doc = json.load(f)
    except (OSError, ValueError):
        return None
    if doc.get("kernel_source_sha256") != kernel_source_sha256():
        return None
    return doc.get("bytes_per_launch")


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def host_cores() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def cpu_baseline(trace, budget_s: float = 20.0, max_q: int = 16384):
    """The oracle as it stands, one thread, on the first n queries of the stream
    (n doubled until one run takes at least half the budget)."""
    from oracle import ref
    ref.build()
    n = 256
    while True:
        t0 = time.perf_counter()
        ref.place(trace.n_workers, trace.kv_capacity, trace.res_offsets, trace.res_l_in, trace.res_l_pred,
                  trace.res_generated, trace.model, trace.q_l_in[:n], trace.q_l_pred[:n], n_threads=1)
        dt = time.perf_counter() - t0
        if dt >= budget_s / 2 or n >= max_q:
            break
        n = min(max_q, 2 * n)
    nc = host_cores()
    return {"value": n * trace.n_workers / dt, "unit": "pair-evals/s", "cores": 1, "kind": "oracle",
            "host_cores": nc, "cpu_model": cpu_model(),
            "sample": "first %d of %d queries x %d workers of the large workload, 1 core of %d (%s), %.1f s"
                      % (n, trace.n_queries, trace.n_workers, nc, cpu_model(), dt)}


def no_gc(fn):
    """Run fn with the Python garbage collector off (a collector pass over
    torch's object graph takes tens of ms and is not the library's time)."""
    gc.collect()
    gc.disable()
    try:
        return fn()
    finally:
        gc.enable()


def time_workload(name: str, runs: int, tile: int = 4096):
    """Place a whole workload `runs` times from a fresh load (not timed), one
    warm-up first: wall time of the placement call (it returns when its stream
    work is done), and per-kernel device time from the library's events."""
    import torch

    from paper_2405_06856_amd import aladdin
    from paper_2405_06856_amd import workloads as wl
    t = wl.make_config(name)
    ev = aladdin.Evaluator(0, tile=tile)
    dev = ev.device
    ql = torch.as_tensor(t.q_l_in, dtype=torch.int32).to(dev)
    qp = torch.as_tensor(t.q_l_pred, dtype=torch.int32).to(dev)
    Q = t.n_queries
    out = torch.empty(Q, dtype=torch.int32, device=dev)
    dg = torch.empty(Q * aladdin.DIAG_DTYPE.itemsize, dtype=torch.uint8, device=dev)
    walls = []
    kinds = ("build", "eval", "select", "commit")
    kern = {k: 0.0 for k in kinds}
    rounds = 0
    for r in range(runs + 1):
        ev.load_trace(t)
        torch.cuda.synchronize()
        if r > 0:
            ev.profiling(True, kinds=kinds)

        def one():
            t0 = time.perf_counter()
            ev.place_device(ql, qp, t.heartbeat_every, diag=True, out=out, diag_out=dg)
            return time.perf_counter() - t0

        dt = no_gc(one)
        if r > 0:
            walls.append(dt)
            for k in kinds:
                kern[k] += ev.kernel_time(k)[0]
            rounds += ev.kernel_time("commit")[1]
            ev.profiling(False)
    placed = int((out >= 0).sum().item())
    ev.close()
    med = statistics.median(walls)
    pairs = Q * t.n_workers
    T = min(tile, t.heartbeat_every) if t.heartbeat_every else tile
    return {"workers": t.n_workers, "residents_per_worker": int(t.res_offsets[1] - t.res_offsets[0]),
            "queries": Q, "heartbeat_every": t.heartbeat_every, "tile": tile, "pairs": pairs, "placed": placed,
            "runs": runs, "ms_median": med * 1e3, "ms_min": min(walls) * 1e3, "pair_evals_per_s": pairs / med,
            "kernels_ms_per_run": {k: v / runs for k, v in kern.items()}, "rounds_per_run": rounds / runs,
            "tiles_per_run": -(-Q // T)}


def time_sweep(steps: int):
    import torch

    from paper_2405_06856_amd import aladdin
    from paper_2405_06856_amd import workloads as wl
    sw = wl.make_config("sweep")
    sev = aladdin.Evaluator(0, tile=1024)
    for _ in range(2):  # warm-up (and the workspace grows to its size)
        sev.sweep(sw.scenarios, sw.q_l_in, sw.q_l_pred, want_answer=True)
    torch.cuda.synchronize()
    walls = []

    def run():
        res = None
        for _ in range(steps):
            t0 = time.perf_counter()
            res = sev.sweep(sw.scenarios, sw.q_l_in, sw.q_l_pred, want_answer=True)
            walls.append(time.perf_counter() - t0)
        return res

    rej, first, _, (gpus, idx) = no_gc(run)
    sev.close()
    med = statistics.median(walls)
    return {"sweeps_per_s": 1.0 / med, "ms_per_sweep": med * 1e3, "ms_min": min(walls) * 1e3, "runs": steps,
            "scenarios": len(sw.scenarios), "queries": sw.n_queries, "min_total_gpus": gpus,
            "min_gpus_scenario": idx, "answer_from": "device (ald_sweep_scenarios out_min_gpus)"}


def scaling_over_rates(rates=(100.0, 200.0, 300.0, 400.0, 500.0), gpus_per_worker: int = 1):
    """Smallest cluster per arrival rate over the sweep's scenarios (heartbeat
    every rate * T_dec queries) and the Eq. 7 line fitted through them.  The
    rates keep the 16,384-query stream at 650 or more decode iterations, well
    past a typical output length, so the clusters reach a steady state."""
    from paper_2405_06856_amd import aladdin, scaling
    from paper_2405_06856_amd import workloads as wl
    sw = wl.make_config("sweep")
    ev = aladdin.Evaluator(0, tile=1024)
    t0 = time.perf_counter()
    pts = scaling.min_cluster_per_rate(ev, sw, rates, gpus_per_worker)
    dt = time.perf_counter() - t0
    ev.close()
    ok = [p for p in pts if p.workers is not None]
    k5 = c5 = None
    if len(ok) >= 2:
        k5, c5 = scaling.fit_eq7([p.rate for p in ok], [p.workers for p in ok])
    return {"gpus_per_worker": gpus_per_worker, "seconds": dt,
            "points": [{"rate": p.rate, "heartbeat_every": p.heartbeat_every, "workers": p.workers} for p in pts],
            "eq7_k5": k5, "eq7_c5": c5}


def time_rebalance(steps: int, oracle_problems: int = 0):
    """Algorithm 2 over the 256-problem workload, inputs resident on the device;
    every call starts from the same placement (a device copy inside the loop)."""
    import numpy as np
    import torch

    from paper_2405_06856_amd import aladdin
    from paper_2405_06856_amd import workloads as wl
    b = wl.make_config("rebalance")
    ev = aladdin.Evaluator(0)
    dev = ev.device
    d32 = lambda a: torch.as_tensor(np.ascontiguousarray(a), dtype=torch.int32).to(dev)
    old = [d32(x) for x in (b.old_worker, b.old_l_pred, b.old_l_out, b.old_l_real, b.old_l_repred)]
    nl, nw0 = d32(b.new_l_pred), d32(b.new_worker)
    nw = torch.empty_like(nw0)
    Wt = int(b.n_workers.sum())
    le = torch.empty(Wt, dtype=torch.int64, device=dev)
    be = torch.empty_like(le)
    mv = torch.empty(b.P, dtype=torch.int32, device=dev)
    obj = torch.empty(4 * b.P, dtype=torch.int64, device=dev)
    models = (aladdin.Model * b.P)(*[aladdin.to_model(m) for m in b.models])

    def call():
        nw.copy_(nw0)
        ev.call(aladdin.ald_rebalance, b.P, b.n_workers, models, b.old_offsets, *old, b.new_offsets, nl, nw,
                le, be, mv, 0, None, obj)

    for _ in range(2):
        call()
    ev.profiling(True, kinds=("rebalance",))
    torch.cuda.synchronize()
    walls = []

    def run():
        for _ in range(steps):
            t0 = time.perf_counter()
            call()
            walls.append(time.perf_counter() - t0)

    no_gc(run)
    k_ms, k_n = ev.kernel_time("rebalance")
    moves = int(mv.sum().item())
    ev.close()
    med = statistics.median(walls)
    out = {"problems_per_s": b.P / med, "ms_per_call": med * 1e3, "ms_min": min(walls) * 1e3,
           "kernel_ms_per_call": k_ms / max(k_n, 1), "problems": b.P, "workers": Wt,
           "ongoing": int(b.old_offsets[-1]), "new": int(b.new_offsets[-1]), "moves": moves}
    if oracle_problems > 0:
        from oracle import ref  # the CPU baseline leg may use the oracle
        t0 = time.perf_counter()
        for p in range(oracle_problems):
            ref.rebalance(*b.problem(p))
        out["oracle_problems_per_s"] = oracle_problems / (time.perf_counter() - t0)
        out["oracle_sample"] = "first %d problems, 1 core of %d" % (oracle_problems, host_cores())
    return out


def time_large(steps: int, warmup: int, calibrate_copy: int = 0):
    """The headline: K steps of the large workload on the library's stream."""
    import numpy as np
    import torch

    from paper_2405_06856_amd import aladdin
    from paper_2405_06856_amd import workloads as wl
    dev = torch.device("cuda", 0)
    if calibrate_copy > 0:  # a copy of known traffic, for scaling memory counters
        n = calibrate_copy * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    trace = wl.make_config("large")
    R = int(trace.res_offsets[1] - trace.res_offsets[0])
    W, Q = trace.n_workers, trace.n_queries
    pairs = W * Q
    ev = aladdin.Evaluator(0, tile=TILE_LARGE)
    t_load0 = time.perf_counter()
    ev.load_trace(trace)
    load_s = time.perf_counter() - t_load0
    ql = torch.as_tensor(trace.q_l_in, dtype=torch.int32).to(dev)
    qp = torch.as_tensor(trace.q_l_pred, dtype=torch.int32).to(dev)
    before = ev.summary()
    out = torch.empty(Q, dtype=torch.int32, device=dev)
    dg = torch.empty(Q * aladdin.DIAG_DTYPE.itemsize, dtype=torch.uint8, device=dev)
    status = torch.full((max(steps, warmup, 1),), 12345, dtype=torch.int32, device=dev)
    for k in range(warmup):
        ev.place_async(ql, qp, 0, diag=True, out=out, diag_out=dg, status=status[k:k + 1])
    torch.cuda.synchronize()
    # No query of this stream fits anywhere, so the worker state is the same at
    # the start of every step (checked below).  The steps are asynchronous
    # calls issued back to back, as a serving loop would issue them; each
    # writes its own status word, and every one must read ALD_OK (every query
    # decided in the rounds enqueued).  Inside the timed region only the
    # pair-evaluation kernel is timed (two events per step, without a
    # system-scope fence).
    assert (status[:warmup].cpu().numpy() == aladdin.ALD_OK).all(), "a warm-up step did not finish"
    status.fill_(12345)
    ev.profiling(True, kinds=("eval",))
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()

    def run():
        start.record(ev.stream)
        t0 = time.perf_counter()
        for k in range(steps):
            ev.place_async(ql, qp, 0, diag=True, out=out, diag_out=dg, status=status[k:k + 1])
        stop.record(ev.stream)
        torch.cuda.synchronize()
        return time.perf_counter() - t0

    wall = no_gc(run)
    gpu_ms = start.elapsed_time(stop)
    codes = status[:steps].cpu().numpy()
    assert (codes == aladdin.ALD_OK).all(), "timed steps that did not finish: %s" % codes[codes != aladdin.ALD_OK]
    eval_ms, eval_n = ev.kernel_time("eval")
    # latency of one step: synchronous calls, which return when their stream
    # work is done (host clock), in a separate pass
    ev.profiling(False)
    walls = []

    def run_sync():
        for _ in range(steps):
            t1 = time.perf_counter()
            ev.place_device(ql, qp, 0, diag=True, out=out, diag_out=dg)
            walls.append(time.perf_counter() - t1)

    no_gc(run_sync)
    # per-kernel breakdown from a separate, untimed pass
    ev.profiling(True)
    for _ in range(steps):
        ev.place_device(ql, qp, 0, diag=True, out=out, diag_out=dg)
    torch.cuda.synchronize()
    kern = {k: ev.kernel_time(k)[0] / steps for k in ("build", "eval", "select", "commit")}
    ev.profiling(False)
    placed = int((out >= 0).sum().item())
    after = ev.summary()
    ev.close()
    assert placed == 0 and all(np.array_equal(before[k], after[k]) for k in before), \
        "state changed during the large-workload steps"
    eval_avg_ms = eval_ms / max(eval_n, 1)
    pairs_per_launch = pairs * steps / max(eval_n, 1)
    return {"R": R, "pairs": pairs, "gpu_ms": gpu_ms, "wall": wall, "walls": walls, "eval_avg_ms": eval_avg_ms,
            "pairs_per_launch": pairs_per_launch, "kernels": kern, "load_s": load_s, "trace": trace}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--sweep-steps", type=int, default=5)
    ap.add_argument("--runs", type=int, default=5, help="timed runs of the long workload (twice as many of the "
                                                        "tiny and medium ones)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-rebalance", action="store_true")
    ap.add_argument("--no-scaling", action="store_true", help="skip the smallest cluster per arrival rate")
    ap.add_argument("--no-workloads", action="store_true", help="skip the tiny, medium and long workloads")
    ap.add_argument("--only", choices=("large", "sweep", "rebalance", "long", "medium", "tiny"),
                    help="time one part only (for profiling)")
    ap.add_argument("--sweep-only", action="store_true", help="same as --only sweep")
    ap.add_argument("--rebalance-only", action="store_true", help="same as --only rebalance")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="also run a plain device-to-device copy of MIB MiB (a reference kernel of known "
                         "traffic for scaling memory counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the evaluator runs on a single device "
              "(multi-GPU sharding is a design note, not built)", file=sys.stderr)
        sys.exit(2)
    only = args.only or ("sweep" if args.sweep_only else ("rebalance" if args.rebalance_only else None))
    if only == "sweep":
        print(json.dumps({"sweep": time_sweep(args.sweep_steps)}), flush=True)
        return
    if only == "rebalance":
        print(json.dumps({"rebalance": time_rebalance(args.steps)}), flush=True)
        return
    if only in ("long", "medium", "tiny"):
        print(json.dumps({only: time_workload(only, args.runs)}), flush=True)
        return
    if only == "large":
        args.no_workloads = args.no_sweep = args.no_rebalance = args.no_scaling = args.no_cpu = True

    L = time_large(args.steps, args.warmup, args.calibrate_copy)
    ms_per_step = L["gpu_ms"] / args.steps
    value = L["pairs"] / (ms_per_step / 1e3)
    eval_s = L["eval_avg_ms"] / 1e3
    achieved_tops = OPS_PER_PAIR * L["pairs_per_launch"] / eval_s / 1e12
    traffic = measured_traffic() if L["pairs_per_launch"] == L["pairs"] else None
    walls = sorted(L["walls"])
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "pair-evals/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32/int64 tokens + fp64 latencies",
        "data": "synthetic",
        "config": {"workload": "large: 512 workers x 512 resident requests, 65536 queries, KV 262144 tokens, "
                               "lognormal lengths (input mu 6.5 sigma 1.2 [16,8192], output mu 5.5 sigma 1.0 "
                               "[8,2048]), diagnostics on",
                   "pairs_per_step": L["pairs"], "tile": TILE_LARGE, "parallelism": "single GPU"},
        "step_ms": {"median": statistics.median(walls) * 1e3, "min": walls[0] * 1e3, "mean_device": ms_per_step,
                    "clock": "mean_device (= ms_per_step): events around the timed region of asynchronous steps "
                             "issued back to back; median and min: host clock per synchronous step (returns when "
                             "its stream work is done), a separate pass"},
        "roofline": {"bound": "alu", "achieved": achieved_tops, "peak": VALU_PEAK_TOPS, "unit": "Tops/s",
                     "frac": achieved_tops / VALU_PEAK_TOPS, "traffic": traffic,
                     "kernel": "k_eval (pair evaluation)", "kernel_avg_ms": L["eval_avg_ms"],
                     "ops_per_pair": OPS_PER_PAIR, "pairs_per_launch": L["pairs_per_launch"],
                     "hbm_frac": (traffic / eval_s / 1e9 / HBM_PEAK_GBS) if traffic else None,
                     "scan_equivalent_GBps": scan_equivalent_bytes_per_pair(L["R"]) * L["pairs_per_launch"]
                     / eval_s / 1e9},
        "kernels_ms_per_step": L["kernels"],
        "wall_ms_per_step": L["wall"] * 1e3 / args.steps,
        "load_ms": L["load_s"] * 1e3,
    }
    if not args.no_workloads:
        line["workloads"] = {n: time_workload(n, args.runs if n == "long" else 2 * args.runs)
                             for n in ("tiny", "medium", "long")}
    line["sweep"] = None if args.no_sweep else time_sweep(args.sweep_steps)
    line["rebalance"] = None if args.no_rebalance else time_rebalance(args.steps, 0 if args.no_cpu else 8)
    line["eq7_scaling"] = None if (args.no_sweep or args.no_scaling) else scaling_over_rates()
    if not args.no_cpu:
        line["cpu_baseline"] = cpu_baseline(L["trace"])
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
