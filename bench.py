#!/usr/bin/env python3
"""Benchmark of the global policy pass on one MI355X.

One step = one full pass (validation, remaining critical path, readiness,
slack, routing, ordering) over the paper-scale snapshot: 4,096 workflows x 32
futures = 131,072 in-flight futures (the largest point of the paper's
scalability study, Section 6.3), inputs already resident in HBM.  That is the
headline: futures/s per pass, whole job.

The same JSON line carries, from the same run:
  roofline         the dominant kernel of the headline pass: algorithmic bytes
                   per launch over its mean duration (HIP events recorded by
                   the library on its own stream), and its measured HBM traffic
                   (two rocprofv3 --pmc child runs, FETCH_SIZE then WRITE_SIZE,
                   scaled by what the same counters read for a plain copy);
  first_pass       paper scale: latency of the first pass over a changed
                   snapshot (1 % of in-flight futures completed, or every
                   deadline moved), the pass a controller makes once per change;
  wide_mapreduce   1,049,088 futures with 1,048,576 ready: pass latency,
                   kernels and roofline (the workload where the HBM roofline
                   is the fair yardstick);
  dynamic          the map/reduce graph evolving over 100 steps (1.05M ->
                   12.4M futures) in the graph store: first-pass and
                   repeat-pass latency per step, full passes beside them
                   every 25 steps, and (one_pass_per_change) the first passes
                   again with no repeated pass in between;
  cpu_baseline     the CPU oracle timed on this host, one core.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload paper-scale]

Other workloads: tiny, deep-chains, wide-mapreduce, dynamic, levels (one-level
per-event decisions against two-level passes over 1K-131K futures).
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import platform
import shutil
import statistics
import subprocess
import sys
import tempfile
import time

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E
ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)


# ---------------------------------------------------------------- byte models

def alg_bytes(kernel: str, N: int, E: int, R: int, W: int, M: int, grouped: bool) -> float:
    """Algorithmic bytes one launch of a kernel must move: every input it needs
    read once and every output it produces written once, at the widths of the
    C ABI (int64 times, int32 ids and offsets, uint8 flags).  Re-reads, counters,
    look-back words and other traffic an implementation adds are not counted.

    sweep      per future 21 (est 8, done 1, dep_off 4, rem 8), per dependency 4,
               per ready future 28 (type 4, loc 4, staged slack 8, route 4,
               cost 8), per workflow 8 (deadline), per instance 16
    nodes      per future 25 (wf, type, loc, dep_off 4 each, est 8, done 1),
               per workflow 8, per instance 16
    sort_hist  per ready future 8 (slack key)
    sort_pass  per ready future 24 (key 8 + payload 4, read and written)
    last pass  per ready future 48 (key, payload, staged route and cost read;
               order, slack, route, cost written)
    sort_bucket per ready future 48 (bucketed slack, position, route, cost
               read; order, slack, route, cost written)
    """
    if kernel == "sweep":
        b = 21 * N + 4 * E + 28 * R + 8 * W + 16 * M
        if grouped:
            b += 4 * N  # workflow ids
        return float(b)
    if kernel == "nodes":
        return float(25 * N + 8 * W + 16 * M)
    if kernel == "sort_bucket":
        return float(48 * R)
    if kernel == "sort_hist":
        return float(8 * R)
    if kernel == "sort_pass3":
        return float(48 * R)
    if kernel.startswith("sort_pass"):
        return float(24 * R)
    return 0.0


def pass_alg_bytes(N: int, E: int, R: int, W: int, M: int) -> float:
    """What one whole pass must move: per future 21, per dependency 4, per ready
    future 36 (wf, type, loc read; order, slack, route, cost written), per
    workflow 8, per instance 16."""
    return float(21 * N + 4 * E + 36 * R + 8 * W + 16 * M)


# The rocprofv3 kernel names of the library's timing labels.
KERNEL_SYMBOL = {"sweep": "k_sweep", "sort_bucket": "k_bucket_sort", "nodes": "k_nodes"}


def workload(name: str):
    from paper_2601_05109_amd import workloads as wl
    if name not in wl.WORKLOADS:
        raise SystemExit(f"unknown workload {name}")
    return wl.WORKLOADS[name]()


def pct(xs, f):
    xs = sorted(xs)
    return xs[min(len(xs) - 1, int(f * len(xs)))] if xs else None


def rnd(x, d=2):
    return None if x is None else round(float(x), d)


# ---------------------------------------------------------------- one workload

class Runner:
    """A snapshot resident in HBM, a handle on the torch stream and one
    synchronous pass per call."""

    def __init__(self, p, policy_bits=0, priority=None):
        import torch
        from paper_2601_05109_amd import nalar
        self.torch, self.nalar, self.p = torch, nalar, p
        self.dev = torch.device("cuda", 0)
        self.stream = torch.cuda.current_stream(self.dev)
        self.dp = nalar.DeviceProblem.from_host(p, self.dev)
        self.out = nalar.DeviceResult.alloc(p.n_nodes, self.dev)
        self.pol = nalar.Policy(device=0, stream=self.stream, reserve_nodes=p.n_nodes,
                                reserve_workflows=p.n_workflows)
        self.cp = self.dp.c_struct(policy=policy_bits, priority=priority)
        self.cr = self.out.c_struct()  # built once, as a caller's loop would

    def one(self) -> int:
        rc = self.nalar.nalar_policy_pass(self.pol.handle, self.cp, self.cr)
        if rc != self.nalar.NALAR_OK:
            raise RuntimeError(f"pass failed {rc}: {self.pol.last_error()}")
        return int(self.cr.n_ready)

    def swap(self, p):
        """Upload another snapshot of the same shape (not timed)."""
        self.p = p
        self.dp = self.nalar.DeviceProblem.from_host(p, self.dev)
        self.cp = self.dp.c_struct()
        self.torch.cuda.synchronize()

    def timed(self, steps: int):
        """Wall time of each synchronous call, and the device time of all of
        them from HIP events on the stream."""
        torch = self.torch
        lat = []
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev0.record(self.stream)
        for _ in range(steps):
            t = time.perf_counter()
            self.one()
            lat.append(time.perf_counter() - t)
        ev1.record(self.stream)
        torch.cuda.synchronize()
        return lat, time.perf_counter() - t0, ev0.elapsed_time(ev1)

    def kernels(self, steps: int) -> dict:
        """Mean duration of each kernel (HIP events on the library stream)."""
        self.pol.set_timing(True)
        acc: dict[str, list[float]] = {}
        for _ in range(steps):
            self.one()
            for name, ms in self.pol.timing():
                acc.setdefault(name, []).append(ms)
        self.pol.set_timing(False)
        return {k: statistics.mean(v) for k, v in acc.items()}

    def close(self):
        self.pol.close()


def roofline_of(kern: dict, p, R: int) -> dict:
    N, E, W, M = p.n_nodes, p.n_edges, p.n_workflows, p.n_instances
    grouped = not p.wf_contiguous
    dom = max((k for k in kern if alg_bytes(k, N, E, R, W, M, grouped) > 0), key=lambda k: kern[k])
    b = alg_bytes(dom, N, E, R, W, M, grouped)
    achieved = b / (kern[dom] * 1e-3) / 1e9
    return {"bound": "hbm", "kernel": dom, "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS, "traffic": None, "alg_bytes_per_launch": b,
            "launch_us": 1e3 * kern[dom]}


# ---------------------------------------------------------------- legs

def leg_headline(args):
    from paper_2601_05109_amd import nalar
    p = workload(args.workload)
    bits = {"least-slack": 0, "srtf": nalar.NALAR_ORDER_SRTF, "lpt": nalar.NALAR_ORDER_LPT,
            "stateful": nalar.NALAR_ROUTE_STATEFUL,
            "lpt+stateful": nalar.NALAR_ORDER_LPT | nalar.NALAR_ROUTE_STATEFUL,
            "greedy": nalar.NALAR_ROUTE_GREEDY,
            "greedy+stateful": nalar.NALAR_ROUTE_GREEDY | nalar.NALAR_ROUTE_STATEFUL}[args.policy]
    prio = None
    if args.priority_levels > 0:
        import numpy as np
        import torch
        lv = np.random.default_rng(7).integers(0, args.priority_levels, p.n_workflows).astype(np.uint8)
        prio = torch.from_numpy(lv).to("cuda")
    run = Runner(p, bits, prio)
    try:
        for _ in range(args.warmup):
            R = run.one()
        lat, wall, gpu_ms = run.timed(args.steps)
        cold = []
        if args.cold > 0:  # overwrite more than the L2 and the MALL before each pass
            torch = run.torch
            evict = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
            for _ in range(args.cold):
                evict.fill_(1)
                torch.cuda.synchronize()
                t = time.perf_counter()
                run.one()
                cold.append(time.perf_counter() - t)
            del evict
            torch.cuda.synchronize()
        kern = run.kernels(args.steps)
    finally:
        run.close()
    N, E, W, M = p.n_nodes, p.n_edges, p.n_workflows, p.n_instances
    ms_per_step = 1e3 * wall / args.steps
    t_dev_us = 1e3 * gpu_ms / args.steps
    b_pass = pass_alg_bytes(N, E, R, W, M)
    lat_us = [1e6 * x for x in lat]
    cold_us = [1e6 * x for x in cold]
    return {
        "metric": "futures/sec per global policy pass",
        "value": N / (ms_per_step * 1e-3),
        "unit": "futures/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic (seeded generator, paper-scale shape)",
        "config": {"workload": f"{p.name}: {W} workflows x {N // max(W, 1)} futures = {N} futures, "
                               f"{E} dependencies, {R} ready, K=8 types, {M} instances",
                   "n_futures": N, "n_ready": R, "policy": args.policy,
                   "priority_levels": args.priority_levels},
        "latency_us": {"p50": pct(lat_us, 0.5), "p99": pct(lat_us, 0.99), "min": min(lat_us),
                       "gpu_event_mean": t_dev_us},
        "cold_latency_us": ({"p50": pct(cold_us, 0.5), "max": max(cold_us), "passes": len(cold_us),
                             "evict_bytes": 512 << 20} if cold_us else None),
        "kernels_us": {k: round(1e3 * v, 2) for k, v in kern.items()},
        "roofline": roofline_of(kern, p, R),
        "pass_roofline": {"alg_bytes": b_pass, "device_us": t_dev_us,
                          "achieved": b_pass / (t_dev_us * 1e-6) / 1e9,
                          "frac": b_pass / (t_dev_us * 1e-6) / 1e9 / HBM_PEAK_GBS},
    }


def leg_first_pass(args, changes: int = 20):
    """Paper scale: the pass a controller makes once per changed snapshot.
    The handle first settles on the base snapshot; then each change (1 % of
    in-flight futures completed, or every deadline moved by up to 1 s,
    alternating, each from the base) is uploaded untimed and passed once,
    timed: that first pass plans its sort from the previous snapshot."""
    from paper_2601_05109_amd import workloads as wl
    base = workload("paper-scale")
    run = Runner(base)
    first, again = [], []
    try:
        for _ in range(args.warmup):
            run.one()
        for i in range(changes):
            q = wl.churned(base, 1000 + i) if i % 2 == 0 else wl.deadline_shifted(base, 2000 + i)
            run.swap(q)
            t = time.perf_counter()
            run.one()
            first.append(1e6 * (time.perf_counter() - t))
            t = time.perf_counter()
            run.one()
            again.append(1e6 * (time.perf_counter() - t))
    finally:
        run.close()
    return {"changes": changes, "kinds": "1% of in-flight futures completed / every deadline moved by up to 1 s",
            "first_pass_us": {"p50": pct(first, 0.5), "p99": pct(first, 0.99), "max": max(first)},
            "second_pass_us": {"p50": pct(again, 0.5), "p99": pct(again, 0.99)}}


def leg_wide(args):
    p = workload("wide-mapreduce")
    run = Runner(p)
    try:
        for _ in range(max(3, args.warmup)):
            R = run.one()
        lat, wall, gpu_ms = run.timed(args.steps)
        kern = run.kernels(min(args.steps, 20))
    finally:
        run.close()
    lat_us = [1e6 * x for x in lat]
    t_dev_us = 1e3 * gpu_ms / args.steps
    b_pass = pass_alg_bytes(p.n_nodes, p.n_edges, R, p.n_workflows, p.n_instances)
    return {"workload": f"{p.name}: {p.n_nodes} futures, {p.n_edges} dependencies, {R} ready, "
                        f"{p.n_instances} instances",
            "n_futures": p.n_nodes, "n_ready": R, "passes": args.steps,
            "futures_per_s": p.n_nodes / (wall / args.steps),
            "latency_us": {"p50": pct(lat_us, 0.5), "p99": pct(lat_us, 0.99), "gpu_event_mean": t_dev_us},
            "kernels_us": {k: round(1e3 * v, 2) for k, v in kern.items()},
            "roofline": roofline_of(kern, p, R),
            "pass_roofline": {"alg_bytes": b_pass, "device_us": t_dev_us,
                              "frac": b_pass / (t_dev_us * 1e-6) / 1e9 / HBM_PEAK_GBS}}


def run_dynamic(steps: int, reps: int, use_store: bool, log=None) -> dict:
    """The evolving map/reduce graph: each snapshot is uploaded (timed apart,
    not part of a pass), then passed once (the first pass over it, timed) and
    ``reps`` more times (median).  With ``use_store`` the snapshot reaches the
    device-resident graph store as the delta from the previous one, the
    passes are the store's incremental ones, and every 25 steps a full pass
    over the same store is timed beside them."""
    import numpy as np
    import torch
    from paper_2601_05109_amd import nalar, workloads as wl

    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
    pol = nalar.Policy(device=0, stream=stream)
    store = nalar.Store(pol) if use_store else None
    prev_n, prev_done, out = 0, None, None
    rows = []
    t_all = time.perf_counter()
    try:
        for step, p in enumerate(wl.dynamic_stream(steps=steps)):
            N = p.n_nodes
            t = time.perf_counter()
            if store is None:
                dp = nalar.DeviceProblem.from_host(p, dev)
                cp = dp.c_struct()
            else:
                if prev_n == 0:
                    store.set_workflows(p.deadline_us)
                    store.set_instances(p.inst_type, p.inst_load_us, p.inst_speed_permille)
                else:
                    store.complete(np.flatnonzero((p.done[:prev_n] == 1) & (prev_done == 0)).astype(np.int32))
                e0, e1 = int(p.dep_off[prev_n]), int(p.dep_off[N])
                rc = store.append(p.wf[prev_n:N], p.type[prev_n:N], p.est_us[prev_n:N], p.done[prev_n:N],
                                  p.loc[prev_n:N], p.dep_off[prev_n:N + 1] - e0, p.dep_idx[e0:e1],
                                  contiguous=bool(p.wf_contiguous))
                if rc != nalar.NALAR_OK:
                    raise RuntimeError(f"step {step}: append failed {rc}: {pol.last_error()}")
                prev_n, prev_done = N, p.done[:N].copy()
            torch.cuda.synchronize()
            up_ms = 1e3 * (time.perf_counter() - t)
            if out is None or out.order.shape[0] < N:
                out = nalar.DeviceResult.alloc(int(N * 1.3), dev)
            cr = out.c_struct()

            def one_pass():
                if store is None:
                    rc = nalar.nalar_policy_pass(pol.handle, cp, cr)
                else:
                    rc = nalar.nalar_store_pass(store.handle, p.now_us, p.migration_cost_us, 0, cr)
                if rc != nalar.NALAR_OK:
                    raise RuntimeError(f"step {step}: pass failed {rc}: {pol.last_error()}")
                return int(cr.n_ready)

            def timed_pass():
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                R = one_pass()
                e1.record(stream)
                e1.synchronize()
                return R, 1e3 * e0.elapsed_time(e1)

            R, first_us = timed_pass()
            inc = store.last_pass_incremental if store is not None else False
            reps_us = [timed_pass()[1] for _ in range(reps)]
            row = {"step": step, "n": N, "e": p.n_edges, "ready": R, "first_us": first_us,
                   "us": statistics.median(reps_us) if reps_us else first_us, "upload_ms": up_ms}
            if store is not None:
                row["incremental"] = inc
                if step % 25 == 0 and step > 0:  # a full pass over the same store, for comparison
                    store.set_incremental(False)
                    row["full_us"] = timed_pass()[1]
                    store.set_incremental(True)
            if step % 25 == 0:  # per-kernel events on the library stream
                pol.set_timing(True)
                one_pass()
                row["kernels_us"] = {}
                for name, ms in pol.timing():
                    row["kernels_us"][name] = round(row["kernels_us"].get(name, 0.0) + 1e3 * ms, 2)
                pol.set_timing(False)
            rows.append(row)
            if log and step % 10 == 0:
                log(f"dynamic step {step}: N={N} R={R} first {first_us:.1f} us, repeat {row['us']:.1f} us "
                    f"(upload {up_ms:.1f} ms)" + (f", incremental {row['incremental']}" if store else "")
                    + (f", full {row['full_us']:.1f} us" if "full_us" in row else ""))
    finally:
        if store is not None:
            store.close()
        pol.close()
    later = rows[1:] or rows
    firsts = [r["first_us"] for r in later]
    reps_ = [r["us"] for r in later]
    last = rows[-1]
    extra = {}
    if use_store:
        extra = {"passes": "incremental (the store recomputes the remaining path of the changed futures "
                           "and their ancestors only)",
                 "incremental_steps": sum(1 for r in later if r.get("incremental")),
                 "full_pass_us": {str(r["step"]): round(r["full_us"], 1) for r in rows if "full_us" in r}}
        if "full_us" in last:
            extra["step_last_full_over_incremental"] = round(last["full_us"] / last["first_us"], 2)
    return {"workload": f"dynamic-stream: {rows[0]['n']} -> {last['n']} futures over {len(rows) - 1} steps, "
                        "ids not workflow-contiguous after step 0",
            "input": "device-resident graph store fed by deltas" if use_store else "whole snapshot uploaded every step",
            "steps": len(rows) - 1,
            "first_pass_us": {"p50": pct(firsts, 0.5), "p99": pct(firsts, 0.99)},
            "repeat_pass_us": {"p50": pct(reps_, 0.5), "p99": pct(reps_, 0.99)},
            **extra,
            "step0_us": rows[0]["us"],
            "last_step": {k: last[k] for k in ("step", "n", "e", "ready", "first_us", "us", "full_us") if k in last},
            # per-kernel events of a pass repeated over the last snapshot (no change since the
            # pass before it: for the store, an empty closure)
            "last_step_repeat_kernels_us": next((r["kernels_us"] for r in reversed(rows) if "kernels_us" in r), None),
            "last_step_pass_roofline_frac": pass_alg_bytes(last["n"], last["e"], last["ready"], 256, 256)
            / (last["first_us"] * 1e-6) / 1e9 / HBM_PEAK_GBS,
            "last_step_repeat_pass_roofline_frac": pass_alg_bytes(last["n"], last["e"], last["ready"], 256, 256)
            / (last["us"] * 1e-6) / 1e9 / HBM_PEAK_GBS,
            "last_step_full_pass_roofline_frac": (pass_alg_bytes(last["n"], last["e"], last["ready"], 256, 256)
                                                  / (last["full_us"] * 1e-6) / 1e9 / HBM_PEAK_GBS)
            if "full_us" in last else None,
            "per_step": [{k: (round(v, 2) if isinstance(v, float) else v) for k, v in r.items()} for r in rows],
            "wall_s": time.perf_counter() - t_all}


def log_err(msg):
    print(msg, file=sys.stderr, flush=True)


# ---------------------------------------------------------------- HBM traffic

def traffic_probe(name: str) -> int:
    """Run under rocprofv3 --pmc by the parent: a few passes of one workload,
    then a plain device copy of 256 MiB (the calibration of the counters)."""
    import torch
    run = Runner(workload(name))
    try:
        for _ in range(8):
            run.one()
        torch.cuda.synchronize()
    finally:
        run.close()
    n = (256 << 20) // 4
    src = torch.arange(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print("probe done", flush=True)
    return 0


def _counter_means(outdir: str, counter: str, last: int = 5, reduce=None) -> dict:
    """Mean counter value (KiB) per dispatch over the last ``last`` dispatches
    of each kernel (the steady state: the probe's first pass plans its sort
    without a previous pass), by kernel name; with ``reduce`` (e.g. max), that
    function of every dispatch's value instead."""
    acc: dict[str, list[tuple[int, float]]] = {}
    for path in glob.glob(os.path.join(outdir, "**", "*counter_collection.csv"), recursive=True):
        with open(path, newline="") as fh:
            for row in csv.DictReader(fh):
                if row.get("Counter_Name") != counter:
                    continue
                acc.setdefault(row.get("Kernel_Name", ""), []).append(
                    (int(row.get("Dispatch_Id") or 0), float(row["Counter_Value"])))
    if reduce is not None:
        return {k: reduce(x for _, x in v) for k, v in acc.items()}
    return {k: statistics.mean(x for _, x in sorted(v)[-last:]) for k, v in acc.items()}


def measure_traffic(names_to_kernels: dict, timeout_s: int = 150) -> dict:
    """HBM bytes per launch of the given kernels, from two rocprofv3 --pmc
    child runs of this script's probe (FETCH_SIZE, then WRITE_SIZE), each
    counter scaled by its reading for a copy of known size."""
    prof = shutil.which("rocprofv3")
    if not prof:
        return {"error": "rocprofv3 not found"}
    copy_bytes = 256 << 20
    result = {}
    for workload_name, symbol in names_to_kernels.items():
        got = {}
        for counter in ("FETCH_SIZE", "WRITE_SIZE"):
            with tempfile.TemporaryDirectory(prefix="nalar_pmc_", dir="/tmp") as d:
                cmd = [prof, "--pmc", counter, "-d", d, "-o", "t", "--output-format", "csv", "--",
                       sys.executable, os.path.abspath(__file__), "--traffic-probe", workload_name]
                env = dict(os.environ, TMPDIR="/tmp")
                try:
                    subprocess.run(cmd, cwd="/tmp", env=env, timeout=timeout_s, capture_output=True)
                except subprocess.TimeoutExpired:
                    return {"error": f"rocprofv3 --pmc {counter} timed out"}
                means = _counter_means(d, counter)
                largest = _counter_means(d, counter, reduce=max)
            kern = [v for k, v in means.items() if symbol in k]
            # the calibration copy is the largest copyBuffer dispatch (uploads
            # of the snapshot dispatch small ones)
            cal = [v for k, v in largest.items() if "copyBuffer" in k]
            if not kern or not cal:
                return {"error": f"no {counter} rows for {symbol} or the copy"}
            got[counter] = (statistics.mean(kern), max(cal))
        f_kib, f_cal = got["FETCH_SIZE"]
        w_kib, w_cal = got["WRITE_SIZE"]
        f_scale = copy_bytes / (f_cal * 1024.0)
        w_scale = copy_bytes / (w_cal * 1024.0)
        result[workload_name] = {"kernel": symbol, "fetch_kib": f_kib, "write_kib": w_kib,
                                 "fetch_scale": f_scale, "write_scale": w_scale,
                                 "bytes_per_launch": f_kib * 1024.0 * f_scale + w_kib * 1024.0 * w_scale}
    return result


# ---------------------------------------------------------------- CPU baseline

def host_info() -> dict:
    model = platform.processor() or ""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        cxx = subprocess.run(["g++", "--version"], capture_output=True, text=True).stdout.splitlines()[0]
    except (OSError, IndexError):
        cxx = "g++"
    return {"cpu_model": model, "nproc": os.cpu_count(),
            "affinity_cpus": len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else None,
            "compiler": cxx}


def cpu_baseline(p, budget_s: float = 12.0) -> dict:
    """The oracle as it stands, single-threaded on this host, repeated on the
    same snapshot for about ``budget_s`` seconds."""
    import oracle
    oracle.build()
    info = host_info()
    saved = os.sched_getaffinity(0) if hasattr(os, "sched_getaffinity") else None
    try:
        if saved:
            os.sched_setaffinity(0, {sorted(saved)[0]})
        reps, t0 = 0, time.perf_counter()
        while True:
            r = oracle.run(p)
            reps += 1
            el = time.perf_counter() - t0
            if el >= budget_s:
                break
    finally:
        if saved:
            os.sched_setaffinity(0, saved)
    assert r.status == 0
    return {"value": p.n_nodes * reps / el, "unit": "futures/s", "cores": 1, "kind": "oracle",
            "sample": f"{reps} full passes of the oracle over the same {p.n_nodes}-future snapshot "
                      f"({el:.1f} s, one thread pinned to one core of {info['nproc']})",
            "ms_per_pass": 1e3 * el / reps, "host": info,
            "flags": " ".join(oracle.CXXFLAGS)}


# ---------------------------------------------------------------- levels

def levels(args) -> int:
    """One-level versus two-level control (the comparison of Table 4, Section
    6.3) over 1,024 ... 131,072 futures of the paper-scale generator.
    Two-level: one batched pass installs every ready future's priority and
    route at once (median of 100 synchronous passes).  One-level: the central
    controller decides every future event itself: a burst of N events (one per
    future of the snapshot), each decided by its own synchronous
    nalar_policy_decide call against the last pass's view, the k-th waiting for
    the k-1 before it.  Every figure is measured: the per-event latency (median
    call), the burst's completion time and the mean time an event waits for its
    decision."""
    import numpy as np
    import torch
    from paper_2601_05109_amd import nalar, workloads as wl

    dev = torch.device("cuda", 0)
    stream = torch.cuda.current_stream(dev)
    pol = nalar.Policy(device=0, stream=stream)
    rows = []
    try:
        W = 32
        while W * 32 <= 131072:
            p = wl.windowed(W)
            dp = nalar.DeviceProblem.from_host(p, dev)
            view = nalar.DeviceResult.alloc(p.n_nodes, dev)
            cp, cr = dp.c_struct(), view.c_struct()

            def one_pass():
                rc = nalar.nalar_policy_pass(pol.handle, cp, cr)
                if rc != nalar.NALAR_OK:
                    raise RuntimeError(f"pass failed {rc}: {pol.last_error()}")
                return int(cr.n_ready)

            for _ in range(10):
                R = one_pass()
            ts = []
            for _ in range(100):
                t = time.perf_counter()
                one_pass()
                ts.append(time.perf_counter() - t)
            view.n_ready = R
            N = p.n_nodes
            events = torch.from_numpy(np.arange(N, dtype=np.int32)).to(dev)
            cv = nalar.NalarView(rem_us=view.rem.data_ptr(), order=view.order.data_ptr(),
                                 slack_us=view.slack.data_ptr(), n_order=R)
            dec = nalar.DeviceDecisions.alloc(N, dev)
            # one event per call, in id order: the k-th completes at done[k]
            done_at = np.empty(N)
            base = events.data_ptr()
            outs = [nalar.NalarDecisions(slack_us=dec.slack.data_ptr() + 8 * k, route=dec.route.data_ptr() + 4 * k,
                                         cost_us=dec.cost.data_ptr() + 8 * k, rank=dec.rank.data_ptr() + 8 * k)
                    for k in range(N)]
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for k in range(N):
                rc = nalar.nalar_policy_decide(pol.handle, cp, cv, 1, base + 4 * k, outs[k])
                if rc != nalar.NALAR_OK:
                    raise RuntimeError(f"decide failed {rc}: {pol.last_error()}")
                done_at[k] = time.perf_counter() - t0
            burst = done_at[-1]
            per_event = np.median(np.diff(np.concatenate([[0.0], done_at])))
            # the same N decisions in one batched launch, for comparison
            t = time.perf_counter()
            assert nalar.nalar_policy_decide(pol.handle, cp, cv, N, base, dec.c_struct()) == nalar.NALAR_OK
            batched = time.perf_counter() - t
            t_us = 1e6 * statistics.median(ts)
            rows.append({"futures": N, "ready": R,
                         "two_level_pass_us": round(t_us, 2),
                         "two_level_per_future_ns": round(1e3 * t_us / N, 3),
                         "one_level_per_event_us": round(1e6 * per_event, 2),
                         "one_level_burst_ms": round(1e3 * burst, 2),
                         "one_level_mean_wait_ms": round(1e3 * float(done_at.mean()), 2),
                         "one_level_batched_decide_us": round(1e6 * batched, 2)})
            log_err(f"N={N}: pass {t_us:.1f} us, decide {1e6 * per_event:.1f} us/event, burst {1e3 * burst:.1f} ms")
            W *= 2
    finally:
        pol.close()
    res = {"metric": "schedule time, one-level vs two-level control", "unit": "us",
           "n_gpus": 1, "higher_is_better": False, "dtype": "int64",
           "data": "synthetic (seeded generator, paper-scale shape, 32 futures per workflow)",
           "config": {"workload": "futures sweep 1,024 ... 131,072"}, "rows": rows}
    print(json.dumps(res))
    return 0


# ---------------------------------------------------------------- main

def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="paper-scale")
    ap.add_argument("--policy", default="least-slack",
                    choices=["least-slack", "srtf", "lpt", "stateful", "lpt+stateful", "greedy", "greedy+stateful"],
                    help="order by least slack (default), least remaining work (srtf) or most (lpt); "
                         "stateful pins futures to the instance holding their state; greedy routes in "
                         "output order with running instance loads")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--cold", type=int, default=20,
                    help="passes timed after evicting the L2 and the MALL (0: skip)")
    ap.add_argument("--priority-levels", type=int, default=0,
                    help="give every workflow a seeded priority level in [0, L) (set_priority); 0 = none")
    ap.add_argument("--legs", default="all",
                    help="extra legs of the default run: all, none, or a comma list of "
                         "first_pass,wide_mapreduce,dynamic,traffic")
    ap.add_argument("--dyn-steps", type=int, default=100, help="dynamic workload: steps after step 0")
    ap.add_argument("--dyn-reps", type=int, default=3, help="dynamic workload: repeat passes per step")
    ap.add_argument("--store", action="store_true",
                    help="dynamic workload: feed the device-resident graph store by deltas")
    ap.add_argument("--traffic-probe", default=None, help=argparse.SUPPRESS)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the pass shards by "
              "workflow across GPUs by design but that path is not built", file=sys.stderr)
        return 2
    if args.traffic_probe:
        return traffic_probe(args.traffic_probe)
    if args.workload == "dynamic":
        res = run_dynamic(args.dyn_steps, args.dyn_reps, args.store, log_err)
        res.update({"metric": "pass latency per step, evolving graph", "unit": "us", "n_gpus": 1,
                    "higher_is_better": False, "dtype": "int64",
                    "data": "synthetic (seeded generator, evolving map/reduce graph)"})
        print(json.dumps(res))
        return 0
    if args.workload == "levels":
        return levels(args)

    res = leg_headline(args)
    legs = set() if args.legs == "none" else (
        {"first_pass", "wide_mapreduce", "dynamic", "traffic"} if args.legs == "all" else set(args.legs.split(",")))
    if args.workload != "paper-scale" or args.policy != "least-slack" or args.priority_levels:
        legs &= {"traffic"}
    if "first_pass" in legs:
        log_err("leg: first pass after a change (paper scale)")
        res["first_pass"] = leg_first_pass(args)
    if "wide_mapreduce" in legs:
        log_err("leg: wide map/reduce")
        res["wide_mapreduce"] = leg_wide(args)
    if "dynamic" in legs:
        log_err("leg: dynamic stream")
        dyn = run_dynamic(args.dyn_steps, args.dyn_reps, True, log_err)
        dyn.pop("per_step")
        if args.dyn_reps > 0:  # one pass per change, as a controller makes it (no repeats in between)
            log_err("leg: dynamic stream, one pass per change")
            one = run_dynamic(args.dyn_steps, 0, True, log_err)
            dyn["one_pass_per_change"] = {"first_pass_us": one["first_pass_us"],
                                          "incremental_steps": one["incremental_steps"],
                                          "last_step_first_us": one["last_step"]["first_us"],
                                          "full_pass_us": one.get("full_pass_us"), "wall_s": one["wall_s"]}
        res["dynamic"] = dyn
    if "traffic" in legs:
        log_err("leg: HBM traffic (rocprofv3 --pmc child runs)")
        want = {args.workload: KERNEL_SYMBOL.get(res["roofline"]["kernel"], res["roofline"]["kernel"])}
        if "wide_mapreduce" in res:
            k = res["wide_mapreduce"]["roofline"]["kernel"]
            want["wide-mapreduce"] = KERNEL_SYMBOL.get(k, k)
        tr = measure_traffic(want)
        res["traffic_measurement"] = tr
        for wname, target in ((args.workload, res["roofline"]),
                              ("wide-mapreduce", res.get("wide_mapreduce", {}).get("roofline"))):
            if target is not None and isinstance(tr.get(wname), dict):
                target["traffic"] = tr[wname]["bytes_per_launch"]
    if not args.no_cpu:
        log_err("leg: CPU oracle baseline")
        res["cpu_baseline"] = cpu_baseline(workload(args.workload), args.cpu_seconds)
    print(json.dumps(res))
    return 0


if __name__ == "__main__":
    sys.exit(main())
