#!/usr/bin/env python3
"""Throughput of the CCD++ sweep on one MI355X.

A step is one outer iteration of Algorithm 3 on the whole workload: all k
features, each with inner_iters u/v alternations and the fused residual
bookkeeping (one ccdpp_run(1, inner) call).  ccdpp_run leaves the last
feature's residual update pending for the next call's first passes; the timed
region ends with it (the final flush, with the training sum of squares), so K
timed steps do all the work of K outer iterations.  Inputs are resident in HBM
before timing.

  value    = 2 * inner * k * nnz / (seconds per step) / 1e9   [G nonzero visits / s]
  roofline = algorithmic bytes of the dominant kernel per launch / its mean
             duration (HIP events on the handle's stream, inside the timed
             region), against 8 TB/s HBM peak.  The algorithmic bytes follow
             the byte model of the sweep with 4-byte indices and row pointers:
             a plain pass reads index and value of every entry (8 B per entry
             in float), a first pass or flush also writes the value back
             (12 B), plus per pass the row pointers, the per-row factor
             scalars read, the coordinates written and one read of each
             gathered vector.  `frac` is that rate over the peak; `frac_hw`
             is the HBM traffic the hardware counters measured for the same
             kernel (profiles/traffic_*.json) over the same time and peak;
             `frac_stored` prices the bytes the compressed layout must move
             (16-bit or delta-coded indices), which is less than the model.
  cpu_baseline = the fp64 oracle on the host cores, on a bounded sample of
             features of the same matrix: once on one thread, once on all
             the threads the host gives this process

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
KERNEL_NAMES = {0: "ccd_pass_fused", 1: "ccd_pass", 2: "ccd_combine", 3: "ccd_copy", 4: "ccd_flush"}
LAYOUT_NAMES = {0: "rows", 1: "cols"}


def kernel_symbol(kind: int, info: dict, layout: int, wb_stores: bool = True) -> str:
    """The kernel's name as a trace shows it (the sweep kernels are templated on
    LDS staging, 16-bit indices, P == 1 and the value type).  A split item-major
    copy runs two kernels per pass, its tiled part's and its hot part's: "A + B"."""
    v = "double" if info.get("value_bytes", 4) == 8 else "float"
    if kind == 2:  # (4 lanes per row instead of 16 on layouts whose rows have few partials)
        return f"void ccdk::ccd_combine<16, {v}>(ccdk::CombineArgs<{v}>)"
    if kind == 3:
        return f"void ccdk::ccd_copy<{v}>({v} const*, {v}*, long)"
    if layout == 1 and info.get("v_split_rows", 0) > 0:
        hot = dict(info, v_gather=info["v2_gather"], v_tiles=1,
                   v_tile_width=info["v2_tile_width"], v_cache=info["v2_cache"], v_split_rows=0)
        return (kernel_symbol(kind, dict(info, v_split_rows=0), 1, wb_stores) + " + " +
                kernel_symbol(kind, hot, 1, wb_stores))
    pre = "u" if layout == 0 else "v"
    gather = info[f"{pre}_gather"]
    staged = gather in (2, 3)  # tiled, or hot (leading columns staged)
    idx16 = gather == 2 or (gather == 1 and info[f"{pre}_tile_width"] < 32768)
    p1 = info[f"{pre}_tiles"] == 1
    cache = info.get(f"{pre}_cache", 1) - 1  # 0 streaming, 1 write-back stores, 2 cached
    if cache == 1 and (kind == 1 or not wb_stores):
        # The plain pass stores no residual, and automatic write-back stores apply to
        # CCD++ with two or more inner iterations only: the streaming kernel.
        cache = 0
    name = KERNEL_NAMES[kind]
    b = lambda x: "true" if x else "false"
    return f"void ccdk::{name}<{b(staged)}, {b(idx16)}, {b(p1)}, {cache}, {v}>(ccdk::PassArgs<{v}>)"


# Vectors a pass gathers, per (kind, copy): the plain pass its update vector; the first
# pass of a feature over the user-major copy h_t and h_(t-1) (u's update vector is h_t),
# over the item-major copy u, w_t and w_(t-1); the flush the previous feature's vector.
GATHERED = {(0, 0): 2, (0, 1): 3, (1, 0): 1, (1, 1): 1, (4, 0): 1, (4, 1): 1}


def model_bytes(kind: int, layout: int, info: dict) -> float | None:
    """Bytes of one pass (kind 0 first pass, 1 plain pass, 4 flush) over one residual
    copy under the sweep's byte model: 4-byte indices and row pointers, values,
    factor entries and coordinates of the value type."""
    if (kind, layout) not in GATHERED:
        return None
    vb = info.get("value_bytes", 4)
    nnz = info["nnz"]
    rows, cols = (info["m"], info["n"]) if layout == 0 else (info["n"], info["m"])
    b = (4 + vb) * nnz + 4 * (rows + 1)            # index and value read, row pointers
    if kind in (0, 4):
        b += vb * nnz                               # the residual written back
    if kind in (0, 1):
        b += vb * rows                              # the coordinates written
    b += vb * rows * (2 if kind == 0 else 1 if kind == 4 else 0)  # per-row factor scalars
    b += vb * cols * GATHERED[(kind, layout)]        # each gathered vector, once
    return float(b)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def source_digest() -> str:
    h = hashlib.sha256()
    for f in ("sweep.hip", "ccdpp_internal.hpp", "api.hip"):
        with open(os.path.join(ROOT, "paper_1511_02433_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def stored_traffic(key: str, workload: str, precision: str = "f32"):
    """HBM bytes per launch of kernel `key` ("ccd_pass/cols", ...) from the committed
    rocprofv3 counter summary, if it was taken on the current kernel source; else None."""
    suffix = "" if precision == "f32" else f"_{precision}"
    p = os.path.join(ROOT, "profiles", f"traffic_{workload}{suffix}.json")
    if not os.path.exists(p):
        return None
    with open(p) as f:
        t = json.load(f)
    if t.get("source_digest") != source_digest():
        return None
    k = t.get("kernels", {}).get(key)
    return None if k is None else k.get("bytes_per_launch")


def host_threads() -> dict:
    """What the host offers this process: all logical CPUs, the ones this process may
    run on, the thread count the environment sets for OpenMP, and the CPU model."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        affinity = os.cpu_count() or 1
    omp = os.environ.get("OMP_NUM_THREADS", "")
    use = affinity
    if omp.isdigit() and int(omp) > 0:
        use = min(use, int(omp))
    return {"cores_all": os.cpu_count(), "affinity": affinity, "omp_num_threads": omp or None,
            "threads": use, "cpu_model": model}


def cpu_baseline(ds, k, inner, budget_s, algorithm="ccdpp"):
    """The oracle, as it stands, on a bounded sample of the workload: feature updates
    in Algorithm 3's order, first on one thread (about a third of the budget), then
    on every thread the host gives this process (the rest).  `value` is the latter."""
    from oracle import Oracle

    w = ds.workload
    host = host_threads()
    threads = host["threads"]
    log(f"cpu baseline: building the oracle on {w.name}; host {host}")
    o = Oracle(w.m, w.n, k, w.lam, ds.row, ds.col, ds.val, ds.h0(k), threads=threads)
    out = {"unit": "Gnnz/s", "cores": threads, "kind": "oracle", **host}
    if algorithm == "ccd":
        # One whole outer iteration of Algorithm 2 (it cannot be cut per feature).
        t0 = time.perf_counter()
        o.ccd_run(1)
        dt = time.perf_counter() - t0
        o.close()
        log(f"cpu baseline: one element-wise CCD outer iteration in {dt:.2f}s")
        v = 2.0 * k * w.nnz / dt / 1e9
        out.update(value=v, value_all=v, value_1t=None,
                   sample=f"one outer iteration of element-wise CCD on the full {w.name} "
                          f"matrix, fp64 oracle, {threads} threads, {dt:.1f} s")
        return out

    # Feature updates in Algorithm 3's order (features 0..k-1, then the next outer
    # iteration) until the budget of each leg is spent.
    def leg(nthreads, budget, start, cap):
        o.set_threads(nthreads)
        done = 0
        t0 = time.perf_counter()
        while done < cap:
            o.rank((start + done) % k, inner, debug=False)
            done += 1
            if time.perf_counter() - t0 >= budget:
                break
        return done, time.perf_counter() - t0

    n1, dt1 = leg(1, budget_s / 3.0, 0, k)
    log(f"cpu baseline: 1 thread, {n1} feature updates x {inner} inner in {dt1:.2f}s")
    na, dta = leg(threads, budget_s - dt1, n1, 3 * k)
    log(f"cpu baseline: {threads} threads, {na} feature updates x {inner} inner in {dta:.2f}s")
    o.close()
    v1 = 2.0 * inner * w.nnz * n1 / dt1 / 1e9
    va = 2.0 * inner * w.nnz * na / dta / 1e9
    out.update(value=va, value_all=va, value_1t=v1,
               sample=f"feature updates in Algorithm 3's order on the full {w.name} matrix "
                      f"(k {k}, inner {inner}), fp64 oracle: features 0..{n1 - 1} on 1 thread "
                      f"({dt1:.1f} s), then the next {na} ({na / k:.2f} outer iterations) on "
                      f"{threads} threads ({dta:.1f} s)")
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="large", choices=["tiny", "medium", "large", "vlarge"])
    ap.add_argument("--k", type=int, default=0, help="override the number of features")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-prof", action="store_true", help="time without per-kernel events")
    ap.add_argument("--event-every", type=int, default=5,
                    help="bracket every n-th launch of the dominant kernel with HIP events")
    ap.add_argument("--algorithm", default="ccdpp", choices=["ccdpp", "ccd"],
                    help="ccdpp: Algorithm 3 (the headline); ccd: element-wise CCD, Algorithm 2")
    ap.add_argument("--precision", default="f32", choices=["f32", "f64"],
                    help="value type of the residual, factors and sweep arithmetic")
    ap.add_argument("--no-open-loop", action="store_true",
                    help="skip the open-loop (run until converged) measurement")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only copy a MIB-MiB device buffer 3 times (a kernel of known HBM "
                         "traffic, to scale hardware byte counters) and exit")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1511_02433_amd import synth
    from paper_1511_02433_amd.ccdpp import CCDPP

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        nel = args.copy_calibration * (1 << 20) // 4
        x = torch.ones(nel, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        log(f"copied {args.copy_calibration} MiB three times")
        return
    # The HIP runtime sets up its queues on the first work a process sends to the device
    # (about 0.15 s on MI355X).  That happens here, timed on its own, so that
    # device_build_ms times the library's build only.
    t_init = time.perf_counter()
    torch.empty(8 << 20, dtype=torch.uint8).to("cuda").add_(1)
    torch.cuda.synchronize()
    runtime_init_ms = (time.perf_counter() - t_init) * 1e3
    ds = synth.load(args.workload, verbose=True)
    w = ds.workload
    k = args.k or w.k
    inner = w.inner
    log(f"workload {w.describe()} (k={k})")

    from paper_1511_02433_amd.ccdpp import make_options
    g = CCDPP(w.m, w.n, k, w.lam, ds.row, ds.col, ds.val,
              opts=make_options(precision=1 if args.precision == "f64" else 0))
    g.use_torch_stream()
    g.set_factors(np.zeros((w.m, k), np.float32), ds.h0(k))
    info = g.info()
    log(f"device build {info['build_us'] / 1e3:.1f} ms; schedule {info}")

    wb_stores = args.algorithm == "ccdpp" and inner >= 2

    def read_kernels():
        """Per-kernel and per-(kernel, residual copy) timings collected since profile()."""
        kinds, per_layout = {}, {}
        for kind, name in KERNEL_NAMES.items():
            n, tot, b = g.profile_read(kind)
            if n:
                kinds[name] = {"launches": n, "mean_us": tot / n * 1e3, "total_ms": tot,
                               "algo_bytes_per_launch": b / n, "gbs": b / (tot * 1e-3) / 1e9}
            for lay, lname in LAYOUT_NAMES.items():
                n2, t2, b2 = g.profile_read(kind, lay)
                if n2:
                    mb = model_bytes(kind, lay, info)
                    per_layout[f"{name}/{lname}"] = {
                        "kernel": kernel_symbol(kind, info, lay, wb_stores), "kind": kind,
                        "layout": lay,
                        "launches": n2, "mean_us": round(t2 / n2 * 1e3, 3),
                        "total_ms": round(t2, 4), "model_bytes_per_launch": mb,
                        "model_gbs": None if mb is None else round(mb / (t2 / n2 * 1e-3) / 1e9, 1),
                        "stored_bytes_per_launch": b2 / n2,
                        "stored_gbs": round(b2 / (t2 * 1e-3) / 1e9, 1)}
        return kinds, per_layout

    def step():
        if args.algorithm == "ccd":
            g.ccd_run(1)
        else:
            g.run(1, inner)

    def timed(steps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            step()
        g.train_rmse()  # the pending residual update of the last feature, and sum R^2
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / steps

    # Warmup.  The last warmup step times every kernel, which names the dominant one.
    kinds, per_layout = {}, {}
    kinds_steps = 1
    for i in range(args.warmup):
        last = i + 1 == args.warmup and not args.no_prof
        if last:
            g.profile(True)
        step()
        if last:
            g.train_rmse()  # the flush, so that the kernel table shows it once per step
            torch.cuda.synchronize()
            kinds, per_layout = read_kernels()
    torch.cuda.synchronize()
    dom = max(per_layout, key=lambda kk: per_layout[kk]["total_ms"]) if per_layout else None

    # The timed region: exactly `steps` steps.  HIP events on the handle's stream
    # bracket every `event_every`-th launch of the dominant kernel (every launch of
    # every kernel without warmup).
    prof = not args.no_prof
    if prof:
        g.profile(True)
        if dom:
            g.profile_only(per_layout[dom]["kind"], per_layout[dom]["layout"])
            g.profile_every(args.event_every)
    ms = timed(args.steps)
    if prof:
        if dom:
            d = per_layout[dom]
            n, tot, b = g.profile_read(d["kind"], d["layout"])
            live = {"launches": n, "mean_us": round(tot / n * 1e3, 3), "total_ms": round(tot, 4),
                    "stored_bytes_per_launch": b / n}
        else:
            kinds, per_layout = read_kernels()
            kinds_steps = args.steps
            dom = max(per_layout, key=lambda kk: per_layout[kk]["total_ms"])
            live = per_layout[dom]
        g.profile_only(-1, -1)
        g.profile_every(1)
        g.profile(False)
    ms_plain = timed(max(2, args.steps // 2)) if prof else ms
    # Nonzero visits per step: CCD++ visits every entry 2 * inner times per feature;
    # element-wise CCD visits it once per feature in each of its two phases.
    visits = (2.0 if args.algorithm == "ccd" else 2.0 * inner) * k * w.nnz
    value = visits / (ms * 1e-3) / 1e9
    log(f"{ms:.3f} ms/step (events on the dominant kernel), {ms_plain:.3f} ms/step without; "
        f"{value:.1f} Gnnz/s")

    # Roofline of the dominant kernel: the (kernel, residual copy) pair with the most
    # device time per step, timed live in the timed region.
    roofline = None
    if prof and dom:
        d = per_layout[dom]
        sec = live["mean_us"] * 1e-6
        mb = d["model_bytes_per_launch"]
        achieved = mb / sec / 1e9
        stored = live["stored_bytes_per_launch"] / sec / 1e9
        traffic = stored_traffic(dom, w.name, args.precision)
        roofline = {"kernel": d["kernel"], "layout": dom.split("/")[1], "bound": "hbm",
                    "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": traffic,
                    "frac_hw": None if traffic is None
                    else round(traffic / sec / 1e9 / HBM_PEAK_GBS, 4),
                    "frac_stored": round(stored / HBM_PEAK_GBS, 4),
                    "mean_us": live["mean_us"], "launches": live["launches"],
                    "algo_bytes_per_launch": mb,
                    "stored_bytes_per_launch": live["stored_bytes_per_launch"]}
    train_rmse = g.train_rmse()
    test_rmse = g.rmse(ds.test_row, ds.test_col, ds.test_val) if ds.test_row.size else None
    # The open outer loop with monitoring: three more outer iterations, each followed by
    # the objective of eq. 1 and the training and held-out RMSE (the held-out triplets
    # are copied to the device once per call, inside this time).
    open_loop = None
    if not args.no_open_loop and args.algorithm == "ccdpp":
        test = (ds.test_row, ds.test_col, ds.test_val) if ds.test_row.size else None
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        done, hist = g.run_until(3, inner, -1.0, test)
        torch.cuda.synchronize()
        per = (time.perf_counter() - t0) * 1e3 / max(done, 1)
        open_loop = {"outer": done, "ms_per_outer": round(per, 3),
                     "monitor_ms_per_outer": round(per - ms_plain, 3),
                     "objective": float(hist[-1, 0]), "train_rmse": float(hist[-1, 1]),
                     "test_rmse": None if test is None else float(hist[-1, 2])}
        log(f"open loop: {per:.3f} ms per outer iteration with monitoring "
            f"({per - ms_plain:+.3f} ms against the plain step)")
    step_bytes = sum(v["algo_bytes_per_launch"] * v["launches"] for v in kinds.values()) / kinds_steps \
        if kinds else None
    # The byte model over the passes of a step (the combine and commit kernels move
    # O(m + n) bytes and are not part of it).
    step_model = sum(v["model_bytes_per_launch"] * v["launches"] for v in per_layout.values()
                     if v["model_bytes_per_launch"]) / kinds_steps if per_layout else None
    g.close()

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(synth.load(args.workload), k, inner, args.cpu_budget, args.algorithm)

    out = {
        "metric": "CCD++ nonzeros/sec (G/s) + achieved HBM GB/s vs peak; s per outer iter",
        "value": round(value, 3),
        "unit": "Gnnz/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "s_per_outer_iter": round(ms * 1e-3, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.precision,
        "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.m}x{w.n}, nnz={w.nnz}, k={k}, lambda={w.lam}, "
                               + (f"inner={inner}; step = 1 outer iteration" if args.algorithm == "ccdpp"
                                  else "element-wise CCD (Algorithm 2); step = 1 outer iteration"),
                   "m": w.m, "n": w.n, "nnz": w.nnz, "k": k, "inner_iters": inner,
                   "algorithm": args.algorithm},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "model_bytes_per_step": step_model,
        "model_gbs": round(step_model / (ms * 1e-3) / 1e9, 1) if step_model else None,
        "stored_bytes_per_step": step_bytes,
        "stored_gbs": round(step_bytes / (ms * 1e-3) / 1e9, 1) if step_bytes else None,
        "ms_per_step_without_kernel_events": round(ms_plain, 4),
        "kernels_note": ("per-kernel timings: the last warmup step" if kinds_steps == 1
                         else "per-kernel timings: the timed steps"),
        "kernels": kinds,
        "kernels_by_layout": per_layout,
        "train_rmse": train_rmse,
        "test_rmse": test_rmse,
        "device_build_ms": info["build_us"] / 1e3,
        "runtime_init_ms": round(runtime_init_ms, 1),
        "open_loop": open_loop,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
