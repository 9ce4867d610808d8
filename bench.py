"""Benchmark of the MI355X transposition library (Eq. 1 of the HPTT paper).

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step is one execution of the plan (all of the hot path: the plan is
built once, then each step launches the kernel the plan chose) on inputs
already resident in HBM.  Steps cycle through enough buffer sets that no
launch finds its tensors in the 256 MB last-level cache, and before its warm-up
each workload's buffers are swept with reads for 30 ms so that the GPU's
clocks have settled after the host's idle gap (settle()).  The headline workload is the largest
one: the 5-D fp32 transposition of A(3, 2, 640, 480, 96) with perm [4, 2, 0, 3, 1] and
alpha = beta = 1 (B read and written, the paper's default reporting mode, Eq. 2
with lambda = 3); the other named workloads are reported in ``per_workload``,
each with its own roofline block, and the 57-case sweep's distribution in
``per_sweep``.

Bandwidth follows Eq. (2) of the paper: lambda * S bytes per transposition
(S = bytes of one tensor, lambda = 2 when beta = 0, 3 otherwise), reported in
GB/s (1e9 B/s).  Context printed on the same line:
  - roofline: the dominant kernel's achieved GB/s over MI355X's 8 TB/s HBM
    peak, from one HIP event pair around the timed launches (on the launch
    stream), plus the HBM bytes rocprofv3 counted for it when a matching
    counter summary is committed;
  - yardsticks: a same-run 16-byte-per-lane copy kernel (2S) and, for
    beta != 0, an axpby kernel (3S) -- the SAXPY yardstick of Table 2 --
    and hipMemcpyAsync device-to-device;
  - cold: the paper's protocol (Section 4), best and median of single
    launches with the caches cleared in between;
  - cpu_baseline: the CPU oracle on this machine's host, single-threaded, with
    the host's logical CPU count and CPU model.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, AMD published peak
HEADLINE = "transpose5d_3x2x640x480x96_f32"
PROFILE_DIR = os.path.join(ROOT, "profiles")
FLUSH_BYTES = 1 << 30           # > 256 MB last-level cache + 8 x 4 MB L2
ROTATE_BYTES = 2 << 30          # traffic between two uses of one buffer set


def kernel_source_hash() -> str:
    """Hash of the sources that decide what the transposition kernels do."""
    h = hashlib.sha256()
    for f in ("kernel_body.h", "kernels.hip", "plan.cpp", "hptt_args.h", "device_mem.h",
              "tile_kernel.h", "tile_f32_fast.hip", "tile_f32_shifted.hip", "tile_f32_general.hip",
              "tile_shared.hip", "tile_direct.hip", "tile_f64.hip"):
        with open(os.path.join(ROOT, "paper_1704_04374_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def kernel_label(kernel_class: str) -> str:
    """Name of the __global__ function that runs a plan's kernel class."""
    return f"{kernel_class}_kernel"


def profile_path(kernel_class: str, workload: str, kind: str) -> str:
    return os.path.join(PROFILE_DIR, f"{kernel_label(kernel_class)}_{workload}_{kind}.txt")


def load_traffic(kernel_class: str, workload: str):
    """HBM bytes per launch from a committed rocprofv3 counter summary, or
    None when there is none or the kernels changed since it was taken."""
    path = profile_path(kernel_class, workload, "pmc")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_source_hash") != kernel_source_hash():
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def roofline_block(achieved_gbs: float, kernel_class: str, w) -> dict:
    """Roofline of one workload's transposition kernel: achieved GB/s (Eq. 2
    bytes over the kernel's average launch time) against the HBM peak, and the
    HBM bytes per launch that a committed counter summary gives, if any."""
    traffic = load_traffic(kernel_class, w.name)
    return {"bound": "hbm", "achieved": round(achieved_gbs, 1), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(achieved_gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
            "algorithmic_bytes": w.moved_bytes,
            "traffic_over_algorithmic": (None if traffic is None
                                         else round(traffic / w.moved_bytes, 4))}


def _events(torch, n):
    return [torch.cuda.Event(enable_timing=True) for _ in range(n)]


def time_launches(torch, fn, steps: int, warmup: int, dist: bool = True):
    """Run fn(i) for i < warmup, then `steps` more back to back between a
    synchronize on each side: the timed region, with one HIP event pair on
    the launch stream around all of it.  Returns (wall seconds of the
    region, its GPU milliseconds per launch -- each launch's duration plus
    the gap the GPU leaves before the next dependent one, which agrees with
    rocprofv3's kernel trace).  Then `steps` more launches, each between its
    own event pair, give the distribution (time_launches.last); they stay
    out of the timed region, where each event record would add a gap; with
    dist=False they are skipped."""
    for i in range(warmup):
        fn(i)
    torch.cuda.synchronize()
    region = _events(torch, 2)
    t0 = time.perf_counter()
    region[0].record()
    for i in range(steps):
        fn(warmup + i)
    region[1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_launch = region[0].elapsed_time(region[1]) / steps
    if not dist:
        return wall, per_launch
    starts, ends = _events(torch, steps), _events(torch, steps)
    for i in range(steps):
        starts[i].record()
        fn(warmup + steps + i)
        ends[i].record()
    torch.cuda.synchronize()
    ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    time_launches.last = sorted(ms)
    return wall, per_launch


def time_cold(torch, hptt, fn, flush_buf, sink, reps: int):
    """Single launches, each after a read-only sweep of 1 GiB that leaves the
    caches holding only clean, unrelated lines ("caches are cleared in between
    runs", Section 4)."""
    ms = []
    for i in range(reps):
        hptt.yardstick_read(flush_buf, flush_buf.numel() * 4, sink)
        s, e = _events(torch, 2)
        s.record()
        fn(i)
        e.record()
        torch.cuda.synchronize()
        ms.append(s.elapsed_time(e))
    return ms


def preheat(torch, hptt, seconds: float = 0.3):
    """Untimed streaming fills until the GPU has run for `seconds`: launch
    times fall by about 10 % over the first few hundred milliseconds of work
    as the clocks settle, which would otherwise bias the first workload.  (A
    fill, not the copy kernel, so that profiles of the copy kernel contain
    only the measured copies.)"""
    buf = torch.empty(1 << 27, dtype=torch.float32, device="cuda")
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for _ in range(10):
            hptt.yardstick_fill(buf, buf.numel() * 4, 0)
        torch.cuda.synchronize()
    del buf
    torch.cuda.empty_cache()


SETTLE_S = 0.03


def settle(torch, hptt, bufs, sink, seconds: float = SETTLE_S):
    """Read-only sweeps over the workload's own buffers for `seconds` right
    before its timed launches.  After an idle gap (the host allocating and
    planning), the first ~10 ms of HBM-bound work run several percent slow
    while the GPU's clocks settle (MI355X: the 6-D fp32 workload 4.72-4.95
    TB/s over 5 + 20 launches straight after 0.3 s idle, 5.27 after this
    settle; 100 untimed launches of the kernel itself reached 5.09).  Reads
    leave the tensors' values unchanged."""
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < seconds:
        for b in bufs:
            hptt.yardstick_read(b, b.numel() * b.element_size() // 16 * 16, sink)
        torch.cuda.synchronize()


def rotation(w) -> int:
    """Buffer sets cycled through by back-to-back steps, so that at least
    ROTATE_BYTES of other traffic separate two uses of the same tensors and no
    launch finds its inputs in the 256 MB last-level cache."""
    per_set = 2 * w.tensor_bytes
    return max(2, min(8, -(-ROTATE_BYTES // per_set)))


def measure_workload(torch, hptt, w, steps, warmup, reps, flush_buf, sink, full: bool,
                     tune_s: float = 0.0):
    """Time one workload: the transposition and its same-run yardsticks, all
    over the same rotating buffer sets."""
    tdt = torch.float32 if w.dtype == "f32" else torch.float64
    gen = torch.Generator(device="cuda").manual_seed(w.seed_a)
    k = rotation(w)
    # enclosing tensors; A and B below are the sub-tensors' first elements
    PA = [torch.rand(w.parent_numel_a, dtype=tdt, device="cuda", generator=gen) * 2 - 1
          for _ in range(k)]
    PB = [torch.rand(w.parent_numel_b, dtype=tdt, device="cuda", generator=gen) * 2 - 1
          for _ in range(k)]
    As = [x[w.offset_a:] for x in PA]
    Bs = [x[w.offset_b:] for x in PB]
    t0 = time.perf_counter()
    plan = hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype, outer_size_a=w.outer_a,
                            outer_size_b=w.outer_b, **dict(w.knobs))
    plan_us = (time.perf_counter() - t0) * 1e6
    moved = w.moved_bytes
    S = w.tensor_bytes
    out = {"workload": w.name, "plan": plan.describe(), "plan_create_us": round(plan_us, 1),
           "bytes_per_launch": moved, "buffer_sets": k, "kernel_class": plan.info["kernel"]}

    stream = torch.cuda.current_stream().cuda_stream
    runs = [plan.launcher(As[j].data_ptr(), Bs[j].data_ptr(), stream) for j in range(k)]

    def transpose(i):
        runs[i % k]()

    # the yardsticks move 16-byte vectors: time them on S rounded down to 16 B
    S16 = S // 16 * 16
    n16 = S16 // w.elem_bytes

    def copy(i):
        hptt.yardstick_copy(As[i % k], Bs[i % k], S16)

    def memcpy(i):
        Bs[i % k][:w.numel].copy_(As[i % k][:w.numel])

    def axpby(i):
        hptt.yardstick_axpby(w.dtype, w.alpha, As[i % k], w.beta, Bs[i % k], n16)

    def gbs(nbytes, ms):
        return nbytes / (ms * 1e-3) / 1e9

    settle(torch, hptt, PA + PB, sink)
    wall, ms = time_launches(torch, transpose, steps, warmup)
    dist = time_launches.last
    # mean: the timed region's GPU time per launch; min / median / max: one
    # event pair per launch after the region (each pair adds ~2 us)
    out["kernel_us"] = {"mean": round(ms * 1e3, 2), "event_min": round(dist[0] * 1e3, 2),
                        "event_median": round(dist[len(dist) // 2] * 1e3, 2),
                        "event_max": round(dist[-1] * 1e3, 2)}
    out["ms_per_step"] = wall * 1e3 / steps
    out["gbs"] = moved * steps / wall / 1e9
    out["kernel_avg_ms"] = ms
    out["kernel_gbs"] = gbs(moved, ms)
    # the yardstick is the faster of two timings: a single one was seen far
    # below the rest when the GPU was briefly disturbed, which inflates every
    # ratio taken against it
    out["copy_gbs"] = max(gbs(2 * S16, time_launches(torch, copy, steps, warmup)[1])
                          for _ in range(2))
    out["hipmemcpy_d2d_gbs"] = gbs(2 * S, time_launches(torch, memcpy, steps, warmup)[1])
    if w.beta != 0:
        out["axpby_gbs"] = gbs(3 * S16, time_launches(torch, axpby, steps, warmup)[1])
        out["pct_of_axpby"] = 100 * out["kernel_gbs"] / out["axpby_gbs"]
    out["pct_of_copy"] = 100 * out["kernel_gbs"] / out["copy_gbs"]
    out["pct_of_hbm_peak"] = 100 * out["kernel_gbs"] / HBM_PEAK_GBS
    if full:
        fms = time_cold(torch, hptt, transpose, flush_buf, sink, reps)
        cfs = time_cold(torch, hptt, copy, flush_buf, sink, reps)
        out["cold"] = {
            "reps": reps,
            "median_gbs": moved / (statistics.median(fms) * 1e-3) / 1e9,
            "best_gbs": moved / (min(fms) * 1e-3) / 1e9,
            "best_gibs_eq2": moved / (min(fms) * 1e-3) / 2 ** 30,
            "copy_median_gbs": 2 * S16 / (statistics.median(cfs) * 1e-3) / 1e9,
        }
        out["cold"]["median_pct_of_copy"] = (100 * out["cold"]["median_gbs"]
                                             / out["cold"]["copy_median_gbs"])
    if tune_s > 0:
        # the autotune path (Section 3.1), timed like the quick path's plan
        t0 = time.perf_counter()
        tuned, rep = hptt.autotune_plan(w.perm, w.size_a, As[0], Bs[0], w.alpha, w.beta,
                                        w.dtype, timeout=tune_s, outer_size_a=w.outer_a,
                                        outer_size_b=w.outer_b)
        tune_wall = time.perf_counter() - t0
        same = tuned.describe() == plan.describe()
        if same:
            # the quick path's own plan: nothing to compare but noise
            qms = tms = ms
        else:
            # both plans in alternating rounds, so that clock drift between
            # two separate timings does not pass for a speedup
            truns = [tuned.launcher(As[j].data_ptr(), Bs[j].data_ptr(), stream)
                     for j in range(k)]
            qs, ts = [], []
            for r in range(5):
                pair = [(runs, qs), (truns, ts)]
                for rs, acc in (pair if r % 2 == 0 else pair[::-1]):
                    acc.append(time_launches(torch, lambda i, rs=rs: rs[i % k](), steps, warmup,
                                             dist=False)[1])
            qms, tms = statistics.median(qs), statistics.median(ts)
        out["autotune"] = {
            "seconds": round(tune_wall, 2), "candidates": rep["candidates"],
            "timed": rep["timed"], "finalists": rep["finalists"], "confirmed": rep["confirmed"],
            "plan": tuned.describe(), "same_plan_as_quick": same,
            "knobs": {n: v for n, v in rep["options"].items() if v},
            "kernel_gbs": round(gbs(moved, tms), 1),
            "speedup_vs_quick": round(qms / tms, 3),
        }
    del As, Bs, PA, PB
    torch.cuda.empty_cache()
    return out


def host_description() -> dict:
    """The host the CPU baseline ran on: logical CPUs, the CPUs this process
    may use, and the CPU model."""
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
    except (AttributeError, OSError):
        usable = os.cpu_count()
    return {"host_logical_cpus": os.cpu_count(), "host_usable_cpus": usable,
            "host_cpu_model": model}


def cpu_baseline(w, budget_s: float = 12.0):
    """The oracle, as it stands, on this host: repeated whole transpositions
    of the headline workload until about budget_s seconds have passed, on one
    thread (the oracle is a single-threaded loop)."""
    from oracle import oracle
    from paper_1704_04374_amd.workloads import inputs
    A, B0 = inputs(w)
    a = A.numpy()
    b = None if B0 is None else B0.numpy()
    runs, t0 = 0, time.perf_counter()
    while True:
        oracle.transpose(a, w.size_a, w.perm, w.alpha, w.beta, b)
        runs += 1
        el = time.perf_counter() - t0
        if el >= budget_s or runs >= 50:
            break
    out = {"value": round(w.moved_bytes * runs / el / 1e9, 3), "unit": "GB/s",
           "cores": 1, "kind": "oracle",
           "sample": f"{runs} whole transpositions of {w.name} "
                     f"({w.numel} elements each, {el:.1f} s, single thread)"}
    out.update(host_description())
    return out


def summarize_pmc(fetch_dir: str, write_dir: str, workload: str, command: str, out_path: str):
    """Turn two rocprofv3 --pmc runs (FETCH_SIZE, then WRITE_SIZE) into the
    committed summary that load_traffic() reads.  Counters are KiB per
    dispatch; both are scaled by what they read for the copy yardstick of
    known size in the same runs."""
    import csv

    from paper_1704_04374_amd.workloads import BY_NAME

    def per_kernel(d, counter):
        rows = []
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(path) as f:
                rows += [r for r in csv.DictReader(f) if r.get("Counter_Name") == counter]
        acc = {}
        for r in rows:
            acc.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
        return acc

    w = BY_NAME[workload]
    fetch = per_kernel(fetch_dir, "FETCH_SIZE")
    write = per_kernel(write_dir, "WRITE_SIZE")

    def pick(acc, key):
        names = [n for n in acc if key in n]
        if not names:
            raise SystemExit(f"no dispatch of a kernel matching {key!r} in the counter files")
        vals = acc[names[0]]
        return names[0], statistics.median(vals)

    from paper_1704_04374_amd import hptt
    cls = hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype,
                           **dict(w.knobs)).info["kernel"]
    tk, tf = pick(fetch, kernel_label(cls))
    _, tw = pick(write, tk.split("(")[0])
    _, cf = pick(fetch, "copy_kernel")
    _, cw = pick(write, "copy_kernel")
    S = w.tensor_bytes
    f_scale = S / (cf * 1024)    # copy kernel reads exactly S bytes
    w_scale = S / (cw * 1024)    # and writes exactly S bytes
    fetch_b = tf * 1024 * f_scale
    write_b = tw * 1024 * w_scale
    lines = [
        f"# rocprofv3 counter summary: {tk}",
        f"# workload: {w.describe()}",
        f"# command (FETCH_SIZE pass): {command.replace('COUNTER', 'FETCH_SIZE')}",
        f"# command (WRITE_SIZE pass): {command.replace('COUNTER', 'WRITE_SIZE')}",
        "# FETCH_SIZE and WRITE_SIZE are KiB per dispatch (median over dispatches); each is",
        "# scaled by (known bytes / counter) of the copy yardstick kernel in the same run.",
        f"kernel: {tk}",
        f"fetch_kib_per_dispatch: {tf:.1f}",
        f"write_kib_per_dispatch: {tw:.1f}",
        f"copy_fetch_kib_per_dispatch: {cf:.1f}",
        f"copy_write_kib_per_dispatch: {cw:.1f}",
        f"copy_bytes_each_way: {S}",
        f"fetch_scale: {f_scale:.4f}",
        f"write_scale: {w_scale:.4f}",
        f"hbm_fetch_bytes_per_launch: {fetch_b:.0f}",
        f"hbm_write_bytes_per_launch: {write_b:.0f}",
        f"hbm_bytes_per_launch: {fetch_b + write_b:.0f}",
        f"algorithmic_bytes_per_launch: {w.moved_bytes}",
        f"traffic_over_algorithmic: {(fetch_b + write_b) / w.moved_bytes:.4f}",
        f"kernel_source_hash: {kernel_source_hash()}",
    ]
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_counters(dirs, workload: str, command: str, out_path: str):
    """Turn rocprofv3 --pmc runs (one per counter group) into a committed
    summary: the median per dispatch of every counter collected, for the
    workload's transposition kernel and for the same-run copy yardstick."""
    import csv

    from paper_1704_04374_amd.workloads import BY_NAME
    w = BY_NAME[workload]
    acc = {}
    for d in dirs:
        for path in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            with open(path) as f:
                for r in csv.DictReader(f):
                    name = r["Kernel_Name"]
                    kind = ("transposition" if ("tile_kernel" in name or "stream_kernel" in name
                                                or "axpby_kernel<" in name)
                            else "copy" if "copy_kernel" in name else None)
                    if kind:
                        acc.setdefault((kind, r["Counter_Name"]), []).append(
                            float(r["Counter_Value"]))
    if not acc:
        raise SystemExit("no transposition or copy dispatches in the counter files")
    lines = [f"# rocprofv3 counters, workload {w.describe()}",
             f"# command (one run per counter group): {command}",
             f"# algorithmic bytes per transposition (Eq. 2, lambda*S): {w.moved_bytes}",
             "# kernel | counter | median per dispatch | dispatches"]
    for (kind, counter), vals in sorted(acc.items()):
        lines.append(f"{kind} | {counter} | {statistics.median(vals):.1f} | {len(vals)}")
    lines.append(f"kernel_source_hash: {kernel_source_hash()}")
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_trace(trace_dir: str, workload: str, command: str, out_path: str):
    """Turn a rocprofv3 --kernel-trace --stats run into the committed summary:
    per-kernel calls and durations, and the headline kernel's GB/s from its
    average duration and the algorithmic bytes of Eq. (2)."""
    import csv

    from paper_1704_04374_amd.workloads import BY_NAME
    w = BY_NAME[workload]
    paths = glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not paths:
        raise SystemExit(f"no kernel_stats.csv under {trace_dir}")
    with open(paths[0]) as f:
        rows = list(csv.DictReader(f))
    lines = [f"# rocprofv3 kernel statistics, workload {w.describe()}",
             f"# command: {command}",
             f"# algorithmic bytes per transposition (Eq. 2, lambda*S): {w.moved_bytes}",
             "# kernel | calls | average us | min us | max us | GB/s at the average"]
    for r in rows:
        name = r["Name"]
        avg = float(r["AverageNs"])
        nb = None
        if "tile_kernel" in name or "stream_kernel" in name or "axpby_kernel<" in name:
            nb = w.moved_bytes
        elif "copy_kernel" in name:
            nb = 2 * w.tensor_bytes
        short = name if len(name) < 110 else name[:107] + "..."
        gbs = f"{nb / avg:.1f}" if nb else "-"
        lines.append(f"{short} | {r['Calls']} | {avg / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                     f"{float(r['MaxNs']) / 1e3:.2f} | {gbs}")
    lines.append(f"kernel_source_hash: {kernel_source_hash()}")
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def sweep_summary(torch, hptt, steps: int, warmup: int, sink) -> dict:
    """The 57-case sweep (Section 4's benchmark shape, Figs. 6 and 7) on the
    quick path, timed like the named workloads but lean: per case one
    rotation of device buffers, then back-to-back launches of the beta = 1
    plan, the same-run axpby yardstick (the paper's SAXPY), the alpha = 1,
    beta = 0 plan and the same-run copy yardstick.  Returns the distribution
    of % of axpby (beta = 1) and % of copy (beta = 0) with one row per case."""
    from paper_1704_04374_amd.workloads import sweep57
    rows = []
    t_start = time.perf_counter()
    for w in sweep57(beta=1.0):
        k = rotation(w)
        gen = torch.Generator(device="cuda").manual_seed(w.seed_a)
        As = [torch.rand(w.numel, device="cuda", generator=gen) * 2 - 1 for _ in range(k)]
        Bs = [torch.rand(w.numel, device="cuda", generator=gen) * 2 - 1 for _ in range(k)]
        stream = torch.cuda.current_stream().cuda_stream
        p1 = hptt.create_plan(w.perm, w.size_a, w.alpha, w.beta, w.dtype)
        p0 = hptt.create_plan(w.perm, w.size_a, 1.0, 0.0, w.dtype)
        r1 = [p1.launcher(As[j].data_ptr(), Bs[j].data_ptr(), stream) for j in range(k)]
        r0 = [p0.launcher(As[j].data_ptr(), Bs[j].data_ptr(), stream) for j in range(k)]
        settle(torch, hptt, As + Bs, sink)
        S = w.tensor_bytes
        S16 = S // 16 * 16
        ms1 = time_launches(torch, lambda i: r1[i % k](), steps, warmup, dist=False)[1]
        # each yardstick is the faster of two timings (a lone timing was once
        # 15x slow when the GPU was briefly disturbed)
        msx = min(time_launches(torch, lambda i: hptt.yardstick_axpby(
            w.dtype, w.alpha, As[i % k], w.beta, Bs[i % k], S16 // 4), steps, warmup,
            dist=False)[1] for _ in range(2))
        ms0 = time_launches(torch, lambda i: r0[i % k](), steps, warmup, dist=False)[1]
        msc = min(time_launches(torch, lambda i: hptt.yardstick_copy(As[i % k], Bs[i % k], S16),
                                steps, warmup, dist=False)[1] for _ in range(2))
        g1, g0 = 3 * S / ms1 / 1e6, 2 * S / ms0 / 1e6
        row = {"case": w.name, "kernel": p1.info["kernel"], "gbs": round(g1, 1),
               "pct_of_axpby": round(100 * g1 / (3 * S16 / msx / 1e6), 1),
               "beta0_gbs": round(g0, 1),
               "beta0_pct_of_copy": round(100 * g0 / (2 * S16 / msc / 1e6), 1)}
        rows.append(row)
        print(f"[sweep] {w.name}: {row['kernel']} {row['gbs']:.0f} GB/s = "
              f"{row['pct_of_axpby']:.1f}% of axpby; beta=0 {row['beta0_gbs']:.0f} GB/s = "
              f"{row['beta0_pct_of_copy']:.1f}% of copy", file=sys.stderr, flush=True)
        del As, Bs, r1, r0, p1, p0
        torch.cuda.empty_cache()

    def stats(key):
        v = [r[key] for r in rows]
        return {"mean": round(statistics.mean(v), 2), "median": round(statistics.median(v), 2),
                "min": round(min(v), 2), "max": round(max(v), 2)}
    return {"sweep": "57 seeded fp32 transpositions, 2-D to 6-D, 200 MB per tensor, quick path",
            "steps": steps, "warmup": warmup, "seconds": round(time.perf_counter() - t_start, 1),
            "pct_of_axpby": stats("pct_of_axpby"), "gbs": stats("gbs"),
            "beta0_pct_of_copy": stats("beta0_pct_of_copy"), "beta0_gbs": stats("beta0_gbs"),
            "cases_below_60_pct_of_axpby": sum(r["pct_of_axpby"] < 60 for r in rows),
            "cases": rows}


def run_sweep(torch, hptt, args, flush_buf, sink) -> dict:
    """The 57-case sweep (Section 4, Figs. 6 and 7): every case with beta != 0
    against the same-run axpby yardstick (the paper's SAXPY), with and
    without autotuning, and again with beta = 0 against the copy yardstick."""
    from dataclasses import replace

    from paper_1704_04374_amd.workloads import sweep57
    cases = []
    for w in sweep57(beta=1.0):
        r = measure_workload(torch, hptt, w, args.steps, args.warmup, 0, flush_buf, sink,
                             full=False, tune_s=args.autotune)
        w0 = replace(w, name=w.name, beta=0.0, seed_b=None)
        r0 = measure_workload(torch, hptt, w0, args.steps, args.warmup, 0, flush_buf, sink,
                              full=False)
        c = {"case": w.name, "kernel": r["kernel_class"], "plan": r["plan"],
             "gbs": round(r["kernel_gbs"], 1), "pct_of_axpby": round(r["pct_of_axpby"], 1),
             "pct_of_hbm_peak": round(r["pct_of_hbm_peak"], 1),
             "beta0_gbs": round(r0["kernel_gbs"], 1), "beta0_pct_of_copy": round(r0["pct_of_copy"], 1)}
        if "autotune" in r:
            c["tuned_gbs"] = r["autotune"]["kernel_gbs"]
            c["tuned_speedup"] = r["autotune"]["speedup_vs_quick"]
            c["tuned_knobs"] = r["autotune"]["knobs"]
        cases.append(c)
        print(f"[sweep] {w.name}: {c['kernel']} {c['gbs']:.0f} GB/s = {c['pct_of_axpby']:.1f}% of "
              f"axpby; beta=0 {c['beta0_pct_of_copy']:.1f}% of copy"
              + (f"; tuned x{c['tuned_speedup']:.3f}" if "tuned_speedup" in c else ""),
              file=sys.stderr, flush=True)

    def stats(key):
        v = [c[key] for c in cases if key in c]
        return {"mean": round(statistics.mean(v), 3), "median": round(statistics.median(v), 3),
                "min": round(min(v), 3), "max": round(max(v), 3)} if v else None
    return {"sweep": "57 seeded fp32 transpositions, 2-D to 6-D, 200 MB per tensor",
            "steps": args.steps, "warmup": args.warmup, "autotune_seconds": args.autotune,
            "pct_of_axpby": stats("pct_of_axpby"), "beta0_pct_of_copy": stats("beta0_pct_of_copy"),
            "pct_of_hbm_peak": stats("pct_of_hbm_peak"), "tuned_speedup": stats("tuned_speedup"),
            "kernels": {k: sum(c["kernel"] == k for c in cases) for k in
                        sorted(set(c["kernel"] for c in cases))},
            "cases": cases}


def run_contractions(torch, args) -> dict:
    """Contractions by transposition - GEMM - transposition against
    torch.einsum on the same tensors (the speedup of Eq. 3, with einsum in
    the role of the framework without this library's transpositions)."""
    from paper_1704_04374_amd.contraction import Contraction
    from paper_1704_04374_amd.workloads import CONTRACTIONS
    tdt = {"f32": torch.float32, "f64": torch.float64}
    out = []
    for w in CONTRACTIONS:
        gen = torch.Generator(device="cuda").manual_seed(w.seed + 1)
        A = torch.rand(w.numel(w.modes_a), dtype=tdt[w.dtype], device="cuda", generator=gen)
        B = torch.rand(w.numel(w.modes_b), dtype=tdt[w.dtype], device="cuda", generator=gen)
        C = torch.zeros(w.numel(w.modes_c), dtype=tdt[w.dtype], device="cuda")
        t0 = time.perf_counter()
        p = Contraction(w.modes_c, w.modes_a, w.size(w.modes_a), w.modes_b, w.size(w.modes_b),
                        w.alpha, w.beta, w.dtype)
        plan_us = (time.perf_counter() - t0) * 1e6
        p.workspace()
        # torch's view of a Fortran tensor: the same memory, modes reversed
        ta = A.view(*reversed(w.size(w.modes_a)))
        tb = B.view(*reversed(w.size(w.modes_b)))
        eq = f"{w.modes_a[::-1]},{w.modes_b[::-1]}->{w.modes_c[::-1]}"

        def ours(i):
            p.exec(A, B, C)

        def theirs(i):
            torch.einsum(eq, ta, tb).contiguous()

        steps = max(5, args.steps // 10)
        ms_ours = time_launches(torch, ours, steps, 3)[1]
        ms_theirs = time_launches(torch, theirs, steps, 3)[1]
        info = p.info
        r = {"contraction": w.name, "spec": w.spec, "dtype": w.dtype, "plan": p.describe(),
             "plan_create_us": round(plan_us, 1), "ms": round(ms_ours, 4),
             "einsum_ms": round(ms_theirs, 4), "speedup_vs_einsum": round(ms_theirs / ms_ours, 3),
             "tflops": round(info["flops"] / ms_ours / 1e9, 2),
             "einsum_tflops": round(info["flops"] / ms_theirs / 1e9, 2),
             "transposed_bytes": int(info["bytes_transposed"])}
        out.append(r)
        print(f"[contract] {w.name}: {r['ms']:.3f} ms ({r['tflops']} TFLOP/s) vs einsum "
              f"{r['einsum_ms']:.3f} ms: x{r['speedup_vs_einsum']}", file=sys.stderr, flush=True)
        del A, B, C, p
        torch.cuda.empty_cache()
    sp = [r["speedup_vs_einsum"] for r in out]
    return {"contractions": out, "speedup_vs_einsum": {
        "mean": round(statistics.mean(sp), 3), "max": max(sp), "min": min(sp)}}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=HEADLINE)
    ap.add_argument("--reps", type=int, default=20, help="flushed single launches per workload")
    ap.add_argument("--only-headline", action="store_true",
                    help="time only the headline workload (for profiler runs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep-summary", action="store_true",
                    help="skip the 57-case sweep summary of the default run")
    ap.add_argument("--autotune", type=float, default=2.0, metavar="SECONDS",
                    help="also tune each named workload for this long (0: skip)")
    ap.add_argument("--sweep", action="store_true",
                    help="run the 57-case sweep instead and print its summary as JSON")
    ap.add_argument("--contractions", action="store_true",
                    help="time the contraction workloads against torch.einsum instead")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"))
    ap.add_argument("--summarize-trace", metavar="TRACE_DIR")
    ap.add_argument("--summarize-counters", nargs="+", metavar="PMC_DIR")
    ap.add_argument("--pmc-command", default="")
    ap.add_argument("--pmc-out", default="")
    args = ap.parse_args()

    if args.summarize_pmc or args.summarize_trace or args.summarize_counters:
        from paper_1704_04374_amd.workloads import BY_NAME as _W
        _w = _W[args.workload]
        import ctypes  # noqa: F401  (plan creation needs only the host half of the library)
        from paper_1704_04374_amd import hptt as _h
        _cls = _h.create_plan(_w.perm, _w.size_a, _w.alpha, _w.beta, _w.dtype,
                              **dict(_w.knobs)).info["kernel"]
    if args.summarize_pmc:
        out = args.pmc_out or profile_path(_cls, args.workload, "pmc")
        summarize_pmc(*args.summarize_pmc, args.workload, args.pmc_command, out)
        return 0
    if args.summarize_trace:
        out = args.pmc_out or profile_path(_cls, args.workload, "trace")
        summarize_trace(args.summarize_trace, args.workload, args.pmc_command, out)
        return 0
    if args.summarize_counters:
        out = args.pmc_out or profile_path(_cls, args.workload, "counters")
        summarize_counters(args.summarize_counters, args.workload, args.pmc_command, out)
        return 0
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: this transposition library has no multi-GPU "
              "path (use --gpus 1)", file=sys.stderr)
        return 2

    import torch

    from paper_1704_04374_amd import hptt
    from paper_1704_04374_amd.workloads import BY_NAME, SUBTENSOR_WORKLOADS, WORKLOADS

    if not os.path.exists(hptt.LIB_PATH):
        from paper_1704_04374_amd import build
        build.build()
    torch.cuda.set_device(0)
    head = BY_NAME[args.workload]
    flush_buf = torch.zeros(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
    sink = torch.zeros(4096, dtype=torch.int32, device="cuda")
    print(f"[bench] device {torch.cuda.get_device_name(0)}; headline {head.describe()}",
          file=sys.stderr, flush=True)

    # load every kernel's code object now: the first dispatch from a code
    # object not yet loaded leaves the next few milliseconds of kernels
    # several percent slower, which would land on the first workload timed
    hptt.load_kernels()
    preheat(torch, hptt)
    if args.sweep:
        print(json.dumps(run_sweep(torch, hptt, args, flush_buf, sink)), flush=True)
        return 0
    if args.contractions:
        print(json.dumps(run_contractions(torch, args)), flush=True)
        return 0
    headline = measure_workload(torch, hptt, head, args.steps, args.warmup, args.reps, flush_buf,
                                sink, full=not args.only_headline,
                                tune_s=0.0 if args.only_headline else args.autotune)
    print(f"[bench] {head.name}: {headline['gbs']:.0f} GB/s, {headline['pct_of_copy']:.1f}% "
          f"of copy", file=sys.stderr, flush=True)
    per = {}
    if not args.only_headline:
        for w in WORKLOADS + SUBTENSOR_WORKLOADS:
            r = headline if w.name == head.name else measure_workload(
                torch, hptt, w, args.steps, args.warmup, args.reps, flush_buf, sink, full=True,
                tune_s=args.autotune)
            per[w.name] = {k: (round(v, 2) if isinstance(v, float) else v) for k, v in r.items()}
            per[w.name]["roofline"] = roofline_block(r["kernel_gbs"], r["kernel_class"], w)
            tuned = r.get("autotune")
            print(f"[bench] {w.name}: kernel {r['kernel_gbs']:.0f} GB/s, "
                  f"{r['pct_of_copy']:.1f}% of copy, {r['pct_of_hbm_peak']:.1f}% of peak"
                  + (f"; autotuned {tuned['kernel_gbs']:.0f} GB/s ({tuned['timed']} of "
                     f"{tuned['candidates']} plans timed)" if tuned else ""),
                  file=sys.stderr, flush=True)

    roof = roofline_block(headline["kernel_gbs"], headline["kernel_class"], head)
    per_sweep = None
    if not args.only_headline and not args.no_sweep_summary:
        per_sweep = sweep_summary(torch, hptt, min(args.steps, 20), min(args.warmup, 5), sink)
        print(f"[bench] sweep: {per_sweep['pct_of_axpby']['mean']:.1f}% of axpby on average "
              f"(min {per_sweep['pct_of_axpby']['min']:.1f}), beta=0 "
              f"{per_sweep['beta0_pct_of_copy']['mean']:.1f}% of copy, "
              f"{per_sweep['seconds']:.0f} s", file=sys.stderr, flush=True)
    line = {
        "metric": "effective GB/s per transpose (Eq. 2 bytes) and % of HBM peak / same-run copy",
        "value": round(headline["gbs"], 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(headline["ms_per_step"], 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head.dtype,
        "data": "synthetic: seeded uniform [-1,1) tensors resident in HBM",
        "config": {"workload": head.name, "dtype": head.dtype, "size_a": list(head.size_a),
                   "perm": list(head.perm), "alpha": head.alpha, "beta": head.beta,
                   "bytes_per_step": head.moved_bytes},
        "roofline": roof,
        "pct_of_copy": round(headline["pct_of_copy"], 2),
        "copy_gbs": round(headline["copy_gbs"], 1),
        "hipmemcpy_d2d_gbs": round(headline["hipmemcpy_d2d_gbs"], 1),
        "buffer_sets": headline["buffer_sets"],
        "kernel_us": headline["kernel_us"],
        "cold": headline.get("cold"),
        "plan": headline["plan"],
        "plan_create_us": headline["plan_create_us"],
        "kernel_source_hash": kernel_source_hash(),
        "settle_s": SETTLE_S,
        "per_workload": per or None,
        "per_sweep": per_sweep,
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(head)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
