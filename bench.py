#!/usr/bin/env python3
"""Benchmark: batched exemplar-clustering evaluation on one MI355X.

One step = one call of the library on one batch: exemplar_eval (gather and
norms of the exemplars, the fused contraction/min/sum kernel, the fixed-order
second pass) for eval workloads, exemplar_gain (cache + scoring) for greedy
workloads.  Inputs are synthetic, seeded, and resident in HBM before timing
starts.  Prints one JSON line on stdout; progress goes to stderr.

Default workload (the largest single-GPU configuration): 1 000 000 points of
a 100-Gaussian mixture in d = 256, stored as fp16 (fp32 accumulate), 2 048
sets of 32 exemplars.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import platform
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2101_08763_amd import api, synth  # noqa: E402

METRIC = "set evaluations/s and distance terms/s (n·k·l) + % of MFMA/HBM peak"
COPY_PROBE_BYTES = 1 << 30   # plain device copy used to calibrate the HBM byte counters
PROFILES = os.path.join(ROOT, "profiles")
PEAK_TFLOPS = {"fp32": 157.3, "fp16": 2516.6, "bf16": 2516.6}  # dense MFMA, MI355X
HBM_PEAK_GBS = 8000.0  # HBM3E, MI355X
DTYPE_NAME = {"fp32": "f32", "fp16": "f16", "bf16": "bf16"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# Default warm-up and timed lengths.  The GPU's clock governor needs a few
# hundred milliseconds of back-to-back work to settle: kernels timed in the
# first 10-100 calls after idle run up to 10 % slower than under sustained
# load.  So unless --warmup is given, the warm-up runs untimed steps for
# WARMUP_SECONDS (at least MIN_WARMUP steps), and unless --steps is given the
# timed region runs at least MIN_STEPS steps and TIMED_SECONDS.  Explicit
# values are used exactly.
WARMUP_SECONDS = 1.0
MIN_WARMUP = 10
TIMED_SECONDS = 0.5
MIN_STEPS = 50
PROF_SAMPLES = 100   # launches of the dominant kernel timed with HIP events per run


def warm_up(step, warmup, sync, seconds=None):
    """Run the untimed warm-up; return (steps run, seconds per step)."""
    seconds = WARMUP_SECONDS if seconds is None else seconds
    sync()
    t0 = time.perf_counter()
    if warmup is not None:
        for _ in range(warmup):
            step()
        sync()
        return warmup, (time.perf_counter() - t0) / max(warmup, 1)
    n, batch = 0, 1
    while True:
        for _ in range(batch):
            step()
        n += batch
        sync()
        el = time.perf_counter() - t0
        if el >= seconds and n >= MIN_WARMUP:
            return n, el / n
        # about 20 ms of work between synchronisations
        batch = max(1, min(1000, int(0.02 / max(el / n, 1e-7))))


def timed_steps(steps, sec_per_step, min_steps=MIN_STEPS):
    if steps is not None:
        return steps
    return max(min_steps, int(TIMED_SECONDS / max(sec_per_step, 1e-7)) + 1)


def cpu_model() -> str:
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or "unknown"


def cpu_baseline(p: synth.Problem, X64: np.ndarray, budget_s: float):
    """The oracle, as it stands, on the host cores, over a bounded sample of
    the same workload (all sets when they fit in the budget)."""
    import oracle

    o = oracle.load()
    w = p.workload
    threads = o.threads(0)
    if w.mode == "gain":
        probe = p.cands[:1]
        t0 = time.perf_counter()
        o.gain(X64, p.S, probe, threads)
        per = time.perf_counter() - t0
        m = int(max(1, min(len(p.cands), budget_s / max(per, 1e-9))))
        idx = np.unique((np.arange(m) * (len(p.cands) - 1)) // max(m - 1, 1))
        t0 = time.perf_counter()
        o.gain(X64, p.S, p.cands[idx], threads)
        dt = time.perf_counter() - t0
        kk = w.k + 1
    else:
        probe = p.sets[:min(len(p.sets), threads)]
        t0 = time.perf_counter()
        o.eval(X64, probe, threads)
        per = (time.perf_counter() - t0) / len(probe)
        m = int(max(1, min(len(p.sets), budget_s / max(per, 1e-9))))
        idx = np.unique((np.arange(m) * (len(p.sets) - 1)) // max(m - 1, 1))
        # Whole batches are repeated until the budget is used, for a stable rate.
        passes = 0
        t0 = time.perf_counter()
        while True:
            o.eval(X64, p.sets[idx], threads)
            passes += 1
            dt = time.perf_counter() - t0
            if dt >= 0.5 * budget_s or len(idx) < w.l:
                break
        kk = w.k
    m = len(idx) * (passes if w.mode == "eval" else 1)
    sample = ("all sets" if len(idx) == w.l else f"strided sample of {len(idx)} of {w.l} sets")
    if w.mode == "eval" and passes > 1:
        sample += f", {passes} passes"
    return {
        "value": m / dt, "unit": "set evaluations/s", "cores": threads, "kind": "oracle",
        "sample": f"{sample}, fp64 direct evaluation, OpenMP over sets, {threads} threads on {cpu_model()}",
        "seconds": dt, "distance_terms_per_s": w.n * kk * m / dt,
    }


# Files that define each kernel and its launch geometry (host glue such as
# host.cpp, the second pass and the greedy kernels do not change what the
# traffic counters of the kernel read); the compiler flags are hashed too.
KERNEL_FILES = {
    "eval_mfma_kernel": ["device.hpp", "internal.h", "kernels_mfma.hip", "kernels_mfma_bf16.hip",
                         "kernels_mfma_f16.hip", "kernels_mfma_f32.hip", "mfma_kernels.hpp"],
    "eval_bigd_kernel": ["bigd_kernels.hpp", "device.hpp", "internal.h", "kernels_mfma.hip", "kernels_mfma_bigd.hip"],
    "eval_valu_kernel": ["device.hpp", "internal.h", "kernels_aux.hip"],
    "sqnorm_kernel": ["device.hpp", "internal.h", "kernels_sqnorm.hip"],
}


def kernel_source_hash(kernel: str = "eval_mfma_kernel") -> str:
    """Hash of everything that defines the compiled kernel: its sources and
    the compiler flags (without the machine-dependent include paths)."""
    from paper_2101_08763_amd import build as B
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2101_08763_amd", "csrc")
    for f in KERNEL_FILES[kernel]:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode())
            h.update(fh.read())
    flags = [x for x in B.FLAGS if not x.startswith("-I")]
    if kernel in ("eval_mfma_kernel", "eval_bigd_kernel"):
        flags += B.MFMA_FLAGS
    h.update(" ".join([B.ARCH] + flags).encode())
    return h.hexdigest()


def traffic_file(kernel: str, workload: str) -> str:
    return os.path.join(PROFILES, f"{kernel}__{workload}.traffic.json")


def load_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the committed counter runs, or None when the
    kernel sources changed since they were taken (or none were taken)."""
    path = traffic_file(kernel, workload)
    if not os.path.exists(path):
        return None
    t = json.load(open(path))
    if t.get("source_sha256") != kernel_source_hash(kernel):
        return None
    return t["hbm_bytes_per_launch"]


def _pmc_values(run_dir: str, counter: str, name_re: str):
    import re
    vals = []
    for f in glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True):
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] == counter and re.search(name_re, r["Kernel_Name"]):
                vals.append(float(r["Counter_Value"]))
    return vals


def traffic_summary(d: str, kernel: str, workload: str) -> dict:
    """Turn four rocprofv3 --pmc runs under d/ (fetch, write: the workload;
    copy_fetch, copy_write: --copy-probe) into the committed traffic file."""
    kf = _pmc_values(os.path.join(d, "fetch"), "FETCH_SIZE", kernel)
    kw = _pmc_values(os.path.join(d, "write"), "WRITE_SIZE", kernel)
    cf = _pmc_values(os.path.join(d, "copy_fetch"), "FETCH_SIZE", "copyBuffer")
    cw = _pmc_values(os.path.join(d, "copy_write"), "WRITE_SIZE", "copyBuffer")
    if not (kf and kw and cf and cw):
        raise SystemExit(f"missing counter data under {d}")
    fetch_kib, write_kib = statistics.median(kf), statistics.median(kw)
    cfetch_kib, cwrite_kib = statistics.median(cf), statistics.median(cw)
    ff = COPY_PROBE_BYTES / (cfetch_kib * 1024)
    wf = COPY_PROBE_BYTES / (cwrite_kib * 1024)
    out = {
        "kernel": kernel, "workload": workload, "source_sha256": kernel_source_hash(kernel),
        "fetch_kib_per_dispatch": fetch_kib, "write_kib_per_dispatch": write_kib,
        "copy_probe_bytes": COPY_PROBE_BYTES, "copy_fetch_kib": cfetch_kib, "copy_write_kib": cwrite_kib,
        "fetch_scale": ff, "write_scale": wf,
        "hbm_bytes_per_launch": fetch_kib * 1024 * ff + write_kib * 1024 * wf,
        "dispatches": {"fetch": len(kf), "write": len(kw), "copy_fetch": len(cf), "copy_write": len(cw)},
    }
    os.makedirs(PROFILES, exist_ok=True)
    with open(traffic_file(kernel, workload), "w") as fh:
        json.dump(out, fh, indent=1)
    return out


def copy_probe(steps: int):
    """A plain device-to-device copy of COPY_PROBE_BYTES (calibration target
    for FETCH_SIZE / WRITE_SIZE)."""
    import torch
    n = COPY_PROBE_BYTES // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(steps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": COPY_PROBE_BYTES, "launches": steps}))


def run_paper_sweep(args, dev):
    """The three series of Section V-A (d = 100; n, l or k varied over 15
    values with the others at 50 000 / 5 000 / 10), each point timed as
    --sweep-reps separate exemplar_eval calls (median, min, max), next to the
    oracle's rate on the host.  One JSON line per (point, precision) on
    stdout and in --sweep-out; a Markdown table on stderr at the end."""
    import torch

    axes = ["n", "l", "k"] if args.sweep == "all" else args.sweep.split(",")
    precs = args.sweep_precisions.split(",")
    pts = [(a, pt) for a in axes for pt in synth.paper_sweep(a)]
    log(f"paper sweep: {len(pts)} points x {precs}; drawing {max(pt['n'] for _, pt in pts)} points")
    Xbig = synth.paper_sweep_points(max(pt["n"] for _, pt in pts))
    stream = torch.cuda.current_stream()
    sink = open(args.sweep_out, "w") if args.sweep_out else None
    table = []
    for axis, pt in pts:
        n, l, k = pt["n"], pt["l"], pt["k"]
        p = synth.paper_sweep_problem(n, l, k, X=Xbig)
        sets = torch.from_numpy(p.sets).to(dev)
        cpu = None
        if not args.no_cpu_baseline:
            cpu = cpu_baseline(p, p.X.astype(np.float64), args.sweep_cpu_budget)
        for prec in precs:
            Xs, _ = synth.rounded(p.X, prec)
            V = (Xs if isinstance(Xs, torch.Tensor) else torch.from_numpy(Xs)).to(dev).contiguous()
            out = torch.empty(l, dtype=torch.float32, device=dev)
            # the host-side oracle run leaves the GPU idle: let the clocks settle again
            warm_up(lambda: api.exemplar_eval(V, sets, out=out), None, torch.cuda.synchronize,
                    seconds=args.sweep_warmup_seconds)
            api.exemplar_prof_read()
            api.exemplar_prof_enable(True)
            evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                   for _ in range(args.sweep_reps)]
            for a, b in evs:
                a.record(stream)
                api.exemplar_eval(V, sets, out=out)
                b.record(stream)
            torch.cuda.synchronize()
            api.exemplar_prof_enable(False)
            kern_ms, launches = api.exemplar_prof_read()
            times = [a.elapsed_time(b) for a, b in evs]
            med = statistics.median(times)
            kern = kern_ms / max(launches, 1)
            flops = 2.0 * n * l * k * synth.PAPER_SWEEP_D
            rec = {
                "series": axis, "n": n, "l": l, "k": k, "d": synth.PAPER_SWEEP_D, "precision": prec,
                "reps": args.sweep_reps, "ms_median": med, "ms_min": min(times), "ms_max": max(times),
                "set_evals_per_s": l / (med * 1e-3), "kernel_ms": kern,
                "kernel_tflops": flops / (kern * 1e-3) / 1e12,
                "kernel_frac": flops / (kern * 1e-3) / 1e12 / PEAK_TFLOPS[prec],
            }
            if cpu is not None:
                rec["oracle_set_evals_per_s"] = cpu["value"]
                rec["oracle_threads"] = cpu["cores"]
                rec["speedup_vs_oracle"] = rec["set_evals_per_s"] / cpu["value"]
            line = json.dumps(rec)
            print(line, flush=True)
            if sink:
                sink.write(line + "\n")
                sink.flush()
            table.append(rec)
            log(f"{axis}: n={n} l={l} k={k} {prec}: {med:.3f} ms median, kernel {rec['kernel_tflops']:.1f} TFLOP/s "
                f"({100 * rec['kernel_frac']:.1f} %)" + (f", x{rec['speedup_vs_oracle']:.0f} vs oracle" if cpu else ""))
            del V, out
        del sets
    if sink:
        sink.close()
    log("| series | n | l | k | precision | median ms | min ms | max ms | set evals/s | kernel TFLOP/s | "
        "% peak | oracle set evals/s | speedup |")
    log("|---|---|---|---|---|---|---|---|---|---|---|---|---|")
    for r in table:
        o = r.get("oracle_set_evals_per_s")
        log(f"| {r['series']} | {r['n']} | {r['l']} | {r['k']} | {r['precision']} | {r['ms_median']:.3f} | "
            f"{r['ms_min']:.3f} | {r['ms_max']:.3f} | {r['set_evals_per_s']:.3g} | {r['kernel_tflops']:.1f} | "
            f"{100 * r['kernel_frac']:.1f} | " + (f"{o:.3g} | {r['speedup_vs_oracle']:.0f} |" if o else "- | - |"))


def run_streamed(args, w, dev):
    """Out-of-core mode: V and the sets in pinned host memory, streamed through
    the GPU by exemplar_eval_streamed (synchronous calls).  The rate includes
    the host-to-device copies of V on every call; it is reported on its own
    line, never as the default benchmark's value."""
    import torch
    log(f"generating {w.name}: {w.note}")
    p = synth.make(w)
    Xs, _ = synth.rounded(p.X, w.precision)
    V = (Xs if isinstance(Xs, torch.Tensor) else torch.from_numpy(Xs)).contiguous().pin_memory()
    S = torch.from_numpy(p.sets).contiguous()
    out = torch.empty(w.l, dtype=torch.float32)
    call = lambda: api.exemplar_eval_streamed(V, S, rows_per_block=args.rows_per_block, out=out)  # noqa: E731
    warmup, sec = warm_up(call, args.warmup, lambda: None)  # the call is synchronous
    steps = timed_steps(args.steps, sec, min_steps=5)
    api.exemplar_prof_read()
    api.exemplar_prof_enable(True)
    t0 = time.perf_counter()
    for _ in range(steps):
        call()
    dt = (time.perf_counter() - t0) / steps
    api.exemplar_prof_enable(False)
    kern_ms, launches = api.exemplar_prof_read()
    vbytes = V.numel() * V.element_size()
    rec = {
        "metric": "set evaluations/s, V streamed from host memory (PCIe-inclusive)",
        "value": w.l / dt, "unit": "set evaluations/s", "ms_per_call": dt * 1e3, "steps": steps, "warmup": warmup,
        "v_bytes": vbytes, "v_stream_gb_per_s": vbytes / dt / 1e9,
        "kernel_ms_per_call": kern_ms / max(steps, 1), "kernel_launches_per_call": launches / max(steps, 1),
        "rows_per_block": args.rows_per_block, "dtype": DTYPE_NAME[w.precision], "data": "synthetic",
        "config": {"workload": f"{w.name}: {w.note}", "n": w.n, "d": w.d, "l": w.l, "k": w.k},
    }
    print(json.dumps(rec), flush=True)


def run_greedy(args, w, dev):
    """Greedy driver (Algorithm 1 on the device): `--greedy-rounds` rounds of
    scoring every point of V as a candidate, per call.  One JSON line of its
    own; the oracle baseline scores a sample of candidates against the
    mid-run solution S_{K/2} on the host cores."""
    import torch
    K = args.greedy_rounds
    log(f"generating {w.name}: {w.note}")
    p = synth.make(w)
    V = torch.from_numpy(p.X).to(dev).contiguous()
    S_out = torch.empty(K, dtype=torch.int32, device=dev)
    f_out = torch.empty(K, dtype=torch.float32, device=dev)
    warmup, sec = warm_up(lambda: api.exemplar_greedy(V, K, S_out, f_out), args.warmup, torch.cuda.synchronize)
    steps = timed_steps(args.steps, sec, min_steps=3)
    api.exemplar_prof_read()
    api.exemplar_prof_enable(True)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(steps):
        api.exemplar_greedy(V, K, S_out, f_out)
    ev1.record(stream)
    torch.cuda.synchronize()
    api.exemplar_prof_enable(False)
    kern_ms, launches = api.exemplar_prof_read()
    ms = ev0.elapsed_time(ev1) / steps
    n, d = w.n, w.d
    cand_evals = n * K                      # every point is scored in every round
    flops = 2.0 * n * n * d * K             # scoring contractions (the cache update is n * d per round)
    kern_per_call = kern_ms / steps
    rec = {
        "metric": "greedy rounds/s and candidate evaluations/s (exemplar_greedy, Algorithm 1 on the device)",
        "value": K / (ms * 1e-3), "unit": "rounds/s", "ms_per_call": ms, "rounds": K, "steps": steps, "warmup": warmup,
        "candidate_evals_per_s": cand_evals / (ms * 1e-3),
        "scoring_kernel_ms_per_call": kern_per_call, "scoring_launches_per_call": launches / max(steps, 1),
        "roofline": {"bound": "mfma", "achieved": flops / (kern_per_call * 1e-3) / 1e12, "peak": PEAK_TFLOPS["fp32"],
                     "unit": "TFLOP/s", "frac": flops / (kern_per_call * 1e-3) / 1e12 / PEAK_TFLOPS["fp32"]},
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"{w.name} points: {w.note}", "n": n, "d": d, "rounds": K},
        "S": S_out.cpu().tolist(), "f": [float(x) for x in f_out.cpu()],
    }
    if not args.no_cpu_baseline:
        import oracle
        o = oracle.load()
        threads = o.threads(0)
        X64 = p.X.astype(np.float64)
        half = rec["S"][:K // 2]
        probe = np.arange(0, n, max(1, n // 16), dtype=np.int32)[:16]
        t0 = time.perf_counter()
        o.gain(X64, np.asarray(half, np.int32), probe, threads)
        dt = time.perf_counter() - t0
        rec["cpu_baseline"] = {
            "value": len(probe) / dt, "unit": "candidate evaluations/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(probe)} candidates scored against S of size {len(half)} (the GPU's first {len(half)} picks), "
                      f"fp64 direct evaluation, {threads} threads on {cpu_model()}",
            "seconds": dt,
        }
    print(json.dumps(rec), flush=True)


def run_sqnorm(args, w, dev):
    """Squared norms q[i] = ||v_i||^2 (exemplar_sqnorm) of the workload's
    points: one HBM-bound pass over V.  Algorithmic bytes per launch are
    n * d * element size read plus 4 n written; a device copy of V's bytes
    (read + write) is timed beside it as the practical ceiling.  One JSON
    line of its own."""
    import torch
    log(f"generating {w.name}: {w.note}")
    p = synth.make(w)
    Xs, X64 = synth.rounded(p.X, w.precision)
    V = (Xs if isinstance(Xs, torch.Tensor) else torch.from_numpy(Xs)).to(dev).contiguous()
    q = torch.empty(w.n, dtype=torch.float32, device=dev)
    step = lambda: api.exemplar_sqnorm(V, out=q)  # noqa: E731
    warmup, sec = warm_up(step, args.warmup, torch.cuda.synchronize)
    steps = timed_steps(args.steps, sec, min_steps=20)
    stream = torch.cuda.current_stream()

    def timed(fn):
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(steps):
            fn()
        ev1.record(stream)
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / steps

    ms = timed(step)
    vflat = V.reshape(-1)
    dst = torch.empty_like(vflat)
    for _ in range(5):
        dst.copy_(vflat)
    copy_ms = timed(lambda: dst.copy_(vflat))
    vbytes = V.numel() * V.element_size()
    algo = vbytes + 4 * w.n
    achieved = algo / (ms * 1e-3) / 1e9
    rec = {
        "metric": "squared norms/s (exemplar_sqnorm) + % of HBM peak",
        "value": w.n / (ms * 1e-3), "unit": "rows/s", "ms_per_call": ms, "steps": steps, "warmup": warmup,
        "higher_is_better": True, "dtype": DTYPE_NAME[w.precision], "data": "synthetic",
        "config": {"workload": f"{w.name} points: {w.note}", "n": w.n, "d": w.d, "precision": w.precision},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": load_traffic("sqnorm_kernel", w.name),
                     "kernel": "sqnorm_kernel", "bytes_per_launch": algo},
        "device_copy": {"bytes": 2 * vbytes, "ms": copy_ms, "gb_per_s": 2 * vbytes / (copy_ms * 1e-3) / 1e9},
    }
    if not args.no_cpu_baseline:
        import oracle
        o = oracle.load()
        rows = min(w.n, max(1, int(2e8 // max(w.d, 1))))
        t0 = time.perf_counter()
        reps = 0
        while True:
            o.sqnorm(X64[:rows])
            reps += 1
            dt = time.perf_counter() - t0
            if dt >= min(args.cpu_budget, 10.0):
                break
        rec["cpu_baseline"] = {
            "value": rows * reps / dt, "unit": "rows/s", "cores": 1, "kind": "oracle",
            "sample": f"the first {rows} rows, {reps} passes (fp64, one thread) on {cpu_model()}",
            "seconds": dt,
        }
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help=f"timed steps (default: at least {MIN_STEPS} and {TIMED_SECONDS} s of work)")
    ap.add_argument("--warmup", type=int, default=None,
                    help=f"untimed warm-up steps (default: {WARMUP_SECONDS} s of back-to-back steps, "
                         f"at least {MIN_WARMUP})")
    ap.add_argument("--workload", default="large1m", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle time for the CPU baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true", help="run a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--traffic-summary", metavar="DIR",
                    help="summarise rocprofv3 FETCH_SIZE/WRITE_SIZE runs under DIR into profiles/")
    ap.add_argument("--kernel", default="eval_mfma_kernel", help="kernel name for --traffic-summary")
    ap.add_argument("--sweep", metavar="SERIES",
                    help="run the Section V-A series instead: n, l, k (comma-separated) or all")
    ap.add_argument("--sweep-precisions", default="fp32,fp16")
    ap.add_argument("--sweep-reps", type=int, default=15, help="timed calls per sweep point (median reported)")
    ap.add_argument("--sweep-out", metavar="FILE", help="also write the sweep's JSON lines to FILE")
    ap.add_argument("--sweep-cpu-budget", type=float, default=1.0, help="seconds of oracle time per sweep point")
    ap.add_argument("--sweep-warmup-seconds", type=float, default=0.3,
                    help="untimed back-to-back calls before each sweep point's timed calls")
    ap.add_argument("--streamed", action="store_true",
                    help="time exemplar_eval_streamed (V in pinned host memory) instead; one JSON line of its own")
    ap.add_argument("--rows-per-block", type=int, default=0, help="row block of --streamed (0 = library default)")
    ap.add_argument("--greedy-rounds", type=int, default=0, metavar="K",
                    help="time exemplar_greedy with K rounds over the workload's points instead (fp32)")
    ap.add_argument("--sqnorm", action="store_true",
                    help="time exemplar_sqnorm over the workload's points instead (HBM-bound); one JSON line")
    args = ap.parse_args()

    if args.traffic_summary:
        print(json.dumps(traffic_summary(args.traffic_summary, args.kernel, args.workload)))
        return

    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}); the library has no multi-GPU "
              "path in this version.", file=sys.stderr)
        sys.exit(2)

    import torch

    if not torch.cuda.is_available():
        sys.exit("bench.py needs a GPU")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_probe:
        copy_probe(args.steps if args.steps else 5)
        return
    api.load()
    if args.sweep:
        run_paper_sweep(args, dev)
        return

    w = synth.WORKLOADS[args.workload]
    if args.greedy_rounds > 0:
        run_greedy(args, w, dev)
        return
    if args.sqnorm:
        run_sqnorm(args, w, dev)
        return
    if args.streamed:
        if w.mode != "eval":
            sys.exit("--streamed evaluates set batches (an eval workload)")
        run_streamed(args, w, dev)
        return
    log(f"generating {w.name}: {w.note}")
    p = synth.make(w)
    Xs, X64 = synth.rounded(p.X, w.precision)
    V = (Xs if isinstance(Xs, torch.Tensor) else torch.from_numpy(Xs)).to(dev).contiguous()
    if w.mode == "gain":
        S = torch.from_numpy(p.S).to(dev)
        C = torch.from_numpy(p.cands).to(dev)
        out = torch.empty(w.l, dtype=torch.float32, device=dev)
        step = lambda: api.exemplar_gain(V, S, C, out=out)  # noqa: E731
        kk = w.k + 1
        contraction_cols = w.l          # scoring kernel: n x l x d
    else:
        sets = torch.from_numpy(p.sets).to(dev)
        out = torch.empty(w.l, dtype=torch.float32, device=dev)
        step = lambda: api.exemplar_eval(V, sets, out=out)  # noqa: E731
        kk = w.k
        contraction_cols = w.l * w.k    # eval kernel: n x (l k) x d
    prec_code = {"fp32": api.EXEMCL_FP32, "fp16": api.EXEMCL_FP16, "bf16": api.EXEMCL_BF16}[w.precision]
    path, ws = api.exemplar_plan(w.n, w.d, w.l, w.k if w.mode == "eval" else 1, prec_code)
    torch.cuda.synchronize()

    warmup, sec_per_step = warm_up(step, args.warmup, torch.cuda.synchronize)
    steps = timed_steps(args.steps, sec_per_step)
    log(f"warm-up: {warmup} steps ({warmup * sec_per_step:.2f} s); timing {steps} steps")
    api.exemplar_prof_read()  # drop anything recorded before

    stream = torch.cuda.current_stream()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    # The dominant kernel's duration comes from HIP events around a sample
    # of about PROF_SAMPLES launches spread evenly over the timed steps:
    # recording a pair on every step would slow the steps it measures.
    prof_every = max(1, steps // PROF_SAMPLES)
    api.exemplar_prof_enable(prof_every)
    torch.cuda.synchronize()
    ev0.record(stream)
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    api.exemplar_prof_enable(False)
    kern_ms, launches = api.exemplar_prof_read()
    ms = ev0.elapsed_time(ev1)
    ms_per_step = ms / steps
    kern_avg_ms = kern_ms / max(launches, 1)

    value = w.l / (ms_per_step * 1e-3)
    terms = w.n * kk * w.l
    flops_per_launch = 2.0 * w.n * contraction_cols * w.d
    achieved = flops_per_launch / (kern_avg_ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[w.precision]
    log(f"{steps} steps: {ms_per_step * 1e3:.1f} us/step (wall {wall / steps * 1e6:.1f} us/step), "
        f"dominant kernel {kern_avg_ms * 1e3:.1f} us avg over {launches} launches, {achieved:.1f} TFLOP/s")

    res = {
        "metric": METRIC,
        "value": value,
        "unit": "set evaluations/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPE_NAME[w.precision],
        "data": "synthetic",
        "distance_terms_per_s": terms / (ms_per_step * 1e-3),
        "config": {
            "workload": f"{w.name}: {w.note}", "n": w.n, "d": w.d, "l": w.l,
            ("base_set" if w.mode == "gain" else "k"): w.k, "mode": w.mode,
            "precision": w.precision, "seed": w.seed, "path": path, "workspace_bytes": ws,
        },
        "roofline": {
            "bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s", "frac": achieved / peak,
            "traffic": load_traffic("eval_mfma_kernel" if path == "mfma" else "eval_valu_kernel", w.name),
            "kernel": "eval_mfma_kernel" if path == "mfma" else "eval_valu_kernel",
            "kernel_avg_us": kern_avg_ms * 1e3, "flops_per_launch": flops_per_launch,
            "timed_launches": launches, "timed_every": prof_every,
        },
    }
    if not args.no_cpu_baseline:
        log(f"oracle baseline (budget {args.cpu_budget:.0f} s) ...")
        res["cpu_baseline"] = cpu_baseline(p, X64, args.cpu_budget)
        log(f"oracle: {res['cpu_baseline']['value']:.3g} set-evals/s on {res['cpu_baseline']['cores']} threads")
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
