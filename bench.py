#!/usr/bin/env python3
"""Benchmark of the CurvaDion optimizer step (Dion + RMMC gate) on one MI355X.

Workload (default): the 1.3B-shaped layer set -- the 96 weight matrices of a
GPT with d_model 2048 and 24 blocks (2048x6144, 2048x2048, 2048x8192,
8192x2048 per block; 1.208e9 parameters), rank r = 512, bf16 gradients, fp32
momentum / weights / Q, seeded low-rank(64) + noise gradients, tau = 0.5.
A "step" is one Algorithm-2 step over the whole set: buffer update and RMMC
for every layer, the gate, then the branch the gate picks.  The timed region
replays the workload's trajectory from step 1 (its first step always syncs:
prev_norm starts at 0), so both branches are timed.

Prints ONE JSON line: params updated per second (whole job), per-branch step
times, the roofline of the kernel with the largest share of the trajectory,
and the float64 oracle timed on this host's cores on a bounded sample.  An
untimed profiling pass of the same K steps brackets every launch with HIP
events (inside the library; the sync branch's shape batches then run one
after another) to find that kernel and the per-kind table; the timed pass
then brackets only that kernel's launches, since each bracketed launch idles
the GPU for several microseconds.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--policy rmmc|always|never]

Profiling (rocprofv3 under the same command; the summaries go to profiles/):

    rocprofv3 --kernel-trace --stats -f csv -d DIR -o bench -- python3 bench.py
    python3 bench.py --summarize-trace DIR BENCH_JSON OUT
    rocprofv3 --pmc FETCH_SIZE -f csv -d DIR_F -o pmc -- python3 bench.py --copy-calibration 1024 ...
    rocprofv3 --pmc WRITE_SIZE -f csv -d DIR_W -o pmc -- python3 bench.py --copy-calibration 1024 ...
    python3 bench.py --summarize-pmc DIR_F DIR_W OUT --copy-calibration 1024

The counter summary records a digest of the kernels' sources; the bench line
reports the dominant kernel's counted HBM traffic only while that digest still
matches the sources.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import math
import shlex
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "Dion+RMMC optimizer step: params updated/sec/GPU + achieved HBM GB/s"
PEAK_HBM_GBPS = 8000.0
PEAK_TFLOPS = {"f64": 78.6, "f32": 157.3, "bf16": 2500.0}
# bound, MFMA dtype and executed MFMA flops per algorithmic flop, per kernel kind
# (bf16x6: each fp32 product is formed from six bf16 piece products; bf16x9:
# nine slice products of the exact Gram matrix)
KIND_BOUND = {
    "form_buffer": ("hbm", None, 1), "form_buffer_local": ("hbm", None, 1),
    "local_update": ("hbm", None, 1), "gate": ("hbm", None, 1),
    "reduce_splits": ("hbm", None, 1), "colnorm": ("hbm", None, 1),
    "power_bq_f64": ("mfma", "f64", 1), "gram_f64": ("mfma", "f64", 1), "trsm_f64": ("mfma", "f64", 1),
    "power_btp_f64": ("mfma", "f64", 1),
    "cholesky_f64": ("mfma", "f64", 1), "power_bq_bf16x6": ("mfma", "bf16", 6),
    "update_bf16x6": ("mfma", "bf16", 6),
    "power_bq_bf16x3": ("mfma", "bf16", 3), "power_btp_bf16x3": ("mfma", "bf16", 3),
    "update_bf16": ("hbm", None, 1), "gram_bf16x6": ("mfma", "bf16", 6),
    "apply_bf16x6": ("mfma", "bf16", 6), "trtri_f64": ("mfma", "f64", 1),
    # exact Gram matrix: nine slice products per fp64-accurate product
    "gram_bf16x9": ("mfma", "bf16", 9),
    # the buffer pass fused into P~ = B Q (predicted sync steps, bf16 gradients)
    "form_power_bq_bf16x3": ("mfma", "bf16", 3),
    "update_f32": ("hbm", None, 1),
    # small layers: one workgroup per layer, latency-bound; priced against the fp64 peak
    "small_cholqr": ("alu", "f64", 1), "small_update": ("hbm", None, 1),
}
POLICIES = {"rmmc": 0, "always": 1, "never": 2, "every_h": 3}

# kernel kind -> (kernel-name pattern in the profiler's output, source files);
# kinds whose kernel template is shared with other kinds have no pattern
CSRC = os.path.join(ROOT, "paper_2512_13728_amd", "csrc")
_STREAM = ["k_stream.hip", "common.hpp", "plan.hpp"]
_BF = ["k_gemm_bf.hip", "bf16_split.hpp", "mfma_tile.hpp", "common.hpp", "plan.hpp"]
KIND_KERNEL = {
    "form_buffer": (r"k_form_buffer<\w+, 0>", _STREAM),
    "form_buffer_local": (r"k_form_buffer<\w+, 1>", _STREAM),
    "local_update": (r"k_local_update<", _STREAM),
    "gate": (r"k_gate\b", _STREAM),
    "update_bf16": (r"k_update_pl<1,", _BF),
    "update_bf16x6": (r"k_update_pl<3,", _BF),
    "update_f32": (r"k_update_vec<", ["k_update_vec.hip", "common.hpp", "plan.hpp"]),
    "cholesky_f64": (None, ["k_chol.hip", "chol_wave.hpp", "mfma_tile.hpp", "common.hpp", "plan.hpp"]),
}
COPY_PATTERN = r"neg_kernel"          # the calibration copy: b = -a, fp32, elementwise
PMC_PROFILE = os.path.join(ROOT, "profiles", "{workload}_hbm_traffic_pmc.txt")


def source_digest(files) -> str:
    h = hashlib.sha256()
    for f in sorted(files):
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()[:16]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=2)
    p.add_argument("--workload", default="gpt1p3b")
    p.add_argument("--policy", default="rmmc", choices=sorted(POLICIES))
    p.add_argument("--H", type=int, default=4, help="sync period for --policy every_h (Scheduled Sync Dion)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--pool", type=int, default=20, help="distinct gradient sets kept resident")
    p.add_argument("--rank", type=int, default=0, help="override the workload's rank r")
    p.add_argument("--async", dest="async_steps", action="store_true",
                   help="timed steps asynchronous (no host output: both branches enqueued, every kernel "
                        "predicated on the gate's decision in device memory); the decisions are those of "
                        "the blocking profiling pass over the same inputs, checked against the last step's")
    p.add_argument("--stream-inputs", action="store_true",
                   help="draw every step's gradients on the GPU just before the step (outside its "
                        "timed interval) instead of cycling a resident pool; the default for "
                        "trajectories longer than the pool (the 200-step mixed workload)")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="first run a plain streaming copy of MIB MiB (fp32, b = -a) three times, "
                        "the reference for the hardware byte counters")
    p.add_argument("--summarize-trace", nargs=3, metavar=("DIR", "BENCH_JSON", "OUT"),
                   help="write the kernel statistics of a rocprofv3 --kernel-trace --stats run")
    p.add_argument("--summarize-mfma", nargs=2, metavar=("DIR", "OUT"),
                   help="write the per-kernel MFMA busy fraction of a rocprofv3 --pmc "
                        "SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CYCLES GRBM_GUI_ACTIVE run")
    p.add_argument("--summarize-pmc", nargs=3, metavar=("FETCH_DIR", "WRITE_DIR", "OUT"),
                   help="write the per-kernel HBM traffic of two rocprofv3 --pmc runs (give the "
                        "same --copy-calibration size)")
    return p.parse_args()


def _kernel_name(raw: str) -> str:
    name = raw.replace("(anonymous namespace)::", "").replace("void ", "")
    return name.split("(cd::")[0].strip()


def summarize_trace(d: str, bench_json: str, out: str):
    """Kernel statistics (rocprofv3 --kernel-trace --stats, csv) of one bench run."""
    stats = glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True)
    if not stats:
        sys.exit(f"no *kernel_stats.csv under {d}")
    rows = list(csv.DictReader(open(stats[0])))
    ours = [r for r in rows if "cd::" in r["Name"]]
    other_ns = sum(float(r["TotalDurationNs"]) for r in rows if "cd::" not in r["Name"])
    b = json.loads(open(bench_json).read().strip().splitlines()[-1])
    wl = b["config"].get("workload_name", "gpt1p3b")
    lines = [f"# rocprofv3 kernel statistics: {b['config']['workload']}",
             "# commands (from the repository root):",
             f"#   rocprofv3 --kernel-trace --stats -f csv -d {d} -o bench -- "
             f"{b.get('command', 'python3 bench.py ' + WORKLOAD_ARGS.get(wl, '')).strip()} > {bench_json}",
             f"#   python3 bench.py --summarize-trace {d} {bench_json} {out}",
             "# calls include the warmup steps and the untimed profiling pass (the same",
             "# trajectory once more); torch kernels (input generation, state reset)",
             f"# are left out below: {other_ns / 1e6:.1f} ms in total.",
             "# sync-step kernels of different shape batches run concurrently (up to four",
             "# streams): their durations overlap and do not add up to the step time; the",
             "# skip-step kernels (form_buffer, gate) run alone.", "",
             f"{'kernel':64s} {'calls':>6s} {'avg_us':>10s} {'total_ms':>10s}"]
    for r in sorted(ours, key=lambda r: -float(r["TotalDurationNs"])):
        lines.append(f"{_kernel_name(r['Name'])[:64]:64s} {int(r['Calls']):6d} "
                     f"{float(r['AverageNs']) / 1e3:10.1f} {float(r['TotalDurationNs']) / 1e6:10.3f}")
    rf = b["roofline"]
    lines += ["", "# the same run's bench line (timed pass only; HIP events around the dominant",
              "# kernel's launches):",
              f"#   value {b['value']:.4g} params/s, {b['ms_per_step']:.3f} ms/step, "
              f"{b['config']['sync_steps']} sync + {b['config']['local_steps']} local steps",
              f"#   dominant kernel {rf['kernel']}: avg launch {rf['avg_launch_ms'] * 1e3:.1f} us, "
              f"{rf['achieved']} {rf['unit']} of {rf['peak']} ({rf['frac'] * 100:.1f}%)"]
    for k, v in b["branches"].items():
        lines.append(f"#   {k}: {json.dumps(v)}")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _pmc_dispatches(d: str, counter: str):
    """[(dispatch id, kernel name, value)] of one counter, in dispatch order
    (values of one dispatch summed over the rows the profiler writes)."""
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        sys.exit(f"no *counter_collection.csv under {d}")
    per = {}
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            key = int(r["Dispatch_Id"])
            per.setdefault(key, [r["Kernel_Name"], 0.0])[1] += float(r["Counter_Value"])
    return [(k, v[0], v[1]) for k, v in sorted(per.items())]


# kernels of the step's two streaming passes and its gate; every other
# library kernel belongs to the sync branch
STEP_COMMON = (r"k_form_buffer<", r"k_gate\b", r"k_local_update<")


def steps_of(dispatches):
    """Library dispatches (in order) cut into steps: a step starts at its
    first buffer-pass launch (k_form_buffer, or k_form_bq where the pass is
    fused into P~ = B Q) after the previous step's gate and runs until the
    next step's.  Returns [(kind, [indices])], kind "sync" when a sync-branch
    kernel ran."""
    steps, cur, gated = [], None, True
    for i, (_, name, _) in enumerate(dispatches):
        if "cd::" not in name:
            continue
        if re.search(r"k_form_buffer<|k_form_bq<", name) and gated:
            cur = []
            steps.append(cur)
            gated = False
        if re.search(r"k_gate\b", name):
            gated = True
        if cur is not None:
            cur.append(i)
    out = []
    for idx in steps:
        sync = any(not any(re.search(p, dispatches[i][1]) for p in STEP_COMMON) for i in idx)
        out.append(("sync" if sync else "local", idx))
    return out


def _pmc_rows(d: str, counter: str):
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        sys.exit(f"no *counter_collection.csv under {d}")
    per = {}
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            key = (f, r["Dispatch_Id"])
            per.setdefault(key, [r["Kernel_Name"], 0.0])[1] += float(r["Counter_Value"])
    return list(per.values())


def summarize_pmc(fdir: str, wdir: str, out: str, workload: str, cal_mib: int):
    """HBM traffic per dispatch from FETCH_SIZE and WRITE_SIZE (KiB), each
    scaled by what the counter reads for the calibration copy of known size."""
    if cal_mib <= 0:
        sys.exit("--summarize-pmc needs the --copy-calibration size the profiled runs used")
    cal_bytes = cal_mib << 20
    res = {}
    for counter, d in (("FETCH_SIZE", fdir), ("WRITE_SIZE", wdir)):
        rows = _pmc_rows(d, counter)
        copy = [v for k, v in rows if re.search(COPY_PATTERN, k)]
        if not copy:
            sys.exit(f"{counter}: no calibration copy dispatch ({COPY_PATTERN}) in {d}")
        res[counter] = (rows, copy)
    factor = {}
    for counter, (rows, copy) in res.items():
        kib = sorted(copy)[len(copy) // 2]
        factor[counter] = cal_bytes / (kib * 1024.0)
    table = {}
    for counter, (rows, _) in res.items():
        for k, v in rows:
            name = _kernel_name(k)
            if "cd::" not in k:
                continue
            t = table.setdefault(name, {"FETCH_SIZE": [], "WRITE_SIZE": []})
            t[counter].append(v * 1024.0 * factor[counter])
    kinds = {}
    for kind, (pat, files) in KIND_KERNEL.items():
        if pat is None:
            continue
        f_all, w_all = [], []
        for name, t in table.items():
            if re.search(pat, name):
                f_all += t["FETCH_SIZE"]
                w_all += t["WRITE_SIZE"]
        if f_all and w_all:
            kinds[kind] = {"fetch_bytes_per_launch": sum(f_all) / len(f_all),
                           "write_bytes_per_launch": sum(w_all) / len(w_all),
                           "traffic_bytes_per_launch": sum(f_all) / len(f_all) + sum(w_all) / len(w_all),
                           "dispatches": len(f_all), "source_digest": source_digest(files)}
    lines = [f"# rocprofv3 hardware counters: HBM bytes per dispatch, workload {workload}",
             "# commands (from the repository root):",
             f"#   rocprofv3 --pmc FETCH_SIZE --kernel-include-regex 'cd::|neg_kernel' -f csv -d {fdir} -o pmc "
             f"-- python3 bench.py {WORKLOAD_ARGS.get(workload, '')}--no-cpu-baseline --copy-calibration {cal_mib}",
             f"#   rocprofv3 --pmc WRITE_SIZE --kernel-include-regex 'cd::|neg_kernel' -f csv -d {wdir} -o pmc "
             f"-- python3 bench.py {WORKLOAD_ARGS.get(workload, '')}--no-cpu-baseline --copy-calibration {cal_mib}",
             f"#   python3 bench.py {_wl_flag(workload)}--summarize-pmc {fdir} {wdir} {out} --copy-calibration {cal_mib}",
             f"# calibration: a streaming copy (b = -a, fp32) of {cal_bytes} B read + {cal_bytes} B written;",
             f"#   FETCH_SIZE x {factor['FETCH_SIZE']:.4f} and WRITE_SIZE x {factor['WRITE_SIZE']:.4f} give bytes",
             "# all dispatches of the run (warmup steps, profiling pass, timed pass); bytes are scaled, per dispatch", "",
             f"{'kernel':64s} {'disp':>5s} {'fetch_MB':>10s} {'write_MB':>10s}"]
    for name, t in sorted(table.items(), key=lambda kv: -sum(kv[1]["FETCH_SIZE"]) - sum(kv[1]["WRITE_SIZE"])):
        nf = max(len(t["FETCH_SIZE"]), 1)
        nw = max(len(t["WRITE_SIZE"]), 1)
        lines.append(f"{name[:64]:64s} {len(t['FETCH_SIZE']):5d} {sum(t['FETCH_SIZE']) / nf / 1e6:10.2f} "
                     f"{sum(t['WRITE_SIZE']) / nw / 1e6:10.2f}")
    # HBM bytes per step, by branch: the two runs dispatch the same sequence
    fd = _pmc_dispatches(fdir, "FETCH_SIZE")
    wd = _pmc_dispatches(wdir, "WRITE_SIZE")
    fs, ws = steps_of(fd), steps_of(wd)
    if len(fs) != len(ws) or any(a[0] != b[0] or len(a[1]) != len(b[1]) for a, b in zip(fs, ws)):
        sys.exit("the FETCH_SIZE and WRITE_SIZE runs dispatched different step sequences")
    per_branch = {}
    for (kind, fi), (_, wi) in zip(fs, ws):
        fb = sum(fd[i][2] for i in fi) * 1024.0 * factor["FETCH_SIZE"]
        wb = sum(wd[i][2] for i in wi) * 1024.0 * factor["WRITE_SIZE"]
        per_branch.setdefault(kind, []).append((fb, wb))
    steps = {"source_digest": source_digest(ALL_SOURCES)}
    lines += ["", "# HBM bytes per step (every library kernel of the step, the dispatch sequence cut at each",
              "# step's first buffer-pass launch), median over the steps of each branch in the run:"]
    for kind, v in sorted(per_branch.items()):
        fmed = sorted(x[0] for x in v)[len(v) // 2]
        wmed = sorted(x[1] for x in v)[len(v) // 2]
        steps[kind] = {"fetch_bytes": fmed, "write_bytes": wmed, "bytes": fmed + wmed, "steps": len(v)}
        lines.append(f"#   {kind:6s} steps {len(v):4d}  fetch {fmed / 1e9:8.3f} GB  write {wmed / 1e9:8.3f} GB")
    lines += ["", "json " + json.dumps({"workload": workload, "factor": factor, "kinds": kinds, "steps": steps})]
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


ALL_SOURCES = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".hpp", ".cpp")))


def counted_step_bytes(workload: str):
    """Counted HBM bytes per sync and per local step from the committed
    counter summary, or {} if there is none or any kernel source changed since."""
    path = PMC_PROFILE.format(workload=workload)
    if not os.path.exists(path):
        return {}
    for line in open(path):
        if line.startswith("json "):
            st = json.loads(line[5:]).get("steps", {})
            if st.get("source_digest") == source_digest(ALL_SOURCES):
                return {k: v["bytes"] for k, v in st.items() if k in ("sync", "local")}
    return {}


N_CU, N_XCD, SIMD_PER_CU = 256, 8, 4
# the bench arguments that select each profiled workload (default: the 1.3B set)
def _wl_flag(workload: str) -> str:
    """The --workload option a summarising command needs (none for the default)."""
    return "" if workload == "gpt1p3b" else f"--workload {workload} "


WORKLOAD_ARGS = {"gpt1p3b": "", "gpt160m": "--workload gpt160m --steps 50 ",
                 "mixed1p3b": "--workload mixed1p3b --steps 200 ", "single256": "--workload single256 "}


def summarize_mfma(d: str, out: str, workload: str):
    """Per kernel of the library: the MFMA busy fraction counted by the
    hardware, SQ_VALU_MFMA_BUSY_CYCLES / (SIMDs x cycles the kernel ran),
    with the kernel's cycles from GRBM_GUI_ACTIVE (which counts on every XCD:
    divided by their number).  Dispatches of one kernel name are summed."""
    counters = ("SQ_VALU_MFMA_BUSY_CYCLES", "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE")
    vals = {c: _pmc_dispatches(d, c) for c in counters}
    table = {}
    for i, (did, name, mfma) in enumerate(vals["SQ_VALU_MFMA_BUSY_CYCLES"]):
        if "cd::" not in name:
            continue
        t = table.setdefault(_kernel_name(name), {"n": 0, "mfma": 0.0, "busy": 0.0, "gui": 0.0})
        t["n"] += 1
        t["mfma"] += mfma
        t["busy"] += vals["SQ_BUSY_CYCLES"][i][2]
        t["gui"] += vals["GRBM_GUI_ACTIVE"][i][2]
    lines = [f"# rocprofv3 hardware counters: MFMA busy per kernel, workload {workload}",
             "# commands (from the repository root):",
             f"#   rocprofv3 --pmc {' '.join(counters)} --kernel-include-regex 'cd::' -f csv -d {d} -o pmc "
             f"-- python3 bench.py {WORKLOAD_ARGS.get(workload, '')}--no-cpu-baseline --steps 2 --warmup 1 "
             "--policy always",
             f"#   python3 bench.py {_wl_flag(workload)}--summarize-mfma {d} {out}",
             f"# mfma_busy = SQ_VALU_MFMA_BUSY_CYCLES / ({N_CU * SIMD_PER_CU} SIMDs x GRBM_GUI_ACTIVE / {N_XCD} XCDs):",
             "# the fraction of the kernel's cycles in which an average SIMD's matrix unit was busy", "",
             f"{'kernel':64s} {'disp':>5s} {'cycles/disp':>12s} {'mfma_busy':>10s}"]
    summary = {}
    for name, t in sorted(table.items(), key=lambda kv: -kv[1]["gui"]):
        cyc = t["gui"] / N_XCD
        frac = t["mfma"] / (N_CU * SIMD_PER_CU * cyc) if cyc > 0 else 0.0
        summary[name] = {"dispatches": t["n"], "cycles": cyc, "mfma_busy": frac}
        lines.append(f"{name[:64]:64s} {t['n']:5d} {cyc / t['n']:12.4g} {frac:10.4f}")
    lines += ["", "json " + json.dumps({"workload": workload, "kernels": summary})]
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def counted_traffic(workload: str, kind: str):
    """Counted HBM bytes per launch of `kind` from the committed counter
    summary, or None if there is none or the kernel's sources changed since."""
    path = PMC_PROFILE.format(workload=workload)
    if kind not in KIND_KERNEL or not os.path.exists(path):
        return None
    for line in open(path):
        if line.startswith("json "):
            info = json.loads(line[5:]).get("kinds", {}).get(kind)
            if info and info["source_digest"] == source_digest(KIND_KERNEL[kind][1]):
                return info["traffic_bytes_per_launch"]
    return None


def cpu_baseline(w, n_sync: int, n_local: int, steps: int):
    """Time the float64 oracle on one layer of each distinct shape: one sync
    step and one local step each, repeated until ~10 s have passed; scale to
    the full set and to the timed region's mix of branches."""
    import numpy as np
    import oracle as O
    import synthetic as S
    try:
        from threadpoolctl import threadpool_limits
    except Exception:  # pragma: no cover
        threadpool_limits = None
    cores = min(len(os.sched_getaffinity(0)), 16)
    shapes = sorted(set(w.shapes), key=w.shapes.index)
    idx = [w.shapes.index(s) for s in shapes]
    sample_params = sum(m * n for m, n in shapes)
    data = []
    for li in idx:
        M0, X0, Q0 = S.initial_state(w, li, device="cpu")
        st = S.GradientStream(w, li, device="cpu")
        G1, G2 = st.next().double().numpy(), st.next().double().numpy()
        data.append((M0.double().numpy(), X0.double().numpy(), Q0.double().numpy(), G1, G2))
    ctx = threadpool_limits(cores) if threadpool_limits else None
    t_sync = t_local = 0.0
    reps = 0
    t_start = time.perf_counter()
    try:
        while reps == 0 or (time.perf_counter() - t_start < 10.0 and reps < 20):
            Ls = [O.OracleLayer.from_arrays(M, X, Q) for (M, X, Q, _, _) in data]
            t0 = time.perf_counter()
            O.group_step(Ls, [d[3] for d in data], w.mu, w.eta, w.tau, policy=O.POLICY_ALWAYS_SYNC)
            t1 = time.perf_counter()
            O.group_step(Ls, [d[4] for d in data], w.mu, w.eta, w.tau, policy=O.POLICY_NEVER_SYNC)
            t2 = time.perf_counter()
            t_sync += t1 - t0
            t_local += t2 - t1
            reps += 1
    finally:
        if ctx is not None:
            ctx.__exit__(None, None, None)
    per_param_sync = t_sync / reps / sample_params
    per_param_local = t_local / reps / sample_params
    t_job = w.params * (n_sync * per_param_sync + n_local * per_param_local)
    return {
        "value": w.params * steps / t_job,
        "unit": "params/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"float64 oracle, {len(shapes)} layers (one per shape, {sample_params} params), "
                   f"1 sync + 1 local step x {reps} reps; scaled to {w.params} params and the timed "
                   f"mix of {n_sync} sync + {n_local} local steps"),
        "sync_step_s": per_param_sync * w.params,
        "local_step_s": per_param_local * w.params,
    }


def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(*args.summarize_trace)
        return
    if args.summarize_mfma:
        summarize_mfma(*args.summarize_mfma, workload=args.workload)
        return
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, workload=args.workload, cal_mib=args.copy_calibration)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(the data-parallel all-reduces are identities at one worker). "
              "Run without --gpus or with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2512_13728_amd as cdl
    import synthetic as S

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    w = S.WORKLOADS[args.workload]
    if args.rank > 0:
        import dataclasses
        w = dataclasses.replace(w, r=args.rank)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    policy = POLICIES[args.policy]
    K, W = args.steps, args.warmup
    L = len(w.shapes)
    log(f"[bench] workload {w.name}: {L} matrices, {w.params} params, r={w.r}, G {w.grad_dtype}")
    if args.copy_calibration > 0:
        a = torch.ones(args.copy_calibration * (1 << 18), dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            torch.neg(a, out=b)
        torch.cuda.synchronize()
        log(f"[bench] copy calibration: streaming copy b = -a, bytes={a.numel() * 4} read and written")
        del a, b

    if args.H < 1:
        sys.exit("--H must be >= 1")
    layers = [cdl.Layer(m, n, w.r, grad_dtype=w.grad_dtype, tau=w.tau, eps=w.eps, policy=policy, H=args.H)
              for (m, n) in w.shapes]
    group = cdl.Group(layers)
    t0 = time.perf_counter()
    init = [S.initial_state(w, i, device=dev) for i in range(L)]
    M = [s[0].clone() for s in init]
    X = [s[1].clone() for s in init]
    Q = [s[2].clone() for s in init]
    streamed = args.stream_inputs or K > args.pool
    pool = 1 if streamed else max(1, min(args.pool, max(K, W)))
    streams = [S.GradientStream(w, i, device=dev) for i in range(L)]
    grads = [[st.next() for st in streams] for _ in range(pool)]
    torch.cuda.synchronize()
    log(f"[bench] inputs resident in HBM ({pool} gradient set{'s' if pool > 1 else ''}"
        f"{', the rest drawn between steps' if streamed else ''}) in {time.perf_counter() - t0:.1f}s")

    def reset():
        for i in range(L):
            M[i].copy_(init[i][0]); X[i].copy_(init[i][1]); Q[i].copy_(init[i][2])
        torch.cuda.synchronize()
        for lay in layers:
            lay.set_state(0.0, 0)

    for t in range(W):
        group.step(grads[t % pool], M, X, Q, w.mu, w.eta, w.r)
    torch.cuda.synchronize()
    reset()
    log(f"[bench] {W} warmup steps done; timing {K} steps from step 1")

    stream = torch.cuda.current_stream()
    sh = stream.cuda_stream
    # addresses marshalled once (the state tensors and every resident gradient set)
    # (and checked against the layers here, outside the timed steps)
    pM, pX, pQ = group.pack(M, "M"), group.pack(X, "X"), group.pack(Q, "Q", w.r)
    pG = [group.pack(gs, "G") for gs in grads]

    def trajectory(timing_kinds, asyn=False):
        """Steps 1..K from the initial state; kernel launches of the kinds in
        `timing_kinds` (None = every kind) bracketed by HIP events.  asyn: the
        steps are asynchronous (no per-step outcome on the host)."""
        reset()
        flags, rmmcs = [], []
        group.set_timing(True, timing_kinds)
        if streamed:
            # restart the streams so the trajectory is steps 1..K; each step's
            # inputs are drawn before its interval, which brackets only the step
            sts = [S.GradientStream(w, i, device=dev) for i in range(L)]
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                  for _ in range(K)]
            wall = 0.0
            for t in range(K):
                G = pG[0] if t == 0 else group.pack([st.next() for st in sts], "G")
                if t == 0:
                    for st in sts:
                        st.next()
                torch.cuda.synchronize()
                t1 = time.perf_counter()
                ev[t][0].record(stream)
                g, flag, _, _ = group.step(G, pM, pX, pQ, w.mu, w.eta, w.r, sh)
                ev[t][1].record(stream)
                torch.cuda.synchronize()
                wall += time.perf_counter() - t1
                flags.append(flag)
                rmmcs.append(g)
                if (t + 1) % 25 == 0:
                    log(f"[bench]   step {t + 1}: {sum(flags)} syncs so far")
            step_ms = [a.elapsed_time(b) for a, b in ev]
        else:
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
            torch.cuda.synchronize()
            t_start = time.perf_counter()
            ev[0].record(stream)
            for t in range(K):
                if asyn:
                    group.step(pG[t % pool], pM, pX, pQ, w.mu, w.eta, w.r, sh, wait=False)
                else:
                    g, flag, _, _ = group.step(pG[t % pool], pM, pX, pQ, w.mu, w.eta, w.r, sh)
                    flags.append(flag)
                    rmmcs.append(g)
                ev[t + 1].record(stream)
            torch.cuda.synchronize()
            wall = time.perf_counter() - t_start
            step_ms = [ev[t].elapsed_time(ev[t + 1]) for t in range(K)]
        kt = group.kernel_times()
        group.set_timing(False)
        return flags, rmmcs, step_ms, wall, kt

    # An untimed profiling pass of the same K steps brackets every launch (the
    # library then runs the sync branch's shape batches one after another, so
    # that each interval times its kernel alone): the per-kind table and the
    # dominant kernel.  The events idle the GPU for several microseconds at
    # each bracketed launch, so the timed pass, on the untimed schedule,
    # brackets only the dominant kernel's launches.
    prof_flags, prof_rmmcs, _, prof_wall, kt = trajectory(None)
    dom = max(kt.items(), key=lambda kv: kv[1]["total_ms"])[0]
    log(f"[bench] profiling pass: {K} steps in {prof_wall * 1e3:.2f} ms with every launch "
        f"bracketed (sync batches serial); dominant kernel {dom}")
    asyn = args.async_steps and not streamed
    flags, rmmcs, step_ms, elapsed, kt_dom = trajectory([dom], asyn)
    if asyn:
        g_last, f_last, _, _ = group.last_result()
        if f_last != prof_flags[-1] or g_last != prof_rmmcs[-1]:
            sys.exit(f"asynchronous steps diverged from the blocking pass: {g_last} {f_last} vs "
                     f"{prof_rmmcs[-1]} {prof_flags[-1]}")
        flags, rmmcs = prof_flags, prof_rmmcs
    log(f"[bench] timed {K} steps in {elapsed * 1e3:.2f} ms; syncs at "
        f"{[t + 1 for t, f in enumerate(flags) if f]}")

    n_sync = sum(flags)
    n_local = K - n_sync
    sync_ms = [x for x, f in zip(step_ms, flags) if f]
    local_ms = [x for x, f in zip(step_ms, flags) if not f]
    log("[bench] per kind, profiling pass (every launch bracketed):")
    for name, v in sorted(kt.items(), key=lambda kv: -kv[1]["total_ms"]):
        log(f"[bench]   {name:16s} launches {v['launches']:5d}  {v['total_ms']:9.3f} ms  "
            f"{v['bytes'] / max(v['total_ms'], 1e-9) / 1e6:8.1f} GB/s  "
            f"{v['flops'] / max(v['total_ms'], 1e-9) / 1e9:8.2f} TFLOP/s")

    # the dominant kernel's launches in the timed pass
    dv = kt_dom[dom]
    bound, prec, mult = KIND_BOUND.get(dom, ("hbm", None, 1))
    avg_ms = dv["total_ms"] / dv["launches"]
    if bound == "hbm":
        achieved = dv["bytes"] / dv["launches"] / (avg_ms * 1e-3) / 1e9
        peak, unit = PEAK_HBM_GBPS, "GB/s"
    else:
        achieved = mult * dv["flops"] / dv["launches"] / (avg_ms * 1e-3) / 1e12
        peak, unit = PEAK_TFLOPS[prec], "TFLOP/s"
    traffic = counted_traffic(w.name, dom)
    roofline = {"bound": bound, "kernel": dom, "achieved": round(achieved, 3), "peak": peak,
                "unit": unit, "frac": round(achieved / peak, 4), "traffic": traffic,
                "avg_launch_ms": round(avg_ms, 4), "launches": dv["launches"],
                "algorithmic_bytes_per_launch": dv["bytes"] / dv["launches"],
                "algorithmic_flops_per_launch": dv["flops"] / dv["launches"]}

    def branch(ms_list, count):
        if not ms_list:
            return {"count": 0}
        med = float(np.median(ms_list))
        return {"count": count, "median_ms": round(med, 4),
                "p10_ms": round(float(np.percentile(ms_list, 10)), 4),
                "p90_ms": round(float(np.percentile(ms_list, 90)), 4),
                "min_ms": round(min(ms_list), 4), "max_ms": round(max(ms_list), 4),
                "params_per_s": w.params / (med * 1e-3)}

    branches = {"sync": branch(sync_ms, n_sync), "local": branch(local_ms, n_local)}
    counted = counted_step_bytes(w.name)
    # compulsory bytes per step: read G, M, X and write M, X; a sync step also
    # reads and writes Q (n x r per layer)
    gb = 2 if w.grad_dtype == "bf16" else 4
    skip_bytes = (16 + gb) * w.params
    sync_bytes = skip_bytes + 8 * sum(n * w.r for _, n in w.shapes)
    for name, nbytes in (("local", skip_bytes), ("sync", sync_bytes)):
        if branches[name]["count"]:
            t_med = branches[name]["median_ms"] * 1e-3
            gbps = nbytes / t_med / 1e9
            branches[name]["compulsory_bytes"] = nbytes
            branches[name]["algorithmic_GBps"] = gbps
            branches[name]["algorithmic_frac_of_hbm_peak"] = gbps / PEAK_HBM_GBPS
            # hardware-counted bytes of such a step (FETCH_SIZE + WRITE_SIZE,
            # profiles/), null when the kernels changed since they were counted
            cb = counted.get(name)
            branches[name]["counted_bytes"] = cb
            branches[name]["counted_GBps"] = cb / t_med / 1e9 if cb else None
    if branches["sync"]["count"]:
        # a sync step is MFMA work: the method's flops (P~ = BQ, R = B^T P and
        # the rank-r M and X corrections, 8 r flops per parameter, plus two
        # CholQR passes of 2 m r^2 + r^3 / 3 each), and, as a model (not a
        # counter), the time the executed MFMA products (every bf16 piece
        # product at the bf16 peak, fp64 products at the fp64 peak) would need
        # at the published peaks, as a fraction of the step; the counted MFMA
        # busy fraction per kernel is in profiles/
        t_sync = branches["sync"]["median_ms"] * 1e-3
        alg = sum(8.0 * w.r * m * n + 2.0 * (2.0 * m * w.r ** 2 + w.r ** 3 / 3.0) for m, n in w.shapes)
        executed = {}
        for k in kt:
            bound, prec, mult = KIND_BOUND.get(k, ("hbm", None, 1))
            if bound == "mfma":
                executed[prec] = executed.get(prec, 0.0) + mult * kt[k]["flops"] / n_sync
        busy = sum(f / (PEAK_TFLOPS[prec] * 1e12) for prec, f in executed.items())
        branches["sync"].update(algorithmic_flops=alg, algorithmic_TFLOPs=alg / t_sync / 1e12,
                                executed_mfma_flops={p: f for p, f in executed.items()},
                                executed_TFLOPs={p: f / t_sync / 1e12 for p, f in executed.items()},
                                executed_frac_of_peak={p: f / t_sync / 1e12 / PEAK_TFLOPS[p]
                                                       for p, f in executed.items()},
                                mfma_time_model_frac=busy / t_sync)

    cpu = None
    if not args.no_cpu_baseline:
        log("[bench] timing the float64 oracle on a bounded sample ...")
        cpu = cpu_baseline(w, n_sync, n_local, K)
        log(f"[bench] oracle: {cpu['value']:.3e} params/s on {cpu['cores']} cores")

    value = w.params * K / elapsed
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "params/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": W,
        "ms_per_step": elapsed * 1e3 / K,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # the contractions of bf16-gradient layers run on the bf16 MFMA (split
        # fp32 operands for the power iteration, plain bf16 for the rank-r
        # update); fp32-gradient layers compute in fp32 and fp64
        "dtype": "bf16" if w.grad_dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"{w.name}: {L} matrices of the 1.3B-shaped GPT set (d_model 2048, 24 blocks)"
                         if w.name == "gpt1p3b" else w.name),
            "workload_name": w.name,
            "params": w.params, "rank": w.r, "grad_dtype": w.grad_dtype, "state_dtype": "f32",
            "power_iteration_dtype": ("P~ = BQ and R = B^T P on bf16 MFMA with 2-piece fp32 splits "
                                      "(3 products, ~2^-16 relative); CholQR2 pass 0: Gram exact to fp64 "
                                      "accumulation (3 bf16 slices per value, 9 products on bf16 MFMA) and "
                                      "Cholesky in fp64, pass 1 fp32-accurate (bf16 x 6); M/X update bf16 "
                                      "products, fp32 accumulation" if w.grad_dtype == "bf16" else
                                      "P~ = BQ, R = B^T P, Gram and CholQR in fp64; the M/X update on bf16 "
                                      "MFMA with 3-piece fp32 splits (fp32 vector units at r <= 32)"),
            "policy": args.policy + (f" (H = {args.H})" if args.policy == "every_h" else ""),
            "steps_mode": "asynchronous (no host read per step)" if asyn else "blocking (gate read per step)",
            "tau": w.tau, "trajectory_steps": K,
            "sync_steps": n_sync, "local_steps": n_local, "parallelism": "none (1 GPU)",
            "inputs": (f"gradients drawn on the GPU between steps, outside each step's timed interval"
                       if streamed else f"{pool} gradient sets resident in HBM, cycled"),
        },
        # whole trajectory: compulsory bytes (algorithmic) and, where the
        # committed counter summary matches the sources, counted bytes
        "algorithmic_GBps": (n_sync * sync_bytes + n_local * skip_bytes) / elapsed / 1e9,
        "counted_GBps": ((n_sync * counted["sync"] if n_sync else 0.0) +
                         (n_local * counted["local"] if n_local else 0.0)) / elapsed / 1e9
        if (not n_sync or "sync" in counted) and (not n_local or "local" in counted) else None,
        "branches": branches,
        "roofline": roofline,
        "kernels_profiling_pass": {k: {"launches": v["launches"], "total_ms": round(v["total_ms"], 4)}
                                   for k, v in kt.items()},
        "rmmc_trace": [None if (isinstance(x, float) and math.isnan(x)) else x for x in rmmcs],
        "cpu_baseline": cpu,
        # the command line of this run (the profile summaries quote it)
        "command": " ".join(["python3", "bench.py"] + [shlex.quote(a) for a in sys.argv[1:]]),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
