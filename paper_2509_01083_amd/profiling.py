"""Summaries of rocprofv3 output for the statistics kernel's roofline.

Turns a ``--kernel-trace --stats`` run and two ``--pmc`` runs (FETCH_SIZE, then
WRITE_SIZE) of ``bench.py --copy-calibration`` into

* ``traffic.json``: HBM bytes per launch of the row-statistics kernel, each
  counter scaled by what it reads for a streaming kernel of known size
  (bitwise_not over 1 GiB: 1 GiB read, 1 GiB written), tagged with the hash of
  the kernel sources it was measured on (bench.py drops it once they change);
* a short markdown summary with the per-kernel durations and the counters.

    python -m paper_2509_01083_amd.profiling --trace DIR --fetch CSV --write CSV \\
        --workload b256 --json profiles/traffic.json --md profiles/stats_kernel_bf16_b256.md \\
        --command "<the commands that produced the inputs>"
"""
import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KERNEL = "stats_kernel_bf16"
CALIBRATION_KERNEL = "bitwise_not"
CALIBRATION_BYTES = 1 << 30


STEP_SOURCES = ("stats.hip", "verify.hip", "signal.hip", "row_io.hpp", "common.hpp", "draw_device.hpp",
                "signal_device.hpp", "lanes.hpp")


def kernel_source_hash(files=("stats.hip", "row_io.hpp", "common.hpp")):
    """Hash of the sources the statistics kernel (by default) is built from."""
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2509_01083_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def step_source_hash():
    """Hash of the sources of every kernel of the verification step."""
    return kernel_source_hash(STEP_SOURCES)


def short_name(name):
    m = re.search(r"dsde::\(anonymous namespace\)::(\w+)(<[^>(]*>)?", name)
    if m:
        return m.group(1) + (m.group(2) or "")
    if CALIBRATION_KERNEL in name:
        return CALIBRATION_KERNEL
    return None


def counter_values(path, counter):
    """Per-dispatch values of `counter` (KiB) for the library's kernels and the calibration kernel."""
    out = collections.defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            k = short_name(r["Kernel_Name"])
            if k:
                out[k].append(float(r["Counter_Value"]))
    return out


def trace_stats(trace_dir):
    path = glob.glob(os.path.join(trace_dir, "*kernel_stats.csv"))[0]
    rows = []
    with open(path) as f:
        for r in csv.DictReader(f):
            k = short_name(r["Name"])
            if k and k != CALIBRATION_KERNEL:
                rows.append((k, int(r["Calls"]), float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
                             float(r["MaxNs"]) / 1e3))
    return rows


def is_stats(k):
    """The bf16 statistics kernel, in either form (with or without the draft
    entropy accumulator)."""
    return k == KERNEL or k.startswith(KERNEL + "<")


def stats_key(d):
    """The statistics kernel's name among the keys of d (the form with the most
    dispatches when both ran)."""
    keys = [k for k in d if is_stats(k)]
    return max(keys, key=lambda k: len(d[k])) if keys else None


def median(v):
    v = sorted(v)
    return v[len(v) // 2]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", required=True)
    ap.add_argument("--fetch", help="FETCH_SIZE counter CSV (omitted: durations only)")
    ap.add_argument("--write", help="WRITE_SIZE counter CSV")
    ap.add_argument("--workload", default="b256")
    ap.add_argument("--algorithmic-bytes", type=float)
    ap.add_argument("--step-algorithmic-bytes", type=float, help="(2N + B_full) V e + I/O of the step")
    ap.add_argument("--json", help="traffic file to write (needs the counters)")
    ap.add_argument("--md", required=True)
    ap.add_argument("--command", action="append", default=[])
    ap.add_argument("--bench-log", help="output of bench.py run without the profiler (its last line is the JSON)")
    ap.add_argument("--title", help="heading of the summary (default: the statistics kernel and the workload)")
    ap.add_argument("--counter", action="append", default=[],
                    help="NAME=CSV: a --pmc run of one counter, tabulated per kernel (mean over dispatches)")
    ap.add_argument("--elements", type=float,
                    help="element pairs one launch of the statistics kernel processes (for VALU per element)")
    a = ap.parse_args()
    bench = None
    if a.bench_log:
        with open(a.bench_log) as f:
            bench = json.loads(f.read().strip().splitlines()[-1])
    cfg = bench["config"] if bench else {}
    shape = ", ".join(f"{k}={cfg[k]}" for k in ("B", "N", "V") if k in cfg)
    title = a.title or f"{KERNEL}, workload {a.workload}"
    lines = [f"# {title}" + (f" ({shape}, bf16)" if shape else ""), "",
             "Commands (from the repository root):", ""]
    lines += [f"    {c}" for c in a.command]
    lines += ["", "## Kernel durations (rocprofv3 --kernel-trace --stats)", "",
              "| kernel | calls | avg us | min us | max us |", "|---|---|---|---|---|"]
    for k, n, avg, lo, hi in trace_stats(a.trace):
        lines.append(f"| {k} | {n} | {avg:.2f} | {lo:.2f} | {hi:.2f} |")
    if a.counter:
        names = [c.split("=", 1)[0] for c in a.counter]
        vals = {n: counter_values(c.split("=", 1)[1], n) for n, c in zip(names, a.counter)}
        kernels = sorted(set().union(*(set(v) for v in vals.values())) - {CALIBRATION_KERNEL})
        lines += ["", "## Counters (rocprofv3 --pmc, one counter per run; mean over each kernel's dispatches)", "",
                  "| kernel | " + " | ".join(names) + " |", "|---|" + "---|" * len(names)]
        for k in kernels:
            cells = []
            for n in names:
                v = vals[n].get(k)
                cells.append(f"{sum(v) / len(v):,.1f}" if v else "")
            lines.append(f"| {k} | " + " | ".join(cells) + " |")
        sk = stats_key(vals["SQ_INSTS_VALU"]) if "SQ_INSTS_VALU" in vals else None
        if a.elements and sk:
            v = vals["SQ_INSTS_VALU"][sk]
            per = sum(v) / len(v) / a.elements * 64
            lines += ["", f"{sk}: {a.elements:,.0f} element pairs per launch, {per:.1f} VALU wave "
                      "instructions per 64 element pairs."]
    if not (a.fetch and a.write):
        if bench and "loop" in bench:
            lp = bench["loop"]
            lines += ["", "## Controller loop (bench.py without the profiler)", "",
                      f"Per step: mean {lp['ms_per_step']['mean'] * 1e3:.1f} us, median "
                      f"{lp['ms_per_step']['median'] * 1e3:.1f} us, p95 {lp['ms_per_step']['p95'] * 1e3:.1f} us; "
                      f"mean SL {lp['mean_sl']['mean']:.2f}; cap {lp['sl_cap']['mean']:.2f}; "
                      f"{lp['fraction_in_sl_min_branch'] * 100:.0f}% of sequences in the SL_min branch; "
                      f"{bench['value'] / 1e6:.2f} M rows/s over all steps.", ""]
        with open(a.md, "w") as f:
            f.write("\n".join(lines))
        return
    fetch = counter_values(a.fetch, "FETCH_SIZE")
    write = counter_values(a.write, "WRITE_SIZE")
    f_cal = median(fetch[CALIBRATION_KERNEL]) * 1024 / CALIBRATION_BYTES
    w_cal = median(write[CALIBRATION_KERNEL]) * 1024 / CALIBRATION_BYTES
    sk = stats_key(fetch)
    f_k = median(fetch[sk]) * 1024 / f_cal
    w_k = median(write[sk]) * 1024 / w_cal
    traffic = {"workload": a.workload, "kernel": sk, "kernel_source_hash": kernel_source_hash(),
               "fetch_bytes_per_launch": f_k, "write_bytes_per_launch": w_k, "bytes_per_launch": f_k + w_k,
               "fetch_counter_scale": 1.0 / f_cal, "write_counter_scale": 1.0 / w_cal,
               "algorithmic_bytes": a.algorithmic_bytes}
    # every kernel of the step (one launch each per step), for the step's traffic
    step = {}
    for k in sorted(set(fetch) & set(write)):
        if k in (CALIBRATION_KERNEL, "stream_read_kernel"):
            continue
        step[k] = {"fetch_bytes": median(fetch[k]) * 1024 / f_cal, "write_bytes": median(write[k]) * 1024 / w_cal}
    traffic["step_source_hash"] = step_source_hash()
    traffic["step_kernels"] = step
    traffic["step_bytes"] = sum(v["fetch_bytes"] + v["write_bytes"] for v in step.values())
    if a.json:
        with open(a.json, "w") as f:
            json.dump(traffic, f, indent=1)
            f.write("\n")
    lines += ["", "## HBM traffic per launch (rocprofv3 --pmc, one counter per run)", "",
              f"Calibration: {CALIBRATION_KERNEL} over 1 GiB reads FETCH_SIZE = "
              f"{median(fetch[CALIBRATION_KERNEL]):.0f} KiB and WRITE_SIZE = {median(write[CALIBRATION_KERNEL]):.0f} KiB "
              f"per launch, i.e. scale factors {1 / f_cal:.4f} (fetch) and {1 / w_cal:.4f} (write).", "",
              "| kernel | FETCH_SIZE KiB (raw) | WRITE_SIZE KiB (raw) | scaled MB read | scaled MB written |",
              "|---|---|---|---|---|"]
    for k in sorted(set(fetch) & set(write)):
        if k == CALIBRATION_KERNEL:
            continue
        fr, wr = median(fetch[k]), median(write[k])
        lines.append(f"| {k} | {fr:.0f} | {wr:.0f} | {fr * 1024 / f_cal / 1e6:.2f} | {wr * 1024 / w_cal / 1e6:.3f} |")
    if bench:
        r = bench
        ev_us = r["roofline"]["kernel_ms"] * 1e3
        tr_us = [avg for k, _, avg, _, _ in trace_stats(a.trace) if k == sk][0]
        lines += ["", "## HIP events against the trace", "",
                  f"bench.py run without the profiler on the same box: {sk} timed with HIP events "
                  f"{ev_us:.2f} us per launch over {r['steps']} steps (the roofline's `achieved` "
                  f"{r['roofline']['achieved']:.0f} GB/s); the trace above: {tr_us:.2f} us "
                  f"({(ev_us / tr_us - 1) * 100:+.1f}%). Step: {r['ms_per_step'] * 1e3:.2f} us, "
                  f"{r['value'] / 1e6:.2f} M rows/s. Under rocprofv3 each attached completion event "
                  "opens a gap of about 4.6 us before the next kernel, so the figure bench.py prints inside the "
                  "profiled process includes that gap."]
    lines += ["", f"{sk}: {traffic['bytes_per_launch'] / 1e6:.2f} MB per launch measured against "
              f"{a.algorithmic_bytes / 1e6:.2f} MB algorithmic "
              f"({traffic['bytes_per_launch'] / a.algorithmic_bytes:.4f}x).", ""]
    if bench and a.step_algorithmic_bytes:
        lines += [f"Step (every kernel above once): {traffic['step_bytes'] / 1e6:.2f} MB per step measured "
                  f"against {a.step_algorithmic_bytes / 1e6:.2f} MB algorithmic "
                  f"({traffic['step_bytes'] / a.step_algorithmic_bytes:.4f}x).", ""]
    with open(a.md, "w") as f:
        f.write("\n".join(lines))


if __name__ == "__main__":
    main()
