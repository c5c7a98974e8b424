"""HBM traffic of the fused encode kernel from rocprofv3 counter runs.

Two counter-collection runs of ``bench.py`` (one with FETCH_SIZE, one with
WRITE_SIZE; the counters cannot share a pass) give kilobytes per dispatch.
Each counter is calibrated against the plain copy kernel that bench.py runs
once before timing (bitwise_not over 1 GiB of int32: 1 GiB read, 1 GiB
written), and the calibrated bytes of the first step's fused encode launches
are written, with the hash of the kernel sources they were taken on, to a
short text summary that bench.py reads back: a figure taken on other sources
is not reported.

    python -m paper_2602_03839_amd.traffic --fetch DIR --write DIR --bench-json FILE --out FILE
    python -m paper_2602_03839_amd.traffic kernels --dir DIR [--dir DIR ...] --out FILE
    python -m paper_2602_03839_amd.traffic stats --stats-csv FILE --bench-json FILE --out FILE

The second form tabulates every library kernel's counters per dispatch (any
counters, one directory per counter pass), with mean durations.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os

HERE = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = ("encode.hip", "device_common.hpp", "launch.hpp")
CALIB_KERNEL = "bitwise_not"
CALIB_BYTES = (1 << 28) * 4  # read, and written, by the calibration kernel


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(HERE, "csrc", name), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def read_summary(path: str):
    """traffic_bytes_per_launch from a summary, or None if missing or taken on other sources."""
    split = read_summary_split(path)
    return None if split is None else split[0] + split[1]


def read_summary_split(path: str):
    """(fetch_bytes_per_launch, write_bytes_per_launch) from a summary, or None if
    missing or taken on other sources."""
    try:
        with open(path) as fh:
            kv = dict(line.split(":", 1) for line in fh if ":" in line and not line.startswith("#"))
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("source_hash") != kernel_source_hash():
        return None
    try:
        return float(kv["fetch_bytes_per_launch"]), float(kv["write_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _rows(directory: str, counter: str):
    files = glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {directory}")
    out = []
    for f in files:
        with open(f, newline="") as fh:
            for r in csv.DictReader(fh):
                if r.get("Counter_Name") == counter:
                    out.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
    out.sort()
    return out


def _measure(directory: str, counter: str, n_launch: int):
    rows = _rows(directory, counter)
    calib = [v for _, k, v in rows if CALIB_KERNEL in k]
    enc = [v for _, k, v in rows if "encode_kernel" in k and "true>" in k][:n_launch]
    if not calib or len(enc) < n_launch:
        raise SystemExit(f"{counter}: calibration or encode dispatches missing in {directory}")
    scale = CALIB_BYTES / (calib[0] * 1024.0)
    return scale, sum(enc) * 1024.0, enc


def kernel_label(name: str) -> str:
    """Short kernel name: template arguments kept, namespace and parameters dropped."""
    n = name[5:] if name.startswith("void ") else name
    n = n.replace("pulse::", "").replace("(anonymous namespace)::", "")
    depth, cut = 0, len(n)
    for i, ch in enumerate(n):  # the parameter list is the first '(' outside template brackets
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            cut = i
            break
    return n[:cut]


def kernel_table(dirs, counters_wanted=None, match="pulse|bitwise_not"):
    """Per kernel: dispatches, mean duration and the mean of every counter per
    dispatch over the counter-collection runs in `dirs` (FETCH_SIZE and
    WRITE_SIZE in bytes, calibrated on the copy kernel; other counters raw)."""
    import re
    per = {}   # label -> counter -> [values]
    dur = {}   # label -> [ns]
    scale = {}
    for d in dirs:
        files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        for f in files:
            with open(f, newline="") as fh:
                rows = list(csv.DictReader(fh))
            calib = {}
            for r in rows:
                if CALIB_KERNEL in r["Kernel_Name"] and r["Counter_Name"] in ("FETCH_SIZE", "WRITE_SIZE"):
                    calib.setdefault(r["Counter_Name"], float(r["Counter_Value"]))
            for c, v in calib.items():
                scale[c] = CALIB_BYTES / (v * 1024.0)
            for r in rows:
                if not re.search(match, r["Kernel_Name"]):
                    continue
                lab = kernel_label(r["Kernel_Name"])
                c = r["Counter_Name"]
                if counters_wanted and c not in counters_wanted:
                    continue
                v = float(r["Counter_Value"])
                if c in ("FETCH_SIZE", "WRITE_SIZE"):
                    v = v * 1024.0 * scale.get(c, 1.0)
                per.setdefault(lab, {}).setdefault(c, []).append(v)
                try:
                    dur.setdefault(lab, {})[(f, r["Dispatch_Id"])] = (
                        int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
                except (KeyError, ValueError):
                    pass
    return per, dur, scale


def kernels_main(argv):
    ap = argparse.ArgumentParser(prog="traffic kernels",
                                 description="per-kernel counter table from rocprofv3 --pmc runs")
    ap.add_argument("--dir", action="append", required=True, help="a counter-collection output directory")
    ap.add_argument("--out", required=True)
    ap.add_argument("--title", default="per-kernel counters")
    ap.add_argument("--command", action="append", default=[], help="commands that made the runs")
    args = ap.parse_args(argv)
    per, dur, scale = kernel_table(args.dir)
    counters = sorted({c for v in per.values() for c in v})
    lines = [f"# {args.title}", "",
             "Mean per dispatch; FETCH_SIZE / WRITE_SIZE in bytes, each calibrated on the copy kernel "
             "(bitwise_not over 1 GiB: 1 GiB read, 1 GiB written) of the same run "
             f"(factors {', '.join(f'{k} {v:.4f}' for k, v in sorted(scale.items()))}); other counters raw.",
             ""]
    for c in args.command:
        lines.append(f"    {c}")
    lines += ["", "| kernel | dispatches | mean duration (us) | " + " | ".join(counters) + " |",
              "|---|---|---|" + "---|" * len(counters)]
    for lab in sorted(per):
        vals = per[lab]
        nd = max(len(v) for v in vals.values())
        ds = list(dur.get(lab, {}).values())
        md = sum(ds) / len(ds) / 1e3 if ds else float("nan")
        cells = []
        for c in counters:
            v = vals.get(c)
            cells.append(f"{sum(v) / len(v):.4g}" if v else "")
        lines.append(f"| {lab} | {nd} | {md:.1f} | " + " | ".join(cells) + " |")
    with open(args.out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def stats_main(argv):
    """Markdown summary of a rocprofv3 --kernel-trace --stats run of bench.py:
    the library's kernels, and the headline kernel's average beside the
    benchmark's own event timing of the same run."""
    import re
    ap = argparse.ArgumentParser(prog="traffic stats")
    ap.add_argument("--stats-csv", required=True, help="the run's *_kernel_stats.csv")
    ap.add_argument("--bench-json", required=True, help="file holding the JSON line bench.py printed")
    ap.add_argument("--out", required=True)
    ap.add_argument("--trace-csv", help="the run's *_kernel_trace.csv (per-dispatch durations)")
    ap.add_argument("--command", action="append", default=[], help="commands that made the run")
    args = ap.parse_args(argv)
    with open(args.stats_csv, newline="") as fh:
        rows = list(csv.DictReader(fh))
    with open(args.bench_json) as fh:
        d = json.loads([line for line in fh if line.startswith("{")][-1])
    keep = re.compile(r"pulse::|bitwise_not|read2_kernel|rmw_kernel|_oneshot")
    out = ["# rocprofv3 kernel stats of one bench.py run", ""]
    out += ["Commands (repository root as the working directory):", "```"] + args.command + ["```", ""]
    out += ["| Kernel | Calls | Avg (ms) | Min (ms) | Max (ms) | Total (ms) |", "|---|---|---|---|---|---|"]
    for r in rows:
        if not keep.search(r["Name"]):
            continue
        name = "torch bitwise_not over 2^28 int32 (counter calibration copy)" if "bitwise_not" in r["Name"] \
            else kernel_label(r["Name"]).replace("(anonymous namespace)::", "")
        out.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e6:.4f} | "
                   f"{float(r['MinNs']) / 1e6:.4f} | {float(r['MaxNs']) / 1e6:.4f} | "
                   f"{float(r['TotalDurationNs']) / 1e6:.2f} |")
    rf = d["roofline"]
    out += ["", f"bench.py line of this run: fused step {d['ms_per_step']:.3f} ms; HIP events around each step's "
                f"{d['config']['launches_per_step']} launches give an average launch of {rf['avg_launch_ms']:.4f} ms, "
                f"{rf['achieved']:.1f} GB/s = {100 * rf['frac']:.1f}% of 8 TB/s."]
    if args.trace_csv:
        # the headline's dispatches are the first refresh-form encode launches
        # of the run: warm-up steps, then the timed ones
        with open(args.trace_csv, newline="") as fh:
            tr = [r for r in csv.DictReader(fh) if re.search(r"encode_kernel<\d+, \d+, true>", r["Kernel_Name"])]
        tr.sort(key=lambda r: int(r["Dispatch_Id"]))
        nl = int(d["config"]["launches_per_step"])
        first = int(d["warmup"]) * nl
        timed = tr[first:first + int(d["steps"]) * nl]
        if timed:
            a = sum(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in timed) / len(timed) / 1e6
            out.append(f"rocprofv3 trace, the headline's timed dispatches of `{kernel_label(timed[0]['Kernel_Name'])}` "
                       f"(dispatches {first + 1}-{first + len(timed)} of that kernel in this run): average {a:.4f} ms, "
                       f"{100 * abs(a - rf['avg_launch_ms']) / rf['avg_launch_ms']:.1f}% from the events' "
                       f"{rf['avg_launch_ms']:.4f} ms.  (The stats row above averages that kernel over every leg "
                       f"that uses it: the in-place, std-reading, one-tensor, 0.5B and 7B-chain legs too.)")
    out += ["", "Launch sizes differ within a step (the last batch of a step holds fewer tensors), so Min/Max span "
                "the batch sizes.  Kernels outside the library (torch's input generators) are left out."]
    with open(args.out, "w") as fh:
        fh.write("\n".join(out) + "\n")
    print("\n".join(out))


def main():
    import sys
    if len(sys.argv) > 1 and sys.argv[1] == "kernels":
        kernels_main(sys.argv[2:])
        return
    if len(sys.argv) > 1 and sys.argv[1] == "stats":
        stats_main(sys.argv[2:])
        return
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--fetch", required=True, help="output directory of the FETCH_SIZE run")
    ap.add_argument("--write", required=True, help="output directory of the WRITE_SIZE run")
    ap.add_argument("--bench-json", required=True, help="the JSON line bench.py printed in one of the runs")
    ap.add_argument("--out", required=True)
    ap.add_argument("--command", action="append", default=[], help="commands that made the runs")
    args = ap.parse_args()

    with open(args.bench_json) as fh:
        bench = json.loads([line for line in fh if line.startswith("{")][-1])
    n_launch = int(bench["config"]["launches_per_step"])
    alg = float(bench["roofline"]["bytes_per_launch"])
    fs, fraw, fl = _measure(args.fetch, "FETCH_SIZE", n_launch)
    wsc, wraw, wl = _measure(args.write, "WRITE_SIZE", n_launch)
    fetch = fraw * fs / n_launch
    write = wraw * wsc / n_launch
    lines = [
        "# HBM traffic of encode_kernel (refresh form), fused encode+refresh, "
        f"{bench['config']['workload']}, {bench['config']['params']:,} params",
        "# rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE, KiB per dispatch, calibrated on a plain copy kernel",
        *[f"# command: {c}" for c in args.command],
        "# summary: python3 -m paper_2602_03839_amd.traffic " + " ".join(
            f"--{k.replace('_', '-')} {v}" for k, v in (("fetch", args.fetch), ("write", args.write),
                                                          ("bench_json", args.bench_json), ("out", args.out))),
        f"source_hash: {kernel_source_hash()}",
        f"launches_per_step: {n_launch}",
        f"fetch_calibration_factor: {fs:.4f}",
        f"write_calibration_factor: {wsc:.4f}",
        f"fetch_bytes_per_launch: {fetch:.0f}",
        f"write_bytes_per_launch: {write:.0f}",
        f"traffic_bytes_per_launch: {fetch + write:.0f}",
        f"algorithmic_bytes_per_launch: {alg:.0f}",
        f"traffic_over_algorithmic: {(fetch + write) / alg:.4f}",
        f"fetch_kib_per_dispatch: {' '.join(f'{v:.0f}' for v in fl)}",
        f"write_kib_per_dispatch: {' '.join(f'{v:.0f}' for v in wl)}",
    ]
    with open(args.out, "w") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


if __name__ == "__main__":
    main()
