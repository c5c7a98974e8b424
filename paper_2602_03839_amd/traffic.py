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
    try:
        with open(path) as fh:
            kv = dict(line.split(":", 1) for line in fh if ":" in line and not line.startswith("#"))
    except OSError:
        return None
    kv = {k.strip(): v.strip() for k, v in kv.items()}
    if kv.get("source_hash") != kernel_source_hash():
        return None
    try:
        return float(kv["traffic_bytes_per_launch"])
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


def main():
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
