"""Summaries of rocprofv3 output for the codec kernels.

  python -m paper_2608_04991_amd.rocprof_summary stats DIR OUT.txt "COMMAND" [LAST]
      kernel-trace statistics (calls, average and total duration per kernel)
      of a `rocprofv3 --kernel-trace --stats --output-format csv` run; with
      LAST, also the average of the last LAST dispatches of each codec
      kernel (bench.py ends with LAST back-to-back launches of each, the
      run its per-kernel HIP-event durations come from).

  python -m paper_2608_04991_amd.rocprof_summary traffic KERNEL FETCH_DIR WRITE_DIR \
         COPY_FETCH_DIR COPY_WRITE_DIR COPY_BYTES OUT.json "COMMANDS"
      HBM bytes per launch of KERNEL from two `--pmc` runs (FETCH_SIZE, then
      WRITE_SIZE, both in KiB per dispatch), each scaled by what the same
      counter reads for a plain device copy of COPY_BYTES (the copy kernel of
      the HIP runtime), so that the counters are calibrated on this machine.
      The output records a hash of the kernel source it was measured on.
"""
from __future__ import annotations

import csv
import glob
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCE = os.path.join(HERE, "csrc", "rac.hip")
COPY_KERNEL = "__amd_rocclr_copyBuffer"


def source_hash() -> str:
    return hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()[:16]


def _one(pattern: str) -> str:
    files = sorted(glob.glob(pattern, recursive=True))
    if not files:
        raise FileNotFoundError(pattern)
    return files[0]


def stats(dirpath: str, out: str, command: str, last: int = 0) -> None:
    rows = list(csv.DictReader(open(_one(os.path.join(dirpath, "**", "*kernel_stats.csv")))))
    lines = [f"# rocprofv3 kernel-trace statistics", f"# command: {command}", "",
             f"{'calls':>6} {'avg_us':>10} {'min_us':>10} {'max_us':>10} {'total_us':>12} {'pct':>6}  kernel"]
    for r in rows:
        ns = lambda k: float(r[k]) / 1e3
        lines.append(f"{int(r['Calls']):>6} {ns('AverageNs'):>10.2f} {ns('MinNs'):>10.2f} "
                     f"{ns('MaxNs'):>10.2f} {ns('TotalDurationNs'):>12.1f} {float(r['Percentage']):>6.2f}  "
                     f"{r['Name'][:110]}")
    if last:
        trace = list(csv.DictReader(open(_one(os.path.join(dirpath, "**", "*kernel_trace.csv")))))
        lines += ["", f"# last {last} dispatches of each codec kernel (back to back)",
                  f"{'calls':>6} {'avg_us':>10} {'span_us':>10}  kernel"]
        names = sorted({t["Kernel_Name"] for t in trace if "rac_" in t["Kernel_Name"]})
        for name in names:
            ds = [t for t in trace if t["Kernel_Name"] == name][-last:]
            dur = [(int(t["End_Timestamp"]) - int(t["Start_Timestamp"])) / 1e3 for t in ds]
            span = (int(ds[-1]["End_Timestamp"]) - int(ds[0]["Start_Timestamp"])) / 1e3 / len(ds)
            lines.append(f"{len(ds):>6} {sum(dur) / len(dur):>10.2f} {span:>10.2f}  {name[:110]}")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter_avg(dirpath: str, counter: str, match: str) -> float:
    rows = list(csv.DictReader(open(_one(os.path.join(dirpath, "**", "*counter_collection.csv")))))
    vals = [float(r["Counter_Value"]) for r in rows
            if r["Counter_Name"] == counter and match in r["Kernel_Name"]]
    if not vals:
        raise ValueError(f"no {counter} samples for {match} in {dirpath}")
    return sum(vals) / len(vals)


def traffic(kernel, fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, copy_bytes, out, commands):
    copy_bytes = float(copy_bytes)
    f_kib = _counter_avg(fetch_dir, "FETCH_SIZE", kernel)
    w_kib = _counter_avg(write_dir, "WRITE_SIZE", kernel)
    cf_kib = _counter_avg(copy_fetch_dir, "FETCH_SIZE", COPY_KERNEL)
    cw_kib = _counter_avg(copy_write_dir, "WRITE_SIZE", COPY_KERNEL)
    f_scale = copy_bytes / (cf_kib * 1024.0)
    w_scale = copy_bytes / (cw_kib * 1024.0)
    res = {
        "kernel": kernel,
        "fetch_bytes_per_launch": f_kib * 1024.0 * f_scale,
        "write_bytes_per_launch": w_kib * 1024.0 * w_scale,
        "bytes_per_launch": f_kib * 1024.0 * f_scale + w_kib * 1024.0 * w_scale,
        "raw_fetch_kib": f_kib, "raw_write_kib": w_kib,
        "copy_bytes": copy_bytes, "copy_fetch_kib": cf_kib, "copy_write_kib": cw_kib,
        "fetch_scale": f_scale, "write_scale": w_scale,
        "kernel_source_sha256_16": source_hash(),
        "commands": commands,
    }
    json.dump(res, open(out, "w"), indent=1)
    print(json.dumps(res, indent=1))


if __name__ == "__main__":
    if sys.argv[1] == "stats":
        stats(*sys.argv[2:5], *(int(a) for a in sys.argv[5:6]))
    elif sys.argv[1] == "traffic":
        traffic(*sys.argv[2:10])
    else:
        raise SystemExit(__doc__)
