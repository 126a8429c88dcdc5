"""Summaries of rocprofv3 output for the codec kernels.

  python -m paper_2608_04991_amd.rocprof_summary stats DIR OUT.txt "COMMAND" [LAST]
      kernel-trace statistics (calls, average and total duration per kernel)
      of a `rocprofv3 --kernel-trace --stats --output-format csv` run; with
      LAST, also the average of the last LAST dispatches of each codec
      kernel (the bench's timed steps end the encode kernel's dispatches when
      it runs without extras).

  python -m paper_2608_04991_amd.rocprof_summary blocks DIR MIN OUT.txt "COMMAND" [LABELS.json]
      the same trace split into blocks: every maximal run of at least MIN
      consecutive dispatches of one codec kernel (bench.py --profile launches
      each configuration's encodes back to back, then its decodes), with the
      block's average duration, workgroup count and the label of the
      configuration (LABELS.json: the bench's --profile output, whose
      configurations appear in launch order, two blocks each, or a list).

  python -m paper_2608_04991_amd.rocprof_summary merged DIR MIN OUT.txt "COMMAND" LABELS.json
      the blocks as above, merged by label (the launch-shape sweep repeats
      each configuration's blocks): per label the number of blocks, the
      median of their average durations, the range of those averages and
      the workgroup count.

  python -m paper_2608_04991_amd.rocprof_summary grids DIR SUBSTR OUT.txt "COMMAND"
      per-shape statistics of the kernels whose name holds SUBSTR: one line
      per (kernel, workgroup count), for kernels that interleave with others
      (each launch of a multi-kernel step has its own grid).

  python -m paper_2608_04991_amd.rocprof_summary traffic FETCH_DIR WRITE_DIR \
         COPY_FETCH_DIR COPY_WRITE_DIR COPY_BYTES MIN OUT.json "COMMANDS" [LABELS.json]
      HBM bytes per launch of every block (as above) from two `--pmc` runs of
      the same command (FETCH_SIZE, then WRITE_SIZE, both in KiB per
      dispatch), each scaled by what the same counter reads for a plain
      device copy of COPY_BYTES (the HIP runtime's copy kernel), so the
      counters are calibrated on this machine.  The output records a hash of
      the kernel source it was measured on.
"""
from __future__ import annotations

import csv
import glob
import hashlib
import json
import os
import sys
from collections import defaultdict

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


def _codec(name: str) -> bool:
    return "rac_" in name


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
        lines += ["", f"# last {last} dispatches of each codec kernel",
                  f"{'calls':>6} {'avg_us':>10} {'span_us':>10}  kernel"]
        names = sorted({t["Kernel_Name"] for t in trace if _codec(t["Kernel_Name"])})
        for name in names:
            ds = [t for t in trace if t["Kernel_Name"] == name][-last:]
            dur = [(int(t["End_Timestamp"]) - int(t["Start_Timestamp"])) / 1e3 for t in ds]
            span = (int(ds[-1]["End_Timestamp"]) - int(ds[0]["Start_Timestamp"])) / 1e3 / len(ds)
            lines.append(f"{len(ds):>6} {sum(dur) / len(dur):>10.2f} {span:>10.2f}  {name[:110]}")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _labels(path):
    """Configuration labels in launch order: a list, or the bench's --profile
    output (its configuration keys in order, each giving an encode block and
    a decode block; a configuration whose entries are themselves per launch
    shape gives, per shape, `reps` encode and decode blocks in turn)."""
    if not path:
        return None
    d = json.load(open(path))
    if isinstance(d, list):
        return d
    reps = int(d.get("reps", 1))
    out = []
    for k, v in d.items():
        if isinstance(v, dict):
            if v and all(isinstance(x, dict) for x in v.values()):
                for shape in v:
                    out += [f"{k} {shape} encode", f"{k} {shape} decode"] * reps
            else:
                out += [f"{k} encode", f"{k} decode"]
    return out


def _runs(items, key, min_len):
    """Maximal runs of consecutive items with equal key(item), at least
    min_len long, of codec kernels; items are in dispatch order."""
    runs, cur = [], []
    for it in items:
        if cur and key(it) != key(cur[-1]):
            runs.append(cur)
            cur = []
        cur.append(it)
    if cur:
        runs.append(cur)
    return [r for r in runs if len(r) >= min_len and _codec(r[0]["name"])]


def _trace_dispatches(dirpath):
    trace = list(csv.DictReader(open(_one(os.path.join(dirpath, "**", "*kernel_trace.csv")))))
    out = []
    for t in sorted(trace, key=lambda t: int(t["Dispatch_Id"])):
        wg = int(t["Workgroup_Size_X"]) * int(t["Workgroup_Size_Y"]) * int(t["Workgroup_Size_Z"])
        grid = int(t["Grid_Size_X"]) * int(t["Grid_Size_Y"]) * int(t["Grid_Size_Z"])
        out.append(dict(name=t["Kernel_Name"], us=(int(t["End_Timestamp"]) - int(t["Start_Timestamp"])) / 1e3,
                        blocks=grid // max(wg, 1)))
    return out


def blocks(dirpath: str, min_len: str, out: str, command: str, labels: str = "") -> None:
    runs = _runs(_trace_dispatches(dirpath), lambda d: (d["name"], d["blocks"]), int(min_len))
    lab = _labels(labels)
    lines = ["# rocprofv3 kernel trace, blocks of back-to-back dispatches of one kernel",
             f"# command: {command}", "",
             f"{'block':>5} {'calls':>6} {'avg_us':>10} {'min_us':>10} {'max_us':>10} {'wgs':>6}  label / kernel"]
    for i, r in enumerate(runs):
        us = [d["us"] for d in r]
        tag = lab[i] if lab and i < len(lab) else ""
        lines.append(f"{i:>5} {len(r):>6} {sum(us) / len(us):>10.2f} {min(us):>10.2f} {max(us):>10.2f} "
                     f"{r[0]['blocks']:>6}  {tag} | {r[0]['name'][:100]}")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def merged(dirpath: str, min_len: str, out: str, command: str, labels: str) -> None:
    runs = _runs(_trace_dispatches(dirpath), lambda d: (d["name"], d["blocks"]), int(min_len))
    lab = _labels(labels)
    if len(lab) != len(runs):
        raise ValueError(f"{len(runs)} blocks in the trace but {len(lab)} labels")
    acc = {}
    for tag, r in zip(lab, runs):
        e = acc.setdefault(tag, dict(avgs=[], wgs=r[0]["blocks"], name=r[0]["name"]))
        if (r[0]["blocks"], r[0]["name"]) != (e["wgs"], e["name"]):
            raise ValueError(f"blocks labelled {tag!r} launched different kernels or grids")
        e["avgs"].append(sum(d["us"] for d in r) / len(r))
    kern = lambda n: n.split("(anonymous namespace)::", 1)[-1].split("(")[0]
    lines = ["# rocprofv3 kernel trace, blocks of back-to-back dispatches merged by label",
             f"# command: {command}", "",
             f"{'blocks':>6} {'median_us':>10} {'lo_us':>8} {'hi_us':>8} {'wgs':>6}  label | kernel"]
    for tag, e in acc.items():
        a = sorted(e["avgs"])
        lines.append(f"{len(a):>6} {a[len(a) // 2]:>10.2f} {a[0]:>8.2f} {a[-1]:>8.2f} {e['wgs']:>6}  "
                     f"{tag} | {kern(e['name'])}")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def grids(dirpath: str, substr: str, out: str, command: str) -> None:
    acc = defaultdict(list)
    for d in _trace_dispatches(dirpath):
        if substr in d["name"]:
            acc[(d["name"], d["blocks"])].append(d["us"])
    lines = ["# rocprofv3 kernel trace, per kernel and workgroup count", f"# command: {command}", "",
             f"{'calls':>6} {'avg_us':>10} {'median_us':>10} {'min_us':>10} {'wgs':>6}  kernel"]
    for (name, wgs), us in acc.items():
        u = sorted(us)
        lines.append(f"{len(u):>6} {sum(u) / len(u):>10.2f} {u[len(u) // 2]:>10.2f} {u[0]:>10.2f} {wgs:>6}  {name[:100]}")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter_dispatches(dirpath: str, counter: str):
    rows = list(csv.DictReader(open(_one(os.path.join(dirpath, "**", "*counter_collection.csv")))))
    vals, names, grid = defaultdict(float), {}, {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        i = int(r["Dispatch_Id"])
        vals[i] += float(r["Counter_Value"])
        names[i] = r["Kernel_Name"]
        grid[i] = int(r["Grid_Size"]) // max(int(r["Workgroup_Size"]), 1)
    return [dict(name=names[i], kib=vals[i], blocks=grid[i]) for i in sorted(vals)]


def traffic(fetch_dir, write_dir, copy_fetch_dir, copy_write_dir, copy_bytes, min_len, out, commands,
            labels="") -> None:
    copy_bytes = float(copy_bytes)
    key = lambda d: (d["name"], d["blocks"])
    fr = _runs(_counter_dispatches(fetch_dir, "FETCH_SIZE"), key, int(min_len))
    wr = _runs(_counter_dispatches(write_dir, "WRITE_SIZE"), key, int(min_len))
    if [r[0]["name"] for r in fr] != [r[0]["name"] for r in wr]:
        raise ValueError("the FETCH_SIZE and WRITE_SIZE runs launched different kernel blocks")
    cf = [d["kib"] for d in _counter_dispatches(copy_fetch_dir, "FETCH_SIZE") if d["name"] == COPY_KERNEL]
    cw = [d["kib"] for d in _counter_dispatches(copy_write_dir, "WRITE_SIZE") if d["name"] == COPY_KERNEL]
    cf_kib, cw_kib = sum(cf) / len(cf), sum(cw) / len(cw)
    f_scale = copy_bytes / (cf_kib * 1024.0)
    w_scale = copy_bytes / (cw_kib * 1024.0)
    lab = _labels(labels)
    res = {"copy_bytes": copy_bytes, "copy_fetch_kib": cf_kib, "copy_write_kib": cw_kib,
           "fetch_scale": f_scale, "write_scale": w_scale,
           "kernel_source_sha256_16": source_hash(), "commands": commands, "blocks": []}
    for i, (f, w) in enumerate(zip(fr, wr)):
        fk = sum(d["kib"] for d in f) / len(f)
        wk = sum(d["kib"] for d in w) / len(w)
        res["blocks"].append({
            "label": lab[i] if lab and i < len(lab) else "", "kernel": f[0]["name"], "launches": len(f),
            "raw_fetch_kib": fk, "raw_write_kib": wk,
            "fetch_bytes_per_launch": fk * 1024.0 * f_scale, "write_bytes_per_launch": wk * 1024.0 * w_scale,
            "bytes_per_launch": fk * 1024.0 * f_scale + wk * 1024.0 * w_scale})
    json.dump(res, open(out, "w"), indent=1)
    print(json.dumps(res, indent=1))


def block_traffic(path: str, label: str):
    """Bytes per launch of the block labelled `label` in a traffic summary,
    or None when the summary is missing, was taken on another kernel source
    or has no such block."""
    if not os.path.exists(path):
        return None
    t = json.load(open(path))
    if t.get("kernel_source_sha256_16") != source_hash():
        return None
    for b in t.get("blocks", []):
        if b["label"] == label:
            return b["bytes_per_launch"]
    return None


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "stats":
        stats(*sys.argv[2:5], *(int(a) for a in sys.argv[5:6]))
    elif len(sys.argv) > 1 and sys.argv[1] == "blocks":
        blocks(*sys.argv[2:7])
    elif len(sys.argv) > 1 and sys.argv[1] == "merged":
        merged(*sys.argv[2:7])
    elif len(sys.argv) > 1 and sys.argv[1] == "grids":
        grids(*sys.argv[2:6])
    elif len(sys.argv) > 1 and sys.argv[1] == "traffic":
        traffic(*sys.argv[2:11])
    else:
        raise SystemExit(__doc__)
