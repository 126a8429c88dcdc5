"""CPU checks of the profile summaries that bench.py reads: the HBM bytes per
launch from FETCH_SIZE / WRITE_SIZE counter runs, scaled by what the same
counters read for a device copy of known size, and the rule that a summary
taken on another kernel source is not used."""
from __future__ import annotations

import csv
import json
import os

from paper_2608_04991_amd import rocprof_summary as rs

FIELDS = ["Dispatch_Id", "Kernel_Name", "Grid_Size", "Workgroup_Size", "Counter_Name", "Counter_Value"]


def _counters(dirpath, counter, dispatches):
    """A counter_collection.csv of (kernel, grid, KiB) dispatches; each
    dispatch's value is split over two rows, as the counter's instances are."""
    os.makedirs(os.path.join(dirpath, "run"), exist_ok=True)
    with open(os.path.join(dirpath, "run", "p_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for i, (name, grid, kib) in enumerate(dispatches):
            for part in (0.25, 0.75):
                w.writerow({"Dispatch_Id": i + 1, "Kernel_Name": name, "Grid_Size": grid * 256,
                            "Workgroup_Size": 256, "Counter_Name": counter, "Counter_Value": kib * part})


def test_traffic_scales_each_counter_by_the_copy_and_labels_the_blocks(tmp_path):
    enc, dec, other = "rac_encode_rows_kernel<4>", "rac_decode_kernel<4>", "at::native::fill"
    # three encodes and three decodes (plus a non-codec kernel between them)
    _counters(tmp_path / "f", "FETCH_SIZE", [(enc, 100, 1000.0)] * 3 + [(other, 1, 5.0)] + [(dec, 100, 600.0)] * 3)
    _counters(tmp_path / "w", "WRITE_SIZE", [(enc, 100, 2000.0)] * 3 + [(other, 1, 5.0)] + [(dec, 100, 900.0)] * 3)
    # the copy: 1 MiB read and written; the fetch counter reads half of it
    copy = rs.COPY_KERNEL
    _counters(tmp_path / "cf", "FETCH_SIZE", [(copy, 16, 512.0)])
    _counters(tmp_path / "cw", "WRITE_SIZE", [(copy, 16, 1024.0)])
    labels = tmp_path / "labels.json"
    labels.write_text(json.dumps({"profile": "x", "cfg_a": {"encode_us": 1.0}}))
    out = tmp_path / "traffic.json"
    rs.traffic(str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cf"), str(tmp_path / "cw"),
               1 << 20, 3, str(out), "cmd", str(labels))
    t = json.load(open(out))
    assert t["fetch_scale"] == 2.0 and t["write_scale"] == 1.0
    assert t["kernel_source_sha256_16"] == rs.source_hash()
    assert [b["label"] for b in t["blocks"]] == ["cfg_a encode", "cfg_a decode"]
    e, d = t["blocks"]
    assert e["kernel"] == enc and e["launches"] == 3
    assert e["bytes_per_launch"] == 1000.0 * 1024 * 2.0 + 2000.0 * 1024
    assert d["bytes_per_launch"] == 600.0 * 1024 * 2.0 + 900.0 * 1024
    # bench.py's lookup: by label, on the current kernel source only
    assert rs.block_traffic(str(out), "cfg_a encode") == e["bytes_per_launch"]
    assert rs.block_traffic(str(out), "no such block") is None
    assert rs.block_traffic(str(tmp_path / "missing.json"), "cfg_a encode") is None
    t["kernel_source_sha256_16"] = "0" * 16
    out.write_text(json.dumps(t))
    assert rs.block_traffic(str(out), "cfg_a encode") is None


def test_runs_keep_only_long_runs_of_codec_kernels():
    items = [{"name": n, "blocks": b} for n, b in
             [("rac_a", 1), ("rac_a", 1), ("rac_a", 2), ("x", 1), ("x", 1), ("x", 1), ("rac_b", 1), ("rac_b", 1)]]
    key = lambda d: (d["name"], d["blocks"])
    runs = rs._runs(items, key, 2)
    assert [(r[0]["name"], r[0]["blocks"], len(r)) for r in runs] == [("rac_a", 1, 2), ("rac_b", 1, 2)]


def test_labels_expand_launch_shapes_into_repeated_blocks(tmp_path):
    # the launch-shape sweep gives, per configuration and shape, `reps`
    # back-to-back encode and decode blocks
    p = tmp_path / "shapes.json"
    p.write_text(json.dumps({"profile": "launch_shapes", "iters": 20, "reps": 2,
                             "a": {"default": {"encode_us": 1.0}, "per_row": {"encode_us": 2.0}},
                             "b": {"strided": {"encode_us": 3.0}}}))
    assert rs._labels(str(p)) == ["a default encode", "a default decode"] * 2 + \
        ["a per_row encode", "a per_row decode"] * 2 + ["b strided encode", "b strided decode"] * 2
    assert rs._labels(None) is None
    q = tmp_path / "list.json"
    q.write_text(json.dumps(["x", "y"]))
    assert rs._labels(str(q)) == ["x", "y"]


def _trace(dirpath, dispatches):
    """A kernel_trace.csv of (kernel, workgroups, µs) dispatches back to back."""
    os.makedirs(os.path.join(dirpath, "run"), exist_ok=True)
    f = ["Dispatch_Id", "Kernel_Name", "Workgroup_Size_X", "Workgroup_Size_Y", "Workgroup_Size_Z",
         "Grid_Size_X", "Grid_Size_Y", "Grid_Size_Z", "Start_Timestamp", "End_Timestamp"]
    with open(os.path.join(dirpath, "run", "p_kernel_trace.csv"), "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=f)
        w.writeheader()
        t = 1000
        for i, (name, wgs, us) in enumerate(dispatches):
            w.writerow(dict(zip(f, [i + 1, name, 256, 1, 1, wgs * 256, 1, 1, t, t + int(us * 1000)])))
            t += int(us * 1000) + 500


def test_merged_takes_the_median_block_per_label(tmp_path):
    enc = "void (anonymous namespace)::rac_encode_rows_kernel<4, 4>((anonymous namespace)::Args)"
    dec = "void (anonymous namespace)::rac_decode_kernel<4, 1>((anonymous namespace)::Args)"
    d = []
    for rep, (e_us, d_us) in enumerate([(10.0, 6.0), (12.0, 5.0), (11.0, 7.0)]):
        d += [(enc, 100, e_us)] * 4 + [(dec, 50, d_us)] * 4
    d += [("at::native::fill", 1, 1.0)] * 4           # not a codec kernel: no block
    d += [(enc, 200, 20.0)] * 4 + [(dec, 200, 9.0)] * 4
    _trace(tmp_path / "t", d)
    lab = tmp_path / "l.json"
    lab.write_text(json.dumps({"profile": "launch_shapes", "reps": 3,
                               "c": {"default": {}}, "e": {"per_row": {}}}))
    # three repetitions of "c" but one of "e": the label count does not match
    try:
        rs.merged(str(tmp_path / "t"), "3", str(tmp_path / "o.txt"), "cmd", str(lab))
        raise AssertionError("expected a label count mismatch")
    except ValueError as err:
        assert "8 blocks" in str(err) and "12 labels" in str(err)
    d += [(enc, 200, 22.0)] * 4 + [(dec, 200, 8.0)] * 4 + [(enc, 200, 21.0)] * 4 + [(dec, 200, 10.0)] * 4
    _trace(tmp_path / "t", d)
    rs.merged(str(tmp_path / "t"), "3", str(tmp_path / "o.txt"), "cmd", str(lab))
    rows = [l.split() for l in open(tmp_path / "o.txt").read().splitlines()[4:]]
    got = {" ".join(r[5:8]): (int(r[0]), float(r[1]), float(r[2]), float(r[3]), int(r[4])) for r in rows}
    assert got == {"c default encode": (3, 11.0, 10.0, 12.0, 100), "c default decode": (3, 6.0, 5.0, 7.0, 50),
                   "e per_row encode": (3, 21.0, 20.0, 22.0, 200), "e per_row decode": (3, 9.0, 8.0, 10.0, 200)}
    assert all(r[9].startswith("rac_") for r in rows)
