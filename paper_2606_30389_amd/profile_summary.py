"""Summaries of rocprofv3 output for the fused decode step.

Reads the CSV files that `rocprofv3 --kernel-trace --stats --output-format csv` and
`rocprofv3 --pmc FETCH_SIZE` / `--pmc WRITE_SIZE` write, and prints markdown tables:

* per fused launch shape (grid size in 512-thread workgroups, which identifies the
  schedule at a given workload): launches, average / median / min / max duration;
* per launch shape: median FETCH_SIZE and WRITE_SIZE (KiB per dispatch), calibrated by a
  plain device copy of known size that ran in the same process (`bench.py
  --copy-calibration-mib`), as HBM bytes per launch.

With --traffic-out it also writes the JSON record that bench.py reads for the roofline's
`traffic` field, tagged with the hash of the device sources it was measured on.

    python -m paper_2606_30389_amd.profile_summary trace DIR [--names 356=fused_prr_late ...]
    python -m paper_2606_30389_amd.profile_summary counters --fetch DIR --write DIR --copy-mib 256 \\
        --label fused_prr_late --grid 356 --config glm128k [--traffic-out profiles/traffic.json]
"""
import argparse
import csv
import glob
import json
import os
import statistics as st
import sys


ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# the sources of the fused step kernel (the separate kernels live in prr_kernels.hip)
DEVICE_SOURCES = ("prr_fused_impl.h", "prr_fused_bf16.hip", "prr_fused_f16.hip", "prr_fused_p64.hip", "prr_select.h",
                  "prr_device.h", "prr_launch.h")


def kernel_source_hash():
    """Hash of the fused kernel's sources' code (comments, blank lines and trailing blanks left out,
    so that only a change of the code itself invalidates recorded counters)."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in DEVICE_SOURCES:
        path = os.path.join(ROOT, "paper_2606_30389_amd", "csrc", f)
        if not os.path.exists(path):
            continue
        with open(path, encoding="utf-8") as fh:
            text = re.sub(r"/\*.*?\*/", "", fh.read(), flags=re.S)
        lines = (re.sub(r"//.*$", "", ln).rstrip() for ln in text.splitlines())
        h.update(f.encode())
        h.update("\n".join(ln for ln in lines if ln).encode())
    return h.hexdigest()[:16]


def _rows(directory, suffix):
    files = sorted(glob.glob(os.path.join(directory, "**", "*" + suffix), recursive=True))
    if not files:
        raise SystemExit(f"no *{suffix} under {directory}")
    with open(files[0], newline="") as f:
        return list(csv.DictReader(f))


def _grid(row, gx, wx):
    return int(row[gx]) // max(1, int(row[wx]))


def trace_table(directory, kernel="fused_step", names=None, splits=None):
    """Markdown table of the kernel trace by launch shape, and the durations by shape (us).
    splits: {grid: [(label, count), .., (label, None)]} labels consecutive launches of one
    shape in launch order (schedules of the same grid run one after another)."""
    names, splits = names or {}, splits or {}
    rows = [r for r in _rows(directory, "kernel_trace.csv") if kernel in r["Kernel_Name"]]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    by, seen, first = {}, {}, {}
    for r in rows:
        g = _grid(r, "Grid_Size_X", "Workgroup_Size_X")
        i = seen.get(g, 0)
        seen[g] = i + 1
        label = names.get(g, "?")
        if g in splits:
            acc = 0
            for lab, cnt in splits[g]:
                if cnt is None or i < acc + cnt:
                    label = lab
                    break
                acc += cnt
        first.setdefault((g, label), len(first))
        by.setdefault((g, label), []).append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0)
    lines = ["| launch | workgroups | launches | avg us | median us | min us | max us |", "|---|---|---|---|---|---|---|"]
    for (g, label) in sorted(by, key=lambda k: (k[0], first[k])):
        v = by[(g, label)]
        lines.append(f"| {label} | {g} | {len(v)} | {st.mean(v):.2f} | {st.median(v):.2f} | "
                     f"{min(v):.2f} | {max(v):.2f} |")
    return "\n".join(lines), by


def counter_medians(directory, kernel="fused_step"):
    """(values of the calibration copy, {grid: median}) of the one counter a --pmc run
    collected, in KiB.  The calibration copies are the copyBuffer dispatches that moved the
    most (other, smaller device copies of the run are ignored)."""
    copies, by = [], {}
    for r in _rows(directory, "counter_collection.csv"):
        name = r["Kernel_Name"]
        val = float(r["Counter_Value"])
        if "copyBuffer" in name:
            copies.append((int(r["Grid_Size"]), val))
        elif kernel in name:
            by.setdefault(_grid(r, "Grid_Size", "Workgroup_Size"), []).append(val)
    top = max((v for _, v in copies), default=0.0)
    copy = [v for _, v in copies if v >= 0.5 * top] if top > 0 else []
    return copy, {g: st.median(v) for g, v in by.items()}


def counters(fetch_dir, write_dir, copy_mib, kernel="fused_step"):
    """Calibrated HBM bytes per launch by launch shape: {grid: (read, written)}, and the
    calibration factors (bytes the copy moved / what the counter read for it)."""
    fc, fby = counter_medians(fetch_dir, kernel)
    wc, wby = counter_medians(write_dir, kernel)
    if not fc or not wc:
        raise SystemExit("the calibration copy is missing from a counter run (bench.py --copy-calibration-mib)")
    kib = copy_mib * 1024.0
    ff, wf = kib / st.median(fc), kib / st.median(wc)
    out = {}
    for g in sorted(fby):
        rb = int(round(fby[g] * 1024 * ff))
        wb = int(round(wby.get(g, float("nan")) * 1024 * wf)) if g in wby else None
        out[g] = (rb, wb, fby[g], wby.get(g))
    return out, ff, wf, st.median(fc), st.median(wc)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    t = sub.add_parser("trace")
    t.add_argument("dir")
    t.add_argument("--kernel", default="fused_step")
    t.add_argument("--names", nargs="*", default=[], help="GRID=label")
    t.add_argument("--split", nargs="*", default=[],
                   help="GRID=label:count,label:count,..,label (consecutive launches of one shape)")
    c = sub.add_parser("counters")
    c.add_argument("--fetch", required=True)
    c.add_argument("--write", required=True)
    c.add_argument("--copy-mib", type=int, required=True)
    c.add_argument("--kernel", default="fused_step")
    c.add_argument("--label", action="append", default=[], help="schedule label of --grid (same order)")
    c.add_argument("--grid", action="append", type=int, default=[])
    c.add_argument("--config", required=True, help="the workload's name (bench.py --config)")
    c.add_argument("--workload", default="", help="free text: layers and tokens of the counter runs")
    c.add_argument("--traffic-out", default=None, help="JSON record to create or update")
    a = ap.parse_args(argv)
    if a.cmd == "trace":
        names = dict((int(x.split("=")[0]), x.split("=", 1)[1]) for x in a.names)
        splits = {}
        for x in a.split:
            g, spec = x.split("=", 1)
            parts = []
            for item in spec.split(","):
                lab, _, cnt = item.partition(":")
                parts.append((lab, int(cnt) if cnt else None))
            splits[int(g)] = parts
        print(trace_table(a.dir, a.kernel, names, splits)[0])
        return 0
    res, ff, wf, fcopy, wcopy = counters(a.fetch, a.write, a.copy_mib, a.kernel)
    labels = dict(zip(a.grid, a.label))
    print(f"copy calibration ({a.copy_mib} MiB): FETCH_SIZE {fcopy:.1f} KiB (factor {ff:.4f}), "
          f"WRITE_SIZE {wcopy:.1f} KiB (factor {wf:.4f})")
    print("| launch | workgroups | FETCH_SIZE KiB (median) | WRITE_SIZE KiB (median) | read bytes | written bytes | total |")
    print("|---|---|---|---|---|---|---|")
    for g, (rb, wb, fk, wk) in res.items():
        tot = rb + (wb or 0)
        print(f"| {labels.get(g, '?')} | {g} | {fk:.1f} | {wk if wk is None else round(wk, 1)} | {rb:,} | "
              f"{wb if wb is None else format(wb, ',')} | {tot:,} |")
    if a.traffic_out:
        rec = {}
        if os.path.exists(a.traffic_out):
            with open(a.traffic_out) as f:
                rec = json.load(f)
        h = kernel_source_hash()
        if rec.get("kernel_source") != h or rec.get("config") != a.config:
            rec = {"kernel_source": h, "config": a.config, "kernels": {}}
        rec["fetch_factor"], rec["write_factor"] = ff, wf
        if a.workload:
            rec["workload"] = a.workload
        for g, label in labels.items():
            if g in res:
                rb, wb, _, _ = res[g]
                rec["kernels"][label] = {"hbm_bytes_per_launch": rb + (wb or 0), "read_bytes": rb, "write_bytes": wb,
                                         "grid": g}
        with open(a.traffic_out, "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")
    return 0


if __name__ == "__main__":
    sys.exit(main())
