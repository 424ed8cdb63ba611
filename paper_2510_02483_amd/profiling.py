"""Summaries of rocprofv3 output for the profiles/ folder.

    python -m paper_2510_02483_amd.profiling stats DIR OUT.txt --cmd "..."
    python -m paper_2510_02483_amd.profiling traffic --kernel NAME --fetch DIR --write DIR \
        --copy-fetch DIR --copy-write DIR --copy-bytes N --out OUT.txt --cmd "..."

`stats` condenses a --kernel-trace --stats run (kernel_stats.csv) into a
table.  `traffic` turns two --pmc runs of a kernel (FETCH_SIZE, then
WRITE_SIZE, in KiB per dispatch) into bytes per launch, each scaled by what
the same counter reads for a plain device copy of known size (bytes read =
bytes written = N), and records the hash of the kernel sources it was taken
with; bench.py reports the figure only while that hash still matches.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
TRAFFIC_JSON = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCES = ("gemm.hip", "common.h", "kernels.h")


def sources_hash() -> str:
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(PKG, "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _csv(directory: str, suffix: str):
    files = glob.glob(os.path.join(directory, "**", f"*{suffix}"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no *{suffix} under {directory}")
    with open(files[0]) as f:
        return list(csv.DictReader(f))


def short_name(name: str) -> str:
    n = name.replace("void ", "").replace("ls::(anonymous namespace)::", "")
    return n.split("(")[0]


def stats(directory: str, out: str, cmd: str, top: int = 25):
    rows = _csv(directory, "kernel_stats.csv")
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    lines = [f"# rocprofv3 kernel statistics", f"# command: {cmd}", "",
             f"{'share':>6} {'calls':>6} {'avg_us':>10} {'min_us':>10} {'max_us':>10}  kernel"]
    for r in rows[:top]:
        lines.append(f"{float(r['Percentage']):5.1f}% {int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:10.1f} "
                     f"{float(r['MinNs']) / 1e3:10.1f} {float(r['MaxNs']) / 1e3:10.1f}  {short_name(r['Name'])}")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter_per_dispatch(directory: str, counter: str, kernel: str):
    rows = _csv(directory, "counter_collection.csv")
    vals = [float(r["Counter_Value"]) for r in rows if r["Counter_Name"] == counter and kernel in r["Kernel_Name"]]
    if not vals:
        raise ValueError(f"no {counter} rows for kernel matching {kernel!r} in {directory}")
    return sum(vals) / len(vals), len(vals)


def traffic(a):
    fetch_kib, nf = _counter_per_dispatch(a.fetch, "FETCH_SIZE", a.kernel)
    write_kib, nw = _counter_per_dispatch(a.write, "WRITE_SIZE", a.kernel)
    cf_kib, _ = _counter_per_dispatch(a.copy_fetch, "FETCH_SIZE", a.copy_kernel)
    cw_kib, _ = _counter_per_dispatch(a.copy_write, "WRITE_SIZE", a.copy_kernel)
    f_scale = a.copy_bytes / (cf_kib * 1024.0)
    w_scale = a.copy_bytes / (cw_kib * 1024.0)
    fetch_b = fetch_kib * 1024.0 * f_scale
    write_b = write_kib * 1024.0 * w_scale
    entry = {"kernel": a.kernel, "label": a.label, "fetch_bytes": fetch_b, "write_bytes": write_b,
             "traffic_bytes": fetch_b + write_b, "fetch_scale": f_scale, "write_scale": w_scale,
             "sources_hash": sources_hash(), "dispatches": [nf, nw]}
    lines = [f"# HBM traffic of {a.label}", f"# kernel: {a.kernel}", f"# command: {a.cmd}", "",
             f"FETCH_SIZE per dispatch: {fetch_kib:.1f} KiB ({nf} dispatches)",
             f"WRITE_SIZE per dispatch: {write_kib:.1f} KiB ({nw} dispatches)",
             f"copy calibration ({a.copy_bytes} bytes read and written): FETCH_SIZE {cf_kib:.1f} KiB, "
             f"WRITE_SIZE {cw_kib:.1f} KiB -> scale {f_scale:.4f} / {w_scale:.4f}",
             f"traffic per launch: fetch {fetch_b / 1e6:.1f} MB + write {write_b / 1e6:.1f} MB = "
             f"{(fetch_b + write_b) / 1e6:.1f} MB", f"kernel sources hash: {entry['sources_hash']}"]
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    data = {}
    if os.path.exists(TRAFFIC_JSON):
        with open(TRAFFIC_JSON) as f:
            data = json.load(f)
    data[a.label] = entry
    with open(TRAFFIC_JSON, "w") as f:
        json.dump(data, f, indent=1)
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="what", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("out")
    s.add_argument("--cmd", required=True)
    t = sub.add_parser("traffic")
    t.add_argument("--kernel", required=True)
    t.add_argument("--label", required=True)
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--copy-fetch", required=True)
    t.add_argument("--copy-write", required=True)
    t.add_argument("--copy-kernel", default="copyBuffer")
    t.add_argument("--copy-bytes", type=float, required=True)
    t.add_argument("--out", required=True)
    t.add_argument("--cmd", required=True)
    a = ap.parse_args()
    if a.what == "stats":
        stats(a.dir, a.out, a.cmd)
    else:
        traffic(a)


if __name__ == "__main__":
    main()
