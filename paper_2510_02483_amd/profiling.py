"""Summaries of rocprofv3 output for the profiles/ folder.

    python -m paper_2510_02483_amd.profiling stats DIR OUT.txt --cmd "..."
    python -m paper_2510_02483_amd.profiling traffic --kernel NAME --fetch DIR --write DIR \
        --copy-fetch DIR --copy-write DIR --copy-bytes N --out OUT.txt --cmd "..." [--trace DIR --trace-cmd "..."]

    python -m paper_2510_02483_amd.profiling launches DIR OUT.txt --cmd "..."
    python -m paper_2510_02483_amd.profiling counters --kernel NAME --cus 256 --simds 4 --xcds 8 OUT.txt DIR... --cmd "..."

`stats` condenses a --kernel-trace --stats run (kernel_stats.csv) into a
table.  `launches` splits the kernel trace of block steps into steps and
names every dispatch after the labelled launch it belongs to (the library
issues a fixed sequence per step), then reports each launch's mean duration.
`counters` averages the counters of several --pmc runs (one counter group
each) per dispatch of a kernel and derives matrix-core and texture-unit busy
fractions from them.  `traffic` turns two --pmc runs (FETCH_SIZE, then WRITE_SIZE, in KiB per
dispatch) of a kernel, or of one labelled launch of the block step, into
bytes per launch, each scaled by what the same counter reads for a plain
device copy of known size (bytes read = bytes written = N), and records the
hash of the kernel sources it was taken with; bench.py reports the figure
only while that hash still matches.
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


# The matrix products of one block step in issue order (each may be followed
# by the reduction of its split K, which counts as part of it).
GEMM_ORDER = ("qkv projection", "output projection", "gate/up projection", "down projection", "dact", "dh2", "dWg/dWu",
              "dWd", "dO", "dWo", "dh1", "dWqkv")


def label_steps(names):
    """Split a sequence of dispatched kernel names into block steps and name
    each dispatch after its labelled launch: [(index, label), ...] per step.
    A step starts at an RMSNorm forward followed by the RoPE table; dispatches
    outside steps (set-up, other work) are left out."""
    starts = [i for i in range(len(names) - 1)
              if "rmsnorm_fwd_kernel" in names[i] and "rope_table_kernel" in names[i + 1]]
    steps = []
    for si, a in enumerate(starts):
        b = starts[si + 1] if si + 1 < len(starts) else len(names)
        seq, g, norm_f, norm_b, last = [], 0, 0, 0, None
        for i in range(a, b):
            n = names[i]
            if "rmsnorm_fwd_kernel" in n:
                lab = "rmsnorm fwd"
                norm_f += 1
            elif "rope_table_kernel" in n:
                lab = "rope table"
            elif "rmsnorm_bwd_kernel" in n or "column_sum_kernel" in n:
                lab = "rmsnorm bwd"
            elif "attn_fwd_kernel" in n:
                lab = "attention fwd"
            elif "attn_bwd" in n:
                lab = "attention bwd"
            elif "kpart_reduce_kernel" in n and last in GEMM_ORDER:
                lab = last
            elif "gemm_kernel" in n and g < len(GEMM_ORDER):
                lab = GEMM_ORDER[g]
                g += 1
            else:
                break  # not a block step's dispatch: the step ended
            seq.append((i, lab))
            last = lab
        if g == len(GEMM_ORDER):
            steps.append(seq)
    return steps


def launches(directory: str, out: str, cmd: str):
    rows = _csv(directory, "kernel_trace.csv")
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    names = [r["Kernel_Name"] for r in rows]
    steps = label_steps(names)
    if not steps:
        raise ValueError(f"no block steps in {directory}")
    per = {}
    for seq in steps:
        tot = {}
        for i, lab in seq:
            r = rows[i]
            tot[lab] = tot.get(lab, 0.0) + (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3
        for lab, us in tot.items():
            per.setdefault(lab, []).append(us)
    order = []
    for _, lab in steps[0]:
        if lab not in order:
            order.append(lab)
    step_us = [sum(v[k] for v in per.values()) for k in range(len(steps))]
    lines = [f"# per-launch durations of the block step from the kernel trace ({len(steps)} steps)",
             f"# command: {cmd}", "",
             f"{'launch':22s} {'mean_us':>9} {'min_us':>9} {'max_us':>9} {'share':>7}"]
    total = sum(sum(v) for v in per.values()) / len(steps)
    for lab in order:
        v = per[lab]
        lines.append(f"{lab:22s} {sum(v) / len(v):9.1f} {min(v):9.1f} {max(v):9.1f} {100 * sum(v) / len(v) / total:6.1f}%")
    lines.append(f"{'sum of kernels':22s} {total:9.1f} {min(step_us):9.1f} {max(step_us):9.1f}")
    with open(out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter_per_dispatch(directory: str, counter: str, kernel: str, launch: str | None = None):
    """Mean of a counter over the dispatches of `kernel` (substring of the
    name) or, with `launch`, over the dispatches of that labelled launch of
    the block step (summed per launch)."""
    if launch is not None:
        rows = _csv(directory, "counter_collection.csv")
        disp = {}
        for r in rows:
            if r["Counter_Name"] == counter:
                d = disp.setdefault(int(r["Dispatch_Id"]), [r["Kernel_Name"], 0.0])
                d[1] += float(r["Counter_Value"])
        ids = sorted(disp)
        steps = label_steps([disp[i][0] for i in ids])
        vals = [sum(disp[ids[i]][1] for i, lab in seq if lab == launch) for seq in steps]
        vals = [v for v in vals if v > 0]
        if not vals:
            raise ValueError(f"no {counter} rows for launch {launch!r} in {directory}")
        return sum(vals) / len(vals), len(vals)
    return _counter_per_kernel(directory, counter, kernel)


def _counter_per_kernel(directory: str, counter: str, kernel: str):
    rows = _csv(directory, "counter_collection.csv")
    vals = [float(r["Counter_Value"]) for r in rows if r["Counter_Name"] == counter and kernel in r["Kernel_Name"]]
    if not vals:
        raise ValueError(f"no {counter} rows for kernel matching {kernel!r} in {directory}")
    return sum(vals) / len(vals), len(vals)


def counters(a):
    sums = {}
    for d in a.dirs:
        rows = _csv(d, "counter_collection.csv")
        per = {}
        for r in rows:
            if a.kernel in r["Kernel_Name"]:
                key = (int(r["Dispatch_Id"]), r["Counter_Name"])
                per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
        for (_, cn), v in per.items():
            sums.setdefault(cn, []).append(v)
    mean = {cn: sum(v) / len(v) for cn, v in sums.items()}
    lines = [f"# counters of {a.kernel}", f"# command (one run per counter group): {a.cmd}",
             "# values: mean per dispatch, summed over the device (GRBM_GUI_ACTIVE summed over the XCDs)", ""]
    lines += [f"   {cn:36s} {mean[cn]:.4g}" for cn in sorted(mean)]
    if "GRBM_GUI_ACTIVE" in mean:
        cyc = mean["GRBM_GUI_ACTIVE"] / a.xcds
        lines.append(f"   derived: kernel cycles per XCD {cyc:.4g}")
        if "SQ_VALU_MFMA_BUSY_CYCLES" in mean:
            lines.append(f"   derived: MFMA busy per SIMD {100 * mean['SQ_VALU_MFMA_BUSY_CYCLES'] / (cyc * a.cus * a.simds):.1f}% of the kernel")
        if "TD_TD_BUSY_sum" in mean:
            lines.append(f"   derived: TD busy per CU {100 * mean['TD_TD_BUSY_sum'] / (cyc * a.cus):.1f}%")
        if "TA_TA_BUSY_sum" in mean:
            lines.append(f"   derived: TA busy per CU {100 * mean['TA_TA_BUSY_sum'] / (cyc * a.cus):.1f}%")
    if "TCP_TCC_READ_REQ_sum" in mean and "TCP_TCC_READ_REQ_LATENCY_sum" in mean:
        lines.append(f"   derived: mean L1->L2 read latency {mean['TCP_TCC_READ_REQ_LATENCY_sum'] / mean['TCP_TCC_READ_REQ_sum']:.0f} cycles")
    if "TCC_HIT_sum" in mean and "TCC_MISS_sum" in mean:
        lines.append(f"   derived: L2 hit rate {100 * mean['TCC_HIT_sum'] / (mean['TCC_HIT_sum'] + mean['TCC_MISS_sum']):.1f}%")
    if "SQ_INSTS_VALU" in mean and mean.get("SQ_INSTS_MFMA", 0) > 0:
        lines.append(f"   derived: non-MFMA VALU instructions per MFMA {(mean['SQ_INSTS_VALU'] - mean['SQ_INSTS_MFMA']) / mean['SQ_INSTS_MFMA']:.2f}")
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _mean_duration_us(directory: str, kernel: str, launch: str | None = None):
    """Mean duration (us) of a dispatch of `kernel` (substring of the name)
    in a --kernel-trace run or, with `launch`, of that labelled launch of the
    block step (its dispatches summed per step)."""
    rows = _csv(directory, "kernel_trace.csv")
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    dur = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3 for r in rows]
    if launch is not None:
        steps = label_steps([r["Kernel_Name"] for r in rows])
        vals = [sum(dur[i] for i, lab in seq if lab == launch) for seq in steps]
        vals = [v for v in vals if v > 0]
    else:
        vals = [d for r, d in zip(rows, dur) if kernel in r["Kernel_Name"]]
    if not vals:
        raise ValueError(f"no dispatches of {launch or kernel!r} in {directory}")
    return sum(vals) / len(vals), len(vals)


def traffic(a):
    fetch_kib, nf = _counter_per_dispatch(a.fetch, "FETCH_SIZE", a.kernel, a.launch)
    write_kib, nw = _counter_per_dispatch(a.write, "WRITE_SIZE", a.kernel, a.launch)
    cf_kib, _ = _counter_per_dispatch(a.copy_fetch, "FETCH_SIZE", a.copy_kernel)
    cw_kib, _ = _counter_per_dispatch(a.copy_write, "WRITE_SIZE", a.copy_kernel)
    f_scale = a.copy_bytes / (cf_kib * 1024.0)
    w_scale = a.copy_bytes / (cw_kib * 1024.0)
    fetch_b = fetch_kib * 1024.0 * f_scale
    write_b = write_kib * 1024.0 * w_scale
    entry = {"kernel": a.kernel, "launch": a.launch, "label": a.label, "fetch_bytes": fetch_b, "write_bytes": write_b,
             "traffic_bytes": fetch_b + write_b, "fetch_scale": f_scale, "write_scale": w_scale,
             "sources_hash": sources_hash(), "dispatches": [nf, nw]}
    lines = [f"# HBM traffic of {a.label}", f"# kernel: {a.kernel}" + (f" (launch {a.launch!r} of the block step)" if a.launch else ""),
             f"# command: {a.cmd}", "",
             f"FETCH_SIZE per dispatch: {fetch_kib:.1f} KiB ({nf} dispatches)",
             f"WRITE_SIZE per dispatch: {write_kib:.1f} KiB ({nw} dispatches)",
             f"copy calibration ({a.copy_bytes} bytes read and written): FETCH_SIZE {cf_kib:.1f} KiB, "
             f"WRITE_SIZE {cw_kib:.1f} KiB -> scale {f_scale:.4f} / {w_scale:.4f}",
             f"traffic per launch: fetch {fetch_b / 1e6:.1f} MB + write {write_b / 1e6:.1f} MB = "
             f"{(fetch_b + write_b) / 1e6:.1f} MB"]
    if a.trace:
        us, nd = _mean_duration_us(a.trace, a.kernel, a.launch)
        entry["mean_us"] = us
        entry["achieved_gbps"] = (fetch_b + write_b) / (us * 1e-6) / 1e9
        lines.append(f"mean duration {us:.1f} us ({nd} dispatches of {a.trace_cmd or a.trace}): "
                     f"achieved {entry['achieved_gbps']:.0f} GB/s of HBM-side traffic (L2 misses)")
    lines.append(f"kernel sources hash: {entry['sources_hash']}")
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
    t.add_argument("--launch", default=None, help="a labelled launch of the block step (dispatches picked by position)")
    t.add_argument("--label", required=True)
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--copy-fetch", required=True)
    t.add_argument("--copy-write", required=True)
    t.add_argument("--copy-kernel", default="copyBuffer")
    t.add_argument("--copy-bytes", type=float, required=True)
    t.add_argument("--out", required=True)
    t.add_argument("--cmd", required=True)
    t.add_argument("--trace", default=None, help="a --kernel-trace run of the same workload, for durations and GB/s")
    t.add_argument("--trace-cmd", default=None, help="the command of that run, for the summary")
    c = sub.add_parser("counters")
    c.add_argument("--kernel", required=True)
    c.add_argument("--cus", type=int, default=256)
    c.add_argument("--simds", type=int, default=4)
    c.add_argument("--xcds", type=int, default=8)
    c.add_argument("out")
    c.add_argument("dirs", nargs="+")
    c.add_argument("--cmd", required=True)
    l = sub.add_parser("launches")
    l.add_argument("dir")
    l.add_argument("out")
    l.add_argument("--cmd", required=True)
    a = ap.parse_args()
    if a.what == "stats":
        stats(a.dir, a.out, a.cmd)
    elif a.what == "counters":
        counters(a)
    elif a.what == "launches":
        launches(a.dir, a.out, a.cmd)
    else:
        traffic(a)


if __name__ == "__main__":
    main()
