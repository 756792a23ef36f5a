"""Turn rocprofv3 counter dumps into per-launch HBM traffic of libwide kernels.

rocprofv3 --pmc FETCH_SIZE (and, in a separate run, WRITE_SIZE) reports KiB
moved between the L2 caches and memory per dispatch.  On MI355X these counters
do not read exactly the bytes moved, so each one is scaled by what it reads
for a plain device copy of known size, recorded in the same run (the
benchmark's --calibration-copy option issues two 1 GiB copies).

The summary also records a digest of the library sources: a traffic figure is
only valid for the kernels as they were when the counters were taken.

    python -m paper_2607_28418_amd.profiling counters --fetch F.csv --write W.csv \\
        --copy-bytes 1073741824 --command "..." --out profiles/x.json
    python -m paper_2607_28418_amd.profiling trace --trace run_kernel_trace.csv \\
        --skip 3 --command "..." --out profiles/x.md
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os
import re

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
COPY_KERNEL = "__amd_rocclr_copyBuffer"
CALIBRATION_COPIES = 2  # bench.py --calibration-copy ends with two copies of copy_bytes


def source_digest() -> str:
    """sha256 over the library's kernel and ABI sources, in name order."""
    h = hashlib.sha256()
    csrc = os.path.join(HERE, "csrc")
    paths = sorted(os.path.join(csrc, f) for f in os.listdir(csrc)
                   if f.endswith((".hip", ".h", ".cpp")))
    paths.append(os.path.join(ROOT, "include", "wide.h"))
    for p in paths:
        h.update(os.path.basename(p).encode())
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def kernel_key(name: str) -> str:
    """'void wide::wide_mn256<true, 64>(wide::MN256Args)' -> 'wide_mn256<true, 64>'."""
    name = re.sub(r"^void ", "", name.strip())
    name = name.replace("(anonymous namespace)::", "")
    name = name.split("(")[0]
    return name.replace("wide::", "")


def counter_means(path: str) -> dict:
    """{kernel key: {counter: mean value per dispatch, 'dispatches': n}}.

    Other device copies of the program (the runtime's, torch's) also run the
    copy kernel, some with the calibration copies' grid; the calibration
    copies are the program's last CALIBRATION_COPIES dispatches of it with
    the largest grid, and only those are kept for it (in dispatch order when the dump numbers the
    dispatches, else in file order)."""
    acc = collections.defaultdict(lambda: collections.defaultdict(list))
    with open(path) as f:
        rows = list(csv.DictReader(f))
    order = lambda i: (int(rows[i]["Dispatch_Id"]) if rows[i].get("Dispatch_Id") else i, i)
    grid = lambda r: int(r.get("Grid_Size") or 0)
    copy_grid = max((grid(r) for r in rows if kernel_key(r["Kernel_Name"]) == COPY_KERNEL), default=0)
    copies = sorted((i for i, r in enumerate(rows)
                     if kernel_key(r["Kernel_Name"]) == COPY_KERNEL and grid(r) == copy_grid), key=order)
    ids = []
    for i in reversed(copies):  # one row per (dispatch, counter): keep the last dispatches' rows
        d = rows[i].get("Dispatch_Id") or i
        if d not in ids:
            if len(ids) == CALIBRATION_COPIES:
                break
            ids.append(d)
    keep = {i for i in copies if (rows[i].get("Dispatch_Id") or i) in ids}
    for i, r in enumerate(rows):
        k = kernel_key(r["Kernel_Name"])
        if k == COPY_KERNEL and i not in keep:
            continue
        acc[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
    out = {}
    for k, cs in acc.items():
        out[k] = {c: sum(v) / len(v) for c, v in cs.items()}
        out[k]["dispatches"] = max(len(v) for v in cs.values())
    return out


def summarize(fetch_csv: str, write_csv: str, copy_bytes: int, command: str) -> dict:
    fetch = counter_means(fetch_csv)
    write = counter_means(write_csv)
    if COPY_KERNEL not in fetch or COPY_KERNEL not in write:
        raise ValueError("the calibration copy kernel is missing from the counter dumps")
    # a copy of copy_bytes reads and writes copy_bytes each
    f_scale = copy_bytes / (fetch[COPY_KERNEL]["FETCH_SIZE"] * 1024.0)
    w_scale = copy_bytes / (write[COPY_KERNEL]["WRITE_SIZE"] * 1024.0)
    kernels = {}
    for k in sorted(set(fetch) & set(write)):
        if k == COPY_KERNEL:
            continue
        fk, wk = fetch[k]["FETCH_SIZE"], write[k]["WRITE_SIZE"]
        kernels[k] = dict(fetch_kib_per_dispatch=round(fk, 1), write_kib_per_dispatch=round(wk, 1),
                          fetch_bytes=round(fk * 1024 * f_scale), write_bytes=round(wk * 1024 * w_scale),
                          dispatches=int(fetch[k]["dispatches"]))
    return dict(command=command, copy_bytes=copy_bytes,
                fetch_scale=round(f_scale, 4), write_scale=round(w_scale, 4),
                source_sha256=source_digest(), kernels=kernels)


def traffic_for(summary_path: str, kernel_label: str):
    """HBM bytes per launch of a kernel from a committed summary, or None when
    the summary is missing or the sources changed since it was taken."""
    if not os.path.exists(summary_path):
        return None
    with open(summary_path) as f:
        s = json.load(f)
    if s.get("source_sha256") != source_digest():
        return None
    for k, v in s["kernels"].items():
        if label_matches(k, kernel_label):
            return v["fetch_bytes"] + v["write_bytes"]
    return None


def label_matches(key: str, label: str) -> bool:
    """Does a demangled kernel key ('wide_mn256<true, 64>') belong to a timing
    label ('wide_mn256<true>' or 'wide_mn256<true>/bk64' or 'wide_kd256')?
    The label names the kernel and, optionally, its leading template argument."""
    base = label.split("/")[0]
    stem = base[:-1] if base.endswith(">") else base
    return key.startswith(stem) and key[len(stem):len(stem) + 1] in ("", "<", ",", ">")


def trace_stats(trace_csv: str, skip: int = 0) -> dict:
    """Per-kernel launch durations (µs) from a rocprofv3 --kernel-trace CSV.
    The first `skip` launches of every kernel (warm-up) are left out."""
    d = collections.defaultdict(list)
    with open(trace_csv) as f:
        for r in csv.DictReader(f):
            d[kernel_key(r["Kernel_Name"])].append(
                (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0)
    out = {}
    for k, v in d.items():
        v = v[skip:] if len(v) > skip else v
        out[k] = dict(launches=len(v), avg_us=sum(v) / len(v), min_us=min(v), max_us=max(v),
                      total_us=sum(v))
    return out


def trace_markdown(stats: dict, command: str, skip: int) -> str:
    total = sum(v["total_us"] for v in stats.values())
    lines = [f"Command: `{command}`", "",
             f"Launch durations from the kernel trace; the first {skip} launches of each kernel "
             "(warm-up) are left out.", "",
             "| kernel | launches | avg µs | min µs | max µs | share |", "|---|---|---|---|---|---|"]
    for k, v in sorted(stats.items(), key=lambda kv: -kv[1]["total_us"]):
        lines.append(f"| `{k}` | {v['launches']} | {v['avg_us']:.2f} | {v['min_us']:.2f} | "
                     f"{v['max_us']:.2f} | {100 * v['total_us'] / total:.1f}% |")
    return "\n".join(lines) + "\n"


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="what", required=True)
    c = sub.add_parser("counters")
    c.add_argument("--fetch", required=True)
    c.add_argument("--write", required=True)
    c.add_argument("--copy-bytes", type=int, default=1 << 30)
    c.add_argument("--command", required=True)
    c.add_argument("--out", required=True)
    t = sub.add_parser("trace")
    t.add_argument("--trace", required=True)
    t.add_argument("--skip", type=int, default=0)
    t.add_argument("--command", required=True)
    t.add_argument("--header", default="")
    t.add_argument("--out", required=True)
    a = ap.parse_args()
    if a.what == "counters":
        s = summarize(a.fetch, a.write, a.copy_bytes, a.command)
        with open(a.out, "w") as f:
            json.dump(s, f, indent=1)
        print(json.dumps(s, indent=1))
    else:
        md = (a.header + "\n\n" if a.header else "") + trace_markdown(
            trace_stats(a.trace, a.skip), a.command, a.skip)
        with open(a.out, "w") as f:
            f.write(md)
        print(md)


if __name__ == "__main__":
    main()
