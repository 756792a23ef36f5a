"""Turn rocprofv3 counter dumps into per-launch HBM traffic of libwide kernels.

rocprofv3 --pmc FETCH_SIZE (and, in a separate run, WRITE_SIZE) reports KiB
moved between the L2 caches and memory per dispatch.  On MI355X these counters
do not read exactly the bytes moved, so each one is scaled by what it reads
for a plain device copy of known size, recorded in the same run (the
benchmark's --calibration-copy option issues two 1 GiB copies).

The summary also records a digest of the library sources (their code, without
comments): a traffic figure is only valid for the kernels as they were when
the counters were taken.

    python -m paper_2607_28418_amd.profiling counters --fetch F.csv --write W.csv \\
        --copy-bytes 1073741824 --command "..." --out profiles/x.json
    python -m paper_2607_28418_amd.profiling trace --trace run_kernel_trace.csv \\
        --skip 3 --command "..." --out profiles/x.md
    python -m paper_2607_28418_amd.profiling mfma --pmc A.csv B.csv --command "..." \\
        --out profiles/x.json

The mfma summary turns SQ_/GRBM_ counter passes (each pass a separate
rocprofv3 --pmc run of the same program) into per-kernel utilisation: the
GRBM_GUI_ACTIVE counter is summed over the chip's 8 XCDs and the SQ_ busy
counters over its 1024 SIMDs (256 CUs), so

    clock_GHz      = GRBM_GUI_ACTIVE / 8 / duration
    mfma_busy      = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE * 128)
    wait_any       = SQ_WAIT_ANY / SQ_WAVE_CYCLES        (waves waiting on anything)
    wait_lds       = SQ_WAIT_INST_LDS / SQ_WAVE_CYCLES
    lds_fifo_full  = SQ_LDS_CMD_FIFO_FULL / (GRBM_GUI_ACTIVE * 32)   (per CU-cycle)
    lds_conflict   = SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE
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


def code_text(src: str) -> str:
    """C/C++/HIP source with comments removed and whitespace runs collapsed:
    what the compiler sees, so that editing a comment does not invalidate a
    profile taken on the same kernels."""
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c == "/" and i + 1 < n and src[i + 1] == "/":
            j = src.find("\n", i)
            i = n if j < 0 else j
            out.append(" ")
        elif c == "/" and i + 1 < n and src[i + 1] == "*":
            j = src.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        elif c in "\"'":
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def source_digest() -> str:
    """sha256 over the library's kernel and ABI sources (comments and
    whitespace left out), in name order."""
    h = hashlib.sha256()
    csrc = os.path.join(HERE, "csrc")
    paths = sorted(os.path.join(csrc, f) for f in os.listdir(csrc)
                   if f.endswith((".hip", ".h", ".cpp")))
    paths.append(os.path.join(ROOT, "include", "wide.h"))
    for p in paths:
        h.update(os.path.basename(p).encode())
        with open(p, encoding="utf-8") as f:
            h.update(code_text(f.read()).encode())
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


XCDS, SIMDS_PER_XCD, CUS_PER_XCD = 8, 128, 32


def pmc_means(paths) -> dict:
    """{kernel key: {counter: mean per dispatch, 'dispatches': n, 'avg_us': mean duration}}
    over one or more counter dumps (one rocprofv3 --pmc run each)."""
    acc = collections.defaultdict(lambda: collections.defaultdict(list))
    dur = collections.defaultdict(dict)
    for n, path in enumerate(paths):
        with open(path) as f:
            for r in csv.DictReader(f):
                k = kernel_key(r["Kernel_Name"])
                acc[k][r["Counter_Name"] + "@%d" % n].append(float(r["Counter_Value"]))
                if r.get("Start_Timestamp") and r.get("End_Timestamp"):
                    dur[k][(n, r.get("Dispatch_Id"))] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
    out = {}
    for k, cs in acc.items():
        m = {}
        for c, v in cs.items():
            name, n = c.rsplit("@", 1)
            m.setdefault(name, {})[n] = sum(v) / len(v)
        # a counter in several passes (GRBM_GUI_ACTIVE) is kept per pass
        out[k] = {"passes": m, "dispatches": max(len(v) for v in cs.values()),
                  "avg_us": (sum(dur[k].values()) / len(dur[k])) if dur[k] else None}
    return out


def mfma_summary(paths, command: str, min_us: float = 5.0) -> dict:
    raw = pmc_means(paths)
    kernels = {}
    for k, v in raw.items():
        us = v["avg_us"]
        if us is None or us < min_us:
            continue
        p = v["passes"]

        def get(name):
            d = p.get(name)
            return None if not d else sum(d.values()) / len(d)

        def same_pass(num, den):
            """num / den with both counters taken in one pass where possible."""
            dn, dd = p.get(num), p.get(den)
            if not dn or not dd:
                return None
            common = set(dn) & set(dd)
            if common:
                n = sorted(common)[0]
                return dn[n] / dd[n] if dd[n] else None
            a, b = get(num), get(den)
            return a / b if b else None

        grbm = get("GRBM_GUI_ACTIVE")
        row = {"dispatches": v["dispatches"], "avg_us": round(us, 2)}
        if grbm:
            row["clock_GHz"] = round(grbm / XCDS / (us * 1e3), 3)
        busy = same_pass("SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE")
        if busy is not None:
            row["mfma_busy"] = round(busy / SIMDS_PER_XCD, 4)  # per SIMD-cycle
        for name, num, den, scale in (("wait_any", "SQ_WAIT_ANY", "SQ_WAVE_CYCLES", 1.0),
                                      ("wait_lds", "SQ_WAIT_INST_LDS", "SQ_WAVE_CYCLES", 1.0),
                                      ("lds_fifo_full", "SQ_LDS_CMD_FIFO_FULL", "GRBM_GUI_ACTIVE", 1.0 / CUS_PER_XCD),
                                      ("lds_data_fifo_full", "SQ_LDS_DATA_FIFO_FULL", "GRBM_GUI_ACTIVE",
                                       1.0 / CUS_PER_XCD),
                                      ("lds_conflict", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", 1.0)):
            r = same_pass(num, den)
            if r is not None:
                row[name] = round(r * scale, 4)
        row["counters"] = {c: round(get(c), 1) for c in sorted(p)}
        kernels[k] = row
    return dict(command=command, passes=len(paths), source_sha256=source_digest(),
                normalisation="GRBM_GUI_ACTIVE summed over 8 XCDs; SQ busy counters over 1024 SIMDs; "
                              "kernels launched for less than min_us are left out: GRBM_GUI_ACTIVE also "
                              "counts cycles around a launch, which only long launches make negligible; "
                              "launches of one kernel name (e.g. a library GEMM used at several shapes) "
                              "are averaged together",
                min_us=min_us,
                kernels=dict(sorted(kernels.items(), key=lambda kv: -kv[1]["avg_us"] * kv[1]["dispatches"])))


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
    mf = sub.add_parser("mfma")
    mf.add_argument("--pmc", nargs="+", required=True)
    mf.add_argument("--command", required=True)
    mf.add_argument("--min-us", type=float, default=5.0)
    mf.add_argument("--out", required=True)
    a = ap.parse_args()
    if a.what == "mfma":
        s = mfma_summary(a.pmc, a.command, a.min_us)
        with open(a.out, "w") as f:
            json.dump(s, f, indent=1)
        print(json.dumps({k: {kk: vv for kk, vv in v.items() if kk != "counters"} for k, v in s["kernels"].items()},
                         indent=1))
    elif a.what == "counters":
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
