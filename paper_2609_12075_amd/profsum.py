"""Summaries of rocprofv3 output for the kernels of this library.

    python -m paper_2609_12075_amd.profsum stats <kernel_stats.csv> [--top N]
    python -m paper_2609_12075_amd.profsum trace <kernel_trace.csv> --kernel REGEX [--last N]
    python -m paper_2609_12075_amd.profsum traffic --fetch <pmc.csv> --write <pmc.csv> \
        --kernel REGEX --copy-bytes N [--out traffic.json]
    python -m paper_2609_12075_amd.profsum mfma <pmc.csv>   (a MfmaUtil + MfmaFlopsBF16 pass)

`traffic` scales the per-dispatch FETCH_SIZE / WRITE_SIZE counters (KiB) of
the named kernel by what the same counters read for the 256 MiB device copy
that `bench.py --copy-probe` runs (rocclr's copyBuffer kernel), and records
the hash of the GEMM source so the figure is dropped once the kernel changes.
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os
import re
import statistics
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
GEMM_SOURCE = os.path.join(PKG, "csrc", "k_gemm.hip")


def source_hash(path: str = GEMM_SOURCE) -> str:
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def stats(path: str, top: int = 20) -> str:
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    tot = sum(float(r["TotalDurationNs"]) for r in rows)
    out = [f"{'total ms':>9} {'%':>6} {'calls':>7} {'avg us':>9}  kernel"]
    for r in rows[:top]:
        out.append(f"{float(r['TotalDurationNs']) / 1e6:9.3f} {float(r['TotalDurationNs']) / tot * 100:6.2f} "
                   f"{int(r['Calls']):7d} {float(r['AverageNs']) / 1e3:9.2f}  {r['Name'][:120]}")
    out.append(f"all kernels: {tot / 1e6:.3f} ms")
    return "\n".join(out)


def trace(path: str, kernel: str, last: int = 0) -> str:
    """Per (kernel, grid) dispatch durations; with last > 0 also the mean of
    each group's last `last` dispatches in time order (a benchmark's final
    replay phase of one projection, timed there with HIP events)."""
    rows = [r for r in csv.DictReader(open(path)) if re.search(kernel, r["Kernel_Name"])]
    g = collections.defaultdict(list)
    for r in rows:
        key = (r["Kernel_Name"][:100], r["Grid_Size_X"], r["Grid_Size_Y"], r["Grid_Size_Z"])
        g[key].append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
    head = f"{'calls':>6} {'avg us':>9} {'median us':>10}"
    if last:
        head += f" {'last ' + str(last) + ' avg us':>16}"
    out = [head + "  grid (threads)  kernel"]
    for k, v in sorted(g.items(), key=lambda kv: -sum(d for _, d in kv[1])):
        d = [x for _, x in v]
        line = f"{len(d):6d} {sum(d) / len(d) / 1e3:9.2f} {statistics.median(d) / 1e3:10.2f}"
        if last:
            tail = [x for _, x in sorted(v)[-last:]]
            line += f" {sum(tail) / len(tail) / 1e3:16.2f}"
        out.append(line + f"  ({k[1]},{k[2]},{k[3]})  {k[0]}")
    return "\n".join(out)


def _counter(path: str, name: str, kernel: str):
    vals = collections.defaultdict(float)
    for r in csv.DictReader(open(path)):
        if r.get("Counter_Name") == name and re.search(kernel, r.get("Kernel_Name", "")):
            vals[r.get("Dispatch_Id", r.get("Correlation_Id"))] += float(r["Counter_Value"])
    return list(vals.values())


def traffic(fetch_csv: str, write_csv: str, kernel: str, copy_bytes: int) -> dict:
    copy_re = "copyBuffer"
    f_k, w_k = _counter(fetch_csv, "FETCH_SIZE", kernel), _counter(write_csv, "WRITE_SIZE", kernel)
    f_c, w_c = _counter(fetch_csv, "FETCH_SIZE", copy_re), _counter(write_csv, "WRITE_SIZE", copy_re)
    if not (f_k and w_k and f_c and w_c):
        raise SystemExit("missing counters for the kernel or the copy probe")
    # the copy reads and writes copy_bytes: scale = bytes per counted KiB
    f_scale = copy_bytes / (max(f_c) * 1024.0)
    w_scale = copy_bytes / (max(w_c) * 1024.0)
    fetch = statistics.median(f_k) * 1024.0 * f_scale
    write = statistics.median(w_k) * 1024.0 * w_scale
    return {"kernel_regex": kernel, "source_hash": source_hash(), "fetch_bytes": fetch, "write_bytes": write,
            "traffic_bytes": fetch + write, "fetch_scale": f_scale, "write_scale": w_scale,
            "dispatches": len(f_k)}


def mfma(path: str) -> str:
    """Per kernel of a `--pmc MfmaUtil MfmaFlopsBF16` pass: dispatches, median
    dispatch duration (counter collection serialises dispatches), counted
    matrix flops per dispatch / that duration, and the mean MfmaUtil."""
    disp = collections.defaultdict(dict)
    for r in csv.DictReader(open(path)):
        d = disp[r["Dispatch_Id"]]
        d["name"] = r["Kernel_Name"]
        d["ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        d[r["Counter_Name"]] = float(r["Counter_Value"])
    g = collections.defaultdict(list)
    for d in disp.values():
        if "MfmaFlopsBF16" in d and "MfmaUtil" in d:
            g[d["name"]].append(d)
    out = [f"{'dispatches':>10} {'median us':>10} {'TFLOP/s':>8} {'MfmaUtil %':>10}  kernel"]
    for name, ds in sorted(g.items(), key=lambda kv: -sum(x["ns"] for x in kv[1])):
        med = statistics.median(x["ns"] for x in ds)
        fl = statistics.median(x["MfmaFlopsBF16"] for x in ds)
        util = sum(x["MfmaUtil"] for x in ds) / len(ds)
        out.append(f"{len(ds):10d} {med / 1e3:10.1f} {fl / med / 1e3:8.0f} {util:10.1f}  {name[:110]}")
    return "\n".join(out)


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats"); s.add_argument("csv"); s.add_argument("--top", type=int, default=20)
    t = sub.add_parser("trace"); t.add_argument("csv"); t.add_argument("--kernel", default=".")
    t.add_argument("--last", type=int, default=0)
    f = sub.add_parser("traffic")
    f.add_argument("--fetch", required=True); f.add_argument("--write", required=True)
    f.add_argument("--kernel", required=True); f.add_argument("--copy-bytes", type=int, required=True)
    f.add_argument("--out")
    mf = sub.add_parser("mfma"); mf.add_argument("csv")
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        print(stats(a.csv, a.top))
    elif a.cmd == "trace":
        print(trace(a.csv, a.kernel, a.last))
    elif a.cmd == "mfma":
        print(mfma(a.csv))
    else:
        res = traffic(a.fetch, a.write, a.kernel, a.copy_bytes)
        js = json.dumps(res, indent=1)
        print(js)
        if a.out:
            open(a.out, "w").write(js + "\n")


if __name__ == "__main__":
    main(sys.argv[1:])
