"""Summarise rocprofv3 CSV output of bench.py per kernel and launch grid.

    python rocprof_summary.py TRACE_DIR [--fetch PMC_DIR] [--write PMC_DIR] [--copy-bytes B]
        [--traffic-json OUT --kernel SUBSTRING --workload NAME --source FILE --tile V
         --command CMD ...]

TRACE_DIR holds the *_kernel_trace.csv of a `rocprofv3 --kernel-trace
--stats --output-format csv` run; PMC_DIR the *_counter_collection.csv of a
`rocprofv3 --pmc FETCH_SIZE` (or WRITE_SIZE) run of the same command.
Launches of one kernel symbol are split by grid size, because the routed and
the shared-expert GEMMs share a symbol.  Counter values (KiB per dispatch)
are also reported scaled by the reading of the plain device copy kernel
(__amd_rocclr_copyBuffer) of --copy-bytes bytes, which moves that many bytes
each way; the copy dispatches taken are those reading the most.

With --traffic-json, the calibrated HBM bytes per launch (FETCH + WRITE) of
the one kernel whose short name contains --kernel are written to OUT, with
the sha256 of the kernel's source file, so that a reader of OUT can tell
whether the counters still describe the current kernel.
"""

import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import re


def short(name):
    name = name.replace("(anonymous namespace)::", "").replace("void ", "")
    name = re.sub(r"\(.*", "", name)
    return name.replace("fs::", "").replace("at::native::", "torch:")[:60]


def one(pattern):
    files = glob.glob(pattern)
    if not files:
        raise SystemExit(f"no file matches {pattern}")
    return files[0]


def trace_table(trace_dir):
    rows = list(csv.DictReader(open(one(os.path.join(trace_dir, "*_kernel_trace.csv")))))
    agg = collections.defaultdict(list)
    for r in rows:
        key = (short(r["Kernel_Name"]), int(r["Grid_Size_X"]))
        agg[key].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    return agg


def counter_table(pmc_dir, counter):
    rows = list(csv.DictReader(open(one(os.path.join(pmc_dir, "*_counter_collection.csv")))))
    agg = collections.defaultdict(list)
    for r in rows:
        if r["Counter_Name"] == counter:
            agg[(short(r["Kernel_Name"]), int(r["Grid_Size"]))].append(float(r["Counter_Value"]))
    return agg


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("trace_dir")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-bytes", type=float, default=None)
    ap.add_argument("--min-us", type=float, default=1.0)
    ap.add_argument("--traffic-json")
    ap.add_argument("--kernel")
    ap.add_argument("--workload")
    ap.add_argument("--source")
    ap.add_argument("--tile", default="")
    ap.add_argument("--command", action="append", default=[])
    a = ap.parse_args()
    scales, kib = {}, {}
    agg = trace_table(a.trace_dir)
    print("| kernel | grid (threads) | launches | avg us | min us | max us |")
    print("|---|---|---|---|---|---|")
    for (k, g), v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        avg = sum(v) / len(v)
        if avg < a.min_us:
            continue
        print(f"| {k} | {g} | {len(v)} | {avg:.2f} | {min(v):.2f} | {max(v):.2f} |")
    for label, d, ctr in (("FETCH_SIZE", a.fetch, "FETCH_SIZE"), ("WRITE_SIZE", a.write, "WRITE_SIZE")):
        if not d:
            continue
        t = counter_table(d, ctr)
        # the reference copy: the largest copy-kernel dispatches (those
        # within 5% of the largest reading), i.e. the --copy-bytes copy
        copy = [v for (k, g), vs in t.items() if k.startswith("__amd_rocclr_copyBuffer") for v in vs]
        copy = [v for v in copy if copy and v >= 0.95 * max(copy)]
        scale = None
        if copy and a.copy_bytes:
            scale = a.copy_bytes / 1024.0 / (sum(copy) / len(copy))
        print()
        print(f"{label} (KiB per dispatch; calibrated = x {scale:.4f} so that the copy kernel reads "
              f"{a.copy_bytes:.0f} bytes)" if scale else f"{label} (KiB per dispatch)")
        print()
        print("| kernel | grid | dispatches | avg KiB | calibrated MB |")
        print("|---|---|---|---|---|")
        scales[label] = scale
        for (k, g), v in sorted(t.items(), key=lambda kv: -sum(kv[1])):
            avg = sum(v) / len(v)
            if a.kernel and a.kernel in k:
                kib.setdefault(label, []).append((k, g, avg))
            cal = f"{avg * scale * 1024 / 1e6:.1f}" if scale else "-"
            print(f"| {k} | {g} | {len(v)} | {avg:.0f} | {cal} |")
    if a.traffic_json:
        for label in ("FETCH_SIZE", "WRITE_SIZE"):
            if len(kib.get(label, [])) != 1 or not scales.get(label):
                raise SystemExit(f"--traffic-json: {label} needs one calibrated kernel matching "
                                 f"{a.kernel!r}, found {kib.get(label)}")
        (kname, grid, fetch), = kib["FETCH_SIZE"]
        (_, _, write), = kib["WRITE_SIZE"]
        total = (fetch * scales["FETCH_SIZE"] + write * scales["WRITE_SIZE"]) * 1024
        rec = {"kernel": f"{kname} (grid {grid} threads)", "workload": a.workload,
               "tile": a.tile, "source": a.source,
               "source_sha256": hashlib.sha256(open(a.source, "rb").read()).hexdigest(),
               "fetch_kib_per_dispatch": round(fetch), "fetch_scale": round(scales["FETCH_SIZE"], 4),
               "write_kib_per_dispatch": round(write), "write_scale": round(scales["WRITE_SIZE"], 4),
               "copy_reference_bytes": int(a.copy_bytes), "hbm_bytes_per_launch": int(total),
               "commands": a.command}
        with open(a.traffic_json, "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")


if __name__ == "__main__":
    main()
