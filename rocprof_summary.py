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

With --overlap, it instead reports, for every copy dispatched on the stream
that carries the largest copies (the Dispatch stand-in), the fraction of the
copy's interval during which a kernel of another stream runs:
|copy ∩ (∪ compute kernels)| / |copy|; --copy-kernel selects the copies by
kernel name (the HBM-speed blit by default, paced_copy for the link-paced
stand-in copies).

With --mfma PMC_DIR (a `rocprofv3 --pmc GRBM_GUI_ACTIVE SQ_VALU_MFMA_BUSY_CYCLES
SQ_INSTS_VALU_MFMA_MOPS_BF16` run), it reports per kernel the fraction of
cycles the MFMA units were busy, SQ_VALU_MFMA_BUSY_CYCLES summed over the
1024 SIMDs / (GRBM_GUI_ACTIVE summed over the 8 XCDs * 128), and the clock
the kernel ran at, GRBM_GUI_ACTIVE / 8 / its duration in the trace.

With --memory PMC_DIR (repeatable; runs holding TCP_TCC_READ_REQ_LATENCY_sum,
TCP_TCC_READ_REQ_sum, TCP_PENDING_STALL_CYCLES_sum, TA_TA_BUSY_sum,
TCC_HIT_sum, TCC_MISS_sum and GRBM_GUI_ACTIVE), it reports per GEMM kernel
the mean L1 -> L2 read latency in cycles, the L2 hit rate, and the shares of
CU cycles in which the L1 waits on pending L2 data and the TA is busy.

With --window SUBSTRING START COUNT, it also prints the mean duration of
launches START .. START+COUNT-1 (in start order, from 0) of the one kernel
whose short name contains SUBSTRING: bench.py runs warm-up steps, the timed
steps and then an untimed pass with every kernel's events on, so the timed
steps' launches are a window of the trace.

With --split SUBSTRING N, the launches of a kernel whose short name
contains SUBSTRING are told apart by their launch index modulo N (shown as
"name #i"): one step may launch the same kernel for two passes, e.g. the
shared and then the routed gate/up.

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
    return name.replace("fs::", "").replace("at::native::", "torch:")[:90]


# --split SUBSTRING N: launches of a kernel whose short name contains
# SUBSTRING are told apart by their index in launch order modulo N (a pass
# that two calls of one step make with the same kernel, e.g. the shared and
# the routed gate/up), shown as "name #i".
SPLIT = None


def named(rows, order_field):
    """(short name with the --split class, row) in the rows' launch order."""
    out, seen = [], collections.Counter()
    # (files without the field keep their own order: the sort is stable)
    for r in sorted(rows, key=lambda r: int(r.get(order_field) or 0)):
        k = short(r["Kernel_Name"])
        if SPLIT and SPLIT[0] in k:
            i = seen[k]
            seen[k] += 1
            k = f"{k} #{i % SPLIT[1]}"
        out.append((k, r))
    return out


def one(pattern):
    files = glob.glob(pattern)
    if not files:
        raise SystemExit(f"no file matches {pattern}")
    return files[0]


def trace_table(trace_dir):
    rows = list(csv.DictReader(open(one(os.path.join(trace_dir, "*_kernel_trace.csv")))))
    agg = collections.defaultdict(list)
    for k, r in named(rows, "Start_Timestamp"):
        key = (k, int(r["Grid_Size_X"]))
        agg[key].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    return agg


def window_report(trace_dir, substring, start, count):
    rows = named(list(csv.DictReader(open(one(os.path.join(trace_dir, "*_kernel_trace.csv"))))),
                 "Start_Timestamp")
    names = {k for k, _ in rows if substring in k}
    if len(names) != 1:
        raise SystemExit(f"--window: {substring!r} matches {sorted(names)}")
    name, = names
    sel = [r for k, r in rows if k == name][start:start + count]
    if len(sel) != count:
        raise SystemExit(f"--window: {name} has {len(sel)} launches in [{start}, {start + count})")
    d = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in sel]
    print()
    print(f"{name}: launches {start}..{start + count - 1} (start order) average "
          f"{sum(d) / len(d):.2f} us (min {min(d):.2f}, max {max(d):.2f})")


def overlap_report(trace_dir, min_us, skip, copy_kernel="copyBuffer", copy_stream=None):
    rows = list(csv.DictReader(open(one(os.path.join(trace_dir, "*_kernel_trace.csv")))))
    span = lambda r: (int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
    copies = [r for r in rows if copy_kernel in r["Kernel_Name"]]
    longest = max(span(r)[1] - span(r)[0] for r in copies)
    streams = {r["Stream_Id"] for r in copies if span(r)[1] - span(r)[0] >= 0.5 * longest}
    if copy_stream is not None:
        streams = {copy_stream}
    if len(streams) != 1:
        raise SystemExit(f"the largest copies run on several streams: {sorted(streams)}")
    cs = streams.pop()
    copies = [span(r) for r in copies if r["Stream_Id"] == cs and span(r)[1] - span(r)[0] >= 1e3 * min_us]
    copies = sorted(copies)[skip:]
    compute = sorted(span(r) for r in rows if r["Stream_Id"] != cs)
    # union of the compute intervals
    merged = []
    for a, b in compute:
        if merged and a <= merged[-1][1]:
            merged[-1][1] = max(merged[-1][1], b)
        else:
            merged.append([a, b])
    fr, dur = [], []
    for a, b in copies:
        cov = sum(max(0, min(b, y) - max(a, x)) for x, y in merged if y > a and x < b)
        fr.append(cov / (b - a))
        dur.append((b - a) / 1e3)
    n = len(fr)
    print(f"copy stream {cs}: {n} copies of at least {min_us} us after the first {skip}")
    print()
    print("| copies | mean copy us | mean overlap | min overlap | max overlap | mean exposed us |")
    print("|---|---|---|---|---|---|")
    exposed = [d * (1 - f) for d, f in zip(dur, fr)]
    print(f"| {n} | {sum(dur) / n:.1f} | {100 * sum(fr) / n:.1f}% | {100 * min(fr):.1f}% | "
          f"{100 * max(fr):.1f}% | {sum(exposed) / n:.1f} |")


def mfma_report(trace_dir, pmc_dir, min_us):
    agg = trace_table(trace_dir)
    cnt = {c: counter_table(pmc_dir, c) for c in ("GRBM_GUI_ACTIVE", "SQ_VALU_MFMA_BUSY_CYCLES")}
    print("| kernel | grid | avg us (trace) | MFMA busy | clock GHz |")
    print("|---|---|---|---|---|")
    for key, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        avg = sum(v) / len(v)
        grbm, busy = cnt["GRBM_GUI_ACTIVE"].get(key), cnt["SQ_VALU_MFMA_BUSY_CYCLES"].get(key)
        if avg < min_us or not grbm or not busy:
            continue
        g, b = sum(grbm) / len(grbm), sum(busy) / len(busy)
        if b == 0:
            continue
        print(f"| {key[0]} | {key[1]} | {avg:.2f} | {100 * b / (g * 128):.1f}% | {g / 8 / avg / 1e3:.2f} |")


def memory_report(trace_dir, pmc_dirs, min_us):
    """Per GEMM kernel: L1 -> L2 read latency, L2 hit rate and the share of
    cycles the L1 stalls on pending L2 data, from counter runs that hold
    TCP_TCC_READ_REQ_LATENCY_sum, TCP_TCC_READ_REQ_sum,
    TCP_PENDING_STALL_CYCLES_sum, TCC_HIT_sum, TCC_MISS_sum and
    GRBM_GUI_ACTIVE (any split over the directories)."""
    agg = trace_table(trace_dir)
    names = ("TCP_TCC_READ_REQ_LATENCY_sum", "TCP_TCC_READ_REQ_sum", "TCP_PENDING_STALL_CYCLES_sum",
             "TCC_HIT_sum", "TCC_MISS_sum", "GRBM_GUI_ACTIVE", "TA_TA_BUSY_sum")
    cnt = {}
    for d in pmc_dirs:
        for c in names:
            t = counter_table(d, c)
            if t:
                cnt[c] = t
    missing = [c for c in names if c not in cnt]
    if missing:
        raise SystemExit(f"--memory: no counter run holds {missing}")
    avg = lambda c, key: (sum(cnt[c][key]) / len(cnt[c][key])) if cnt[c].get(key) else None
    print("| kernel | grid | avg us (trace) | L2 read latency (cycles) | L2 hit rate | "
          "L1 stalled on L2 | TA busy |")
    print("|---|---|---|---|---|---|---|")
    for key, v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        t = sum(v) / len(v)
        vals = {c: avg(c, key) for c in names}
        if t < min_us or any(x is None for x in vals.values()) or not vals["TCP_TCC_READ_REQ_sum"]:
            continue
        if "gemm" not in key[0]:
            continue
        lat = vals["TCP_TCC_READ_REQ_LATENCY_sum"] / vals["TCP_TCC_READ_REQ_sum"]
        hit = vals["TCC_HIT_sum"] / (vals["TCC_HIT_sum"] + vals["TCC_MISS_sum"])
        # per-CU cycles: GRBM_GUI_ACTIVE sums the 8 XCDs; 256 CUs
        cyc = vals["GRBM_GUI_ACTIVE"] / 8 * 256
        print(f"| {key[0]} | {key[1]} | {t:.2f} | {lat:.0f} | {100 * hit:.1f}% | "
              f"{100 * vals['TCP_PENDING_STALL_CYCLES_sum'] / cyc:.1f}% | "
              f"{100 * vals['TA_TA_BUSY_sum'] / cyc:.1f}% |")


def counter_table(pmc_dir, counter):
    rows = list(csv.DictReader(open(one(os.path.join(pmc_dir, "*_counter_collection.csv")))))
    agg = collections.defaultdict(list)
    for k, r in named([r for r in rows if r["Counter_Name"] == counter], "Dispatch_Id"):
        agg[(k, int(r["Grid_Size"]))].append(float(r["Counter_Value"]))
    return agg


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("trace_dir")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-bytes", type=float, default=None)
    ap.add_argument("--min-us", type=float, default=1.0)
    ap.add_argument("--overlap", action="store_true")
    ap.add_argument("--skip", type=int, default=0, help="--overlap: leading copies to skip (warm-up)")
    ap.add_argument("--copy-kernel", default="copyBuffer",
                    help="--overlap: kernel-name substring of the copies (paced_copy: the "
                         "link-paced stand-in copies)")
    ap.add_argument("--copy-stream", default=None,
                    help="--overlap: the stream of the copies to report (when copies of both "
                         "schedules are long, e.g. link-paced copies of the regular schedule "
                         "on the compute stream)")
    ap.add_argument("--mfma")
    ap.add_argument("--memory", action="append", default=[],
                    help="counter-run directories for the GEMM memory-pipeline table")
    ap.add_argument("--traffic-json")
    ap.add_argument("--kernel")
    ap.add_argument("--workload")
    ap.add_argument("--source")
    ap.add_argument("--tile", default="")
    ap.add_argument("--command", action="append", default=[])
    ap.add_argument("--window", nargs=3, metavar=("SUBSTRING", "START", "COUNT"))
    ap.add_argument("--split", nargs=2, metavar=("SUBSTRING", "N"),
                    help="tell a kernel's launches apart by launch index modulo N")
    ap.add_argument("--all-kernels", action="store_true",
                    help="also list torch's kernels (input generation during setup)")
    a = ap.parse_args()
    global SPLIT
    if a.split:
        SPLIT = (a.split[0], int(a.split[1]))
    keep = (lambda k: True) if a.all_kernels else (lambda k: not k.startswith("torch:"))
    scales, kib = {}, {}
    if a.overlap:
        overlap_report(a.trace_dir, a.min_us, a.skip, a.copy_kernel, a.copy_stream)
        return
    if a.mfma:
        mfma_report(a.trace_dir, a.mfma, a.min_us)
        return
    if a.memory:
        memory_report(a.trace_dir, a.memory, a.min_us)
        return
    agg = trace_table(a.trace_dir)
    print("| kernel | grid (threads) | launches | avg us | min us | max us |")
    print("|---|---|---|---|---|---|")
    for (k, g), v in sorted(agg.items(), key=lambda kv: -sum(kv[1])):
        avg = sum(v) / len(v)
        if avg < a.min_us or not keep(k):
            continue
        print(f"| {k} | {g} | {len(v)} | {avg:.2f} | {min(v):.2f} | {max(v):.2f} |")
    if a.window:
        window_report(a.trace_dir, a.window[0], int(a.window[1]), int(a.window[2]))
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
            if not keep(k):
                continue
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
