"""Summarise rocprofv3 output.

Kernel trace (rocpd SQLite output, or the kernel_stats.csv of
--output-format csv) as markdown:
    python -m paper_2608_07974_amd.profile_summary RESULTS_DB|KERNEL_STATS_CSV [--top N]
prints per kernel: calls, total and average duration (from the trace's
top_kernels view), and the share of the traced GPU time.

Counter collection (--pmc ... --output-format csv):
    python -m paper_2608_07974_amd.profile_summary --pmc COUNTER_CSV --kernel SUBSTR
prints, per counter, the dispatch count and the mean per dispatch of every
kernel whose name contains SUBSTR (counter instances summed per dispatch).

Counter report (a kernel trace and counter CSVs of the same program):
    python -m paper_2608_07974_amd.profile_summary --report KERNEL_TRACE.csv \
        --pmc-csvs A.csv B.csv ... --copy COPY_FETCH.csv COPY_WRITE.csv
prints per kernel the effective clock, MFMA busy %, executed bf16 MFMA
TFLOP/s, LDS bank conflicts and HBM bytes and rate.

HBM traffic record (four counter CSVs: FETCH_SIZE and WRITE_SIZE over the
workload and over the 1 GiB copy calibration):
    python -m paper_2608_07974_amd.profile_summary --traffic-record OUT.json \
        --fetch BENCH.csv COPY.csv --write BENCH.csv COPY.csv \
        --kernel SUBSTR --name NAME --workload W --source FILE
writes the per-launch bytes (each counter scaled by true copy bytes over
what it read for the copy) with the sha256 of the kernel's source file.
"""
import argparse
import sqlite3


def summarise(db_path, top=20):
    db = sqlite3.connect(db_path)
    rows = list(db.execute("select name, total_calls, total_duration, average, percentage "
                           "from top_kernels order by total_duration desc"))
    out = ["| kernel | calls | total ms | avg us | share % |", "|---|---:|---:|---:|---:|"]
    for name, calls, total, avg, pct in rows[:top]:
        short = name.split("(")[0].replace("void ", "")
        out.append(f"| `{short}` | {calls} | {total / 1e3:.2f} | {avg:.1f} | {pct:.2f} |")
    return "\n".join(out)


def summarise_stats_csv(path, top=20):
    """The same table from the kernel_stats.csv that --stats writes with
    --output-format csv."""
    rows = sorted(_csv_rows(path), key=lambda r: -float(r["TotalDurationNs"]))
    out = ["| kernel | calls | total ms | avg us | share % |", "|---|---:|---:|---:|---:|"]
    for r in rows[:top]:
        short = r["Name"].split("(")[0].replace("void ", "")
        out.append(f"| `{short}` | {r['Calls']} | {float(r['TotalDurationNs']) / 1e6:.2f} | "
                   f"{float(r['AverageNs']) / 1e3:.1f} | {float(r['Percentage']):.2f} |")
    return "\n".join(out)


def pmc_means(csv_path, kernel):
    """{counter: (dispatches, mean per dispatch)} over dispatches of kernels
    whose name contains `kernel`."""
    import collections
    import csv
    per = collections.defaultdict(lambda: collections.defaultdict(float))
    with open(csv_path) as f:
        for r in csv.DictReader(f):
            if kernel in r["Kernel_Name"]:
                per[r["Counter_Name"]][r["Dispatch_Id"]] += float(r["Counter_Value"])
    return {c: (len(d), sum(d.values()) / len(d)) for c, d in per.items() if d}


def traffic_record(fetch, write, kernel, name, workload, source, copy_bytes=1 << 30):
    import hashlib
    ff = pmc_means(fetch[0], kernel)["FETCH_SIZE"]
    fw = pmc_means(write[0], kernel)["WRITE_SIZE"]
    cf = pmc_means(fetch[1], "copyBuffer")["FETCH_SIZE"][1]
    cw = pmc_means(write[1], "copyBuffer")["WRITE_SIZE"][1]
    kf, kw = copy_bytes / 1024 / cf, copy_bytes / 1024 / cw  # true KiB per counted KiB
    full = ""
    import csv
    with open(fetch[0]) as f:
        for r in csv.DictReader(f):
            if kernel in r["Kernel_Name"]:
                full = r["Kernel_Name"].split("(zl::")[0].replace("void ", "")
                break
    with open(source, "rb") as f:
        sha = hashlib.sha256(f.read()).hexdigest()
    return {"kernel": name, "workload": workload, "rocprof_kernel": full, "source_sha256": sha,
            "dispatches": ff[0], "fetch_kib_per_dispatch": ff[1], "write_kib_per_dispatch": fw[1],
            "copy_factor_fetch": round(kf, 5), "copy_factor_write": round(kw, 5),
            "hbm_bytes_per_launch": int(round((ff[1] * kf + fw[1] * kw) * 1024))}


def short_name(full):
    """Kernel name without namespace and arguments; the direct-to-LDS GEMM
    as gemm_dma_<BM>x<BN>_<layout> (k: K-major, m/n: MN-major operand), as
    the library's own profiler names its launches."""
    import re
    name = full.replace("void ", "").split("(")[0].strip()
    name = re.sub(r"^zl::", "", name)
    m = re.match(r"gemm_dma_kernel<(\d+), (\d+), \d+, \d+, \d+, \d+, \d+, (\w+), (\w+)", name)
    if m:
        return (f"gemm_dma_{m.group(1)}x{m.group(2)}_"
                f"{'k' if m.group(3) == 'true' else 'm'}{'k' if m.group(4) == 'true' else 'n'}")
    return name.split("<")[0]


def _csv_rows(path):
    import csv
    with open(path) as f:
        return list(csv.DictReader(f))


def trace_durations(trace_csv):
    """{short kernel name: (dispatches, mean duration ns)} from a
    --kernel-trace CSV."""
    import collections
    acc = collections.defaultdict(list)
    for r in _csv_rows(trace_csv):
        acc[short_name(r["Kernel_Name"])].append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    return {k: (len(v), sum(v) / len(v)) for k, v in acc.items()}


def counter_means(csv_paths):
    """{short kernel name: {counter: mean per dispatch}} over every
    counter-collection CSV (instances of a counter summed per dispatch)."""
    import collections
    per = collections.defaultdict(lambda: collections.defaultdict(lambda: collections.defaultdict(float)))
    for path in csv_paths:
        for r in _csv_rows(path):
            k = short_name(r["Kernel_Name"])
            per[k][r["Counter_Name"]][(path, r["Dispatch_Id"])] += float(r["Counter_Value"])
    return {k: {c: sum(d.values()) / len(d) for c, d in cs.items()} for k, cs in per.items()}


def counter_report(trace_csv, pmc_csvs, copy_fetch, copy_write, xcc=8, simds=1024, cus=256,
                   copy_bytes=1 << 30, min_share=0.001):
    """Markdown table per kernel: time share, mean duration, effective clock
    (GRBM_GUI_ACTIVE cycles per XCC over the duration), MFMA busy % (MFMA
    busy cycles over GUI-active cycles x SIMDs), executed bf16 MFMA TFLOP/s
    (MOPS x 512 per duration), LDS bank-conflict cycles per LDS-active cycle,
    HBM bytes read and written (FETCH_SIZE, WRITE_SIZE scaled by the 1 GiB
    copy) and their rate."""
    dur = trace_durations(trace_csv)
    cm = counter_means(pmc_csvs)
    def copy_kib(path, counter):
        cm_copy = counter_means([path])
        return next(v[counter] for k, v in cm_copy.items() if "copyBuffer" in k)
    kf = copy_bytes / 1024 / copy_kib(copy_fetch, "FETCH_SIZE")
    kw = copy_bytes / 1024 / copy_kib(copy_write, "WRITE_SIZE")
    total = sum(n * d for n, d in dur.values())
    lines = ["| kernel | dispatches | share % | mean us | clock MHz | MFMA busy % | bf16 MFMA TFLOP/s "
             "| LDS conflict / active | read GB | written GB | HBM GB/s |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    rows = []
    for k, (n, d) in sorted(dur.items(), key=lambda kv: -kv[1][0] * kv[1][1]):
        if n * d / total < min_share or k not in cm:
            continue
        c = cm[k]
        gui = c.get("GRBM_GUI_ACTIVE", 0.0) / xcc
        clock = gui / d * 1e3 if gui else float("nan")
        mfma = 100.0 * c["SQ_VALU_MFMA_BUSY_CYCLES"] / (gui * simds) if gui and "SQ_VALU_MFMA_BUSY_CYCLES" in c else float("nan")
        tf = c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) * 512 / (d * 1e-9) / 1e12
        lds = (c["SQ_LDS_BANK_CONFLICT"] / c["SQ_LDS_IDX_ACTIVE"]
               if c.get("SQ_LDS_IDX_ACTIVE") else float("nan"))
        rd = c.get("FETCH_SIZE", float("nan")) * 1024 * kf / 1e9
        wr = c.get("WRITE_SIZE", float("nan")) * 1024 * kw / 1e9
        gbs = (rd + wr) / (d * 1e-9)
        rows.append(dict(kernel=k, dispatches=n, share=n * d / total, mean_us=d / 1e3, clock_mhz=clock,
                         mfma_busy_pct=mfma, mfma_tflops=tf, lds_conflict=lds, read_gb=rd,
                         write_gb=wr, hbm_gbs=gbs))
        lines.append(f"| `{k}` | {n} | {100 * n * d / total:.1f} | {d / 1e3:.1f} | {clock:.0f} | "
                     f"{mfma:.1f} | {tf:.0f} | {lds:.3f} | {rd:.3f} | {wr:.3f} | {gbs:.0f} |")
    return "\n".join(lines), rows, dict(copy_factor_fetch=kf, copy_factor_write=kw)


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("db", nargs="?")
    ap.add_argument("--top", type=int, default=20)
    ap.add_argument("--pmc", default=None, help="counter-collection CSV")
    ap.add_argument("--kernel", default="", help="kernel-name substring (with --pmc)")
    ap.add_argument("--traffic-record", default=None, help="write the HBM traffic JSON here")
    ap.add_argument("--fetch", nargs=2, default=None)
    ap.add_argument("--write", nargs=2, default=None)
    ap.add_argument("--name", default="")
    ap.add_argument("--workload", default="")
    ap.add_argument("--source", default="")
    ap.add_argument("--report", default=None,
                    help="counter report: kernel-trace CSV, then --pmc-csvs and --copy")
    ap.add_argument("--pmc-csvs", nargs="+", default=[])
    ap.add_argument("--copy", nargs=2, default=None, help="FETCH and WRITE CSVs of the copy")
    ap.add_argument("--json", default=None, help="also write the report rows here")
    a = ap.parse_args()
    if a.report:
        import json
        md, rows, cal = counter_report(a.report, a.pmc_csvs, a.copy[0], a.copy[1])
        print(md)
        if a.json:
            with open(a.json, "w") as f:
                json.dump(dict(rows=rows, **cal), f, indent=1)
    elif a.traffic_record:
        import json
        rec = traffic_record(a.fetch, a.write, a.kernel, a.name, a.workload, a.source)
        with open(a.traffic_record, "w") as f:
            json.dump({"kernels": [rec]}, f, indent=1)
        print(json.dumps(rec, indent=1))
    elif a.db and a.db.endswith(".csv"):
        print(summarise_stats_csv(a.db, a.top))
    elif a.pmc:
        for c, (n, mean) in sorted(pmc_means(a.pmc, a.kernel).items()):
            print(f"{c}: dispatches {n}, mean per dispatch {mean:.6g}")
    else:
        print(summarise(a.db, a.top))
