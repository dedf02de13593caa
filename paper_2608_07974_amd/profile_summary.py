"""Summarise rocprofv3 output.

Kernel trace (rocpd SQLite output) as markdown:
    python -m paper_2608_07974_amd.profile_summary RESULTS_DB [--top N]
prints per kernel: calls, total and average duration (from the trace's
top_kernels view), and the share of the traced GPU time.

Counter collection (--pmc ... --output-format csv):
    python -m paper_2608_07974_amd.profile_summary --pmc COUNTER_CSV --kernel SUBSTR
prints, per counter, the dispatch count and the mean per dispatch of every
kernel whose name contains SUBSTR (counter instances summed per dispatch).

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
    a = ap.parse_args()
    if a.traffic_record:
        import json
        rec = traffic_record(a.fetch, a.write, a.kernel, a.name, a.workload, a.source)
        with open(a.traffic_record, "w") as f:
            json.dump({"kernels": [rec]}, f, indent=1)
        print(json.dumps(rec, indent=1))
    elif a.pmc:
        for c, (n, mean) in sorted(pmc_means(a.pmc, a.kernel).items()):
            print(f"{c}: dispatches {n}, mean per dispatch {mean:.6g}")
    else:
        print(summarise(a.db, a.top))
