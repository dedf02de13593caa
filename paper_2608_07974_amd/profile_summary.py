"""Summarise rocprofv3 output.

Kernel trace (rocpd SQLite output) as markdown:
    python -m paper_2608_07974_amd.profile_summary RESULTS_DB [--top N]
prints per kernel: calls, total and average duration (from the trace's
top_kernels view), and the share of the traced GPU time.

Counter collection (--pmc ... --output-format csv):
    python -m paper_2608_07974_amd.profile_summary --pmc COUNTER_CSV --kernel SUBSTR
prints, per counter, the dispatch count and the mean per dispatch of every
kernel whose name contains SUBSTR (counter instances summed per dispatch).
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


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("db", nargs="?")
    ap.add_argument("--top", type=int, default=20)
    ap.add_argument("--pmc", default=None, help="counter-collection CSV")
    ap.add_argument("--kernel", default="", help="kernel-name substring (with --pmc)")
    a = ap.parse_args()
    if a.pmc:
        for c, (n, mean) in sorted(pmc_means(a.pmc, a.kernel).items()):
            print(f"{c}: dispatches {n}, mean per dispatch {mean:.6g}")
    else:
        print(summarise(a.db, a.top))
