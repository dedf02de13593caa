"""Summarise a rocprofv3 kernel trace (rocpd SQLite output) as markdown.

Usage: python -m paper_2608_07974_amd.profile_summary RESULTS_DB [--top N]
Prints per kernel: calls, total and average duration (from the trace's
top_kernels view), and the share of the traced GPU time.
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


if __name__ == "__main__":
    ap = argparse.ArgumentParser()
    ap.add_argument("db")
    ap.add_argument("--top", type=int, default=20)
    a = ap.parse_args()
    print(summarise(a.db, a.top))
