"""Summarise rocprofv3 results databases (SQLite) as text tables.

  python -m paper_2202_01258_amd.rocprof_summary <results.db> [--top N]
      kernel trace: kernel, calls, total and average duration
  python -m paper_2202_01258_amd.rocprof_summary --pmc <results.db> [--top N]
      counters (--pmc runs): kernel, counter, dispatches, mean value per dispatch
"""
from __future__ import annotations

import argparse
import sqlite3


def summary(db_path: str, top: int = 20) -> str:
    con = sqlite3.connect(db_path)
    rows = con.execute(
        "select name, count(*), sum(end - start), avg(end - start), min(end - start), "
        "max(end - start) from kernels group by name order by sum(end - start) desc").fetchall()
    total = sum(r[2] for r in rows) or 1
    out = [f"{'kernel':70s} {'calls':>6s} {'total_us':>11s} {'avg_us':>9s} "
           f"{'min_us':>9s} {'max_us':>9s} {'pct':>6s}"]
    for name, calls, tot, avg, mn, mx in rows[:top]:
        out.append(f"{name[:70]:70s} {calls:6d} {tot / 1e3:11.3f} {avg / 1e3:9.3f} "
                   f"{mn / 1e3:9.3f} {mx / 1e3:9.3f} {100.0 * tot / total:6.2f}")
    return "\n".join(out)


def pmc_summary(db_path: str, top: int = 20) -> str:
    con = sqlite3.connect(db_path)
    rows = con.execute(
        "select name, counter_name, count(*), avg(counter_value), min(counter_value), "
        "max(counter_value) from pmc_events group by name, counter_name "
        "order by avg(counter_value) * count(*) desc").fetchall()
    out = [f"{'kernel':70s} {'counter':>14s} {'calls':>6s} {'mean':>14s} {'min':>14s} "
           f"{'max':>14s}"]
    for name, ctr, calls, mean, mn, mx in rows[:top]:
        out.append(f"{name[:70]:70s} {ctr:>14s} {calls:6d} {mean:14.2f} {mn:14.2f} {mx:14.2f}")
    return "\n".join(out)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("db")
    ap.add_argument("--top", type=int, default=20)
    ap.add_argument("--pmc", action="store_true")
    a = ap.parse_args()
    print(pmc_summary(a.db, a.top) if a.pmc else summary(a.db, a.top))


if __name__ == "__main__":
    main()
