"""Summarise rocprofv3 results databases (SQLite) as text tables.

  python -m paper_2202_01258_amd.rocprof_summary <results.db> [--top N] [--per-archive]
      kernel trace: kernel, calls, total and average duration; with
      --per-archive one table per archive the program created (dispatches in
      start order, a new archive beginning at each k_clear_archive)
  python -m paper_2202_01258_amd.rocprof_summary --pmc <results.db> [--top N]
      counters (--pmc runs): kernel, counter, dispatches, mean value per dispatch
  python -m paper_2202_01258_amd.rocprof_summary --traffic KERNEL \
          <copy_fetch.db> <copy_write.db> <fetch.db> <write.db> --copy-mib M
      HBM bytes per launch of KERNEL: FETCH_SIZE and WRITE_SIZE (KiB per
      dispatch) each scaled by bytes moved / counter value of a plain copy of
      M MiB, with a digest of the sources that kernel is built from
"""
from __future__ import annotations

import argparse
import hashlib
import os
import sqlite3

TRAFFIC_TAG = "traffic_bytes_per_launch"
VALU_TAG = "valu_insts_per_launch"


def _open(db_path: str) -> sqlite3.Connection:
    """A results database, read-only (no journal or lock files are created)."""
    return sqlite3.connect(f"file:{os.path.abspath(db_path)}?mode=ro&immutable=1", uri=True)


# Sources a kernel's code depends on: every kernel is built from the device
# helpers, the kernel header, the launch code and the build flags; the policy
# kernels also from the rollout header.
_COMMON = ["csrc/qd_device.hpp", "csrc/qd_kernels.hpp", "csrc/qd_lib.hip", "build.py",
           "../include/qd.h"]
_POLICY = ["csrc/qd_rollout.hpp"]


def _code_text(path: str) -> bytes:
    """A source file's code without comments and whitespace runs (C-family
    files), so that editing documentation does not void recorded counters;
    other files as they are."""
    with open(path, "rb") as fh:
        text = fh.read()
    if not path.endswith((".hpp", ".hip", ".h")):
        return text
    src = text.decode()
    out, i, n = [], 0, len(src)
    while i < n:
        c = src[i]
        if c == '"' or c == "'":                      # literals are code
            j = i + 1
            while j < n and src[j] != c:
                j += 2 if src[j] == "\\" else 1
            out.append(src[i:j + 1])
            i = j + 1
        elif src.startswith("//", i):
            i = src.find("\n", i)
            i = n if i < 0 else i
        elif src.startswith("/*", i):
            i = src.find("*/", i + 2)
            i = n if i < 0 else i + 2
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split()).encode()


def sources_digest(kernel: str) -> str:
    """sha256 over the code of the sources `kernel` (a demangled name) is
    built from, in name order; counters taken on other code do not describe
    it."""
    root = os.path.dirname(os.path.abspath(__file__))
    names = list(_COMMON)
    if kernel.startswith(("k_rollout", "k_regen_mlp")):
        names += _POLICY
    h = hashlib.sha256()
    for rel in sorted(names):
        path = os.path.normpath(os.path.join(root, rel))
        h.update(os.path.basename(path).encode())
        h.update(_code_text(path))
    return h.hexdigest()


def _recorded(summary_path: str, tag: str, kernel: str) -> float | None:
    if not os.path.exists(summary_path):
        return None
    want = sources_digest(kernel)
    with open(summary_path) as fh:
        for line in fh:
            parts = line.split(maxsplit=3)
            if len(parts) == 4 and parts[0] == tag and parts[3].strip() == kernel:
                return float(parts[1]) if parts[2] == want else None
    return None


def recorded_traffic(summary_path: str, kernel: str) -> float | None:
    """Bytes per launch recorded for `kernel` in a --traffic summary, or None
    when the file is absent or was taken on other kernel sources."""
    return _recorded(summary_path, TRAFFIC_TAG, kernel)


def recorded_valu(summary_path: str, kernel: str) -> float | None:
    """VALU instructions per launch recorded for `kernel` by --valu, or None
    when the file is absent or was taken on other kernel sources."""
    return _recorded(summary_path, VALU_TAG, kernel)


def _table(rows, top: int) -> list[str]:
    """rows: (name, duration_ns) in any order -> per-kernel statistics lines."""
    per: dict[str, list[int]] = {}
    for name, dur in rows:
        per.setdefault(name, []).append(dur)
    stats = sorted(((n, len(d), sum(d), min(d), max(d)) for n, d in per.items()),
                   key=lambda r: -r[2])
    total = sum(r[2] for r in stats) or 1
    out = [f"{'kernel':70s} {'calls':>6s} {'total_us':>11s} {'avg_us':>9s} "
           f"{'min_us':>9s} {'max_us':>9s} {'pct':>6s}"]
    for name, calls, tot, mn, mx in stats[:top]:
        out.append(f"{name[:70]:70s} {calls:6d} {tot / 1e3:11.3f} {tot / calls / 1e3:9.3f} "
                   f"{mn / 1e3:9.3f} {mx / 1e3:9.3f} {100.0 * tot / total:6.2f}")
    return out


def split_per_archive(rows):
    """Dispatches (name, start, end) in start order, cut into one run per
    archive: each archive's set-up begins with k_clear_archive; what comes
    before the first one forms a run of its own."""
    runs, cur = [], []
    for name, start, end in sorted(rows, key=lambda r: r[1]):
        if "k_clear_archive" in name and cur:
            runs.append(cur)
            cur = []
        cur.append((name, end - start))
    if cur:
        runs.append(cur)
    return runs


def summary(db_path: str, top: int = 20, per_archive: bool = False) -> str:
    con = _open(db_path)
    rows = con.execute("select name, start, end from kernels").fetchall()
    if not per_archive:
        return "\n".join(_table([(n, e - s) for n, s, e in rows], top))
    out = []
    for k, run in enumerate(split_per_archive(rows)):
        out.append(f"-- archive {k} (dispatches {len(run)})")
        out.extend(_table(run, top))
    return "\n".join(out)


def pmc_summary(db_path: str, top: int = 20) -> str:
    con = _open(db_path)
    rows = con.execute(
        "select name, counter_name, count(*), avg(counter_value), min(counter_value), "
        "max(counter_value) from pmc_events group by name, counter_name "
        "order by avg(counter_value) * count(*) desc").fetchall()
    out = [f"{'kernel':70s} {'counter':>14s} {'calls':>6s} {'mean':>14s} {'min':>14s} "
           f"{'max':>14s}"]
    for name, ctr, calls, mean, mn, mx in rows[:top]:
        out.append(f"{name[:70]:70s} {ctr:>14s} {calls:6d} {mean:14.2f} {mn:14.2f} {mx:14.2f}")
    return "\n".join(out)


def _counter_mean(db_path: str, counter: str, name_like: str) -> tuple[float, int]:
    con = _open(db_path)
    row = con.execute("select avg(counter_value), count(*) from pmc_events where counter_name = ? "
                      "and name like ?", (counter, name_like)).fetchone()
    if row is None or row[1] == 0:
        raise SystemExit(f"{db_path}: no {counter} rows for kernels like {name_like!r}")
    return float(row[0]), int(row[1])


def traffic(kernel: str, copy_fetch: str, copy_write: str, fetch: str, write: str,
            copy_mib: int) -> str:
    copy_bytes = copy_mib * 2.0**20
    cf, _ = _counter_mean(copy_fetch, "FETCH_SIZE", "%copyBuffer%")
    cw, _ = _counter_mean(copy_write, "WRITE_SIZE", "%copyBuffer%")
    f_scale, w_scale = copy_bytes / (cf * 1024.0), copy_bytes / (cw * 1024.0)
    kf, nf = _counter_mean(fetch, "FETCH_SIZE", f"%{kernel}%")
    kw, nw = _counter_mean(write, "WRITE_SIZE", f"%{kernel}%")
    rd, wr = kf * 1024.0 * f_scale, kw * 1024.0 * w_scale
    return "\n".join([
        f"copy of {copy_mib} MiB: FETCH_SIZE {cf:.1f} KiB -> scale {f_scale:.4f}; "
        f"WRITE_SIZE {cw:.1f} KiB -> scale {w_scale:.4f}",
        f"{kernel}: FETCH_SIZE {kf:.2f} KiB/dispatch ({nf} dispatches) -> {rd:.0f} B read; "
        f"WRITE_SIZE {kw:.2f} KiB/dispatch ({nw} dispatches) -> {wr:.0f} B written",
        f"{TRAFFIC_TAG} {rd + wr:.0f} {sources_digest(kernel)} {kernel}",
    ])


def valu(kernel: str, db_path: str) -> str:
    """SQ_INSTS_VALU of `kernel` summed over the counter instances of each
    dispatch (a wave64 instruction counts once), averaged over dispatches."""
    con = _open(db_path)
    rows = con.execute("select dispatch_id, sum(counter_value) from pmc_events where "
                       "counter_name = 'SQ_INSTS_VALU' and name like ? group by dispatch_id",
                       (f"%{kernel}%",)).fetchall()
    if not rows:
        raise SystemExit(f"{db_path}: no SQ_INSTS_VALU rows for kernels like {kernel!r}")
    per = [float(r[1]) for r in rows]
    mean = sum(per) / len(per)
    return "\n".join([
        f"{kernel}: SQ_INSTS_VALU per dispatch (all instances) {mean:.0f}, over {len(per)} "
        f"dispatches (min {min(per):.0f}, max {max(per):.0f})",
        f"{VALU_TAG} {mean:.0f} {sources_digest(kernel)} {kernel}",
    ])


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("db", nargs="+")
    ap.add_argument("--top", type=int, default=20)
    ap.add_argument("--pmc", action="store_true")
    ap.add_argument("--traffic", metavar="KERNEL")
    ap.add_argument("--valu", metavar="KERNEL")
    ap.add_argument("--copy-mib", type=int, default=256)
    ap.add_argument("--per-archive", action="store_true")
    a = ap.parse_args()
    if a.traffic:
        if len(a.db) != 4:
            raise SystemExit("--traffic takes copy_fetch.db copy_write.db fetch.db write.db")
        print(traffic(a.traffic, *a.db, a.copy_mib))
    elif a.valu:
        print(valu(a.valu, a.db[0]))
    else:
        print(pmc_summary(a.db[0], a.top) if a.pmc else summary(a.db[0], a.top, a.per_archive))


if __name__ == "__main__":
    main()
