#!/usr/bin/env python3
"""Summarise a rocprofv3 kernel trace (rocpd SQLite output of `rocprofv3 --kernel-trace`).

Dispatches are grouped by kernel and launch shape (grid, workgroup, dynamic LDS), so that the
same kernel template launched for different passes (prefill, verify, draft) is listed apart.

usage: python3 paper_2609_36590_amd/profile_summary.py <run_results.db> [--min-calls N] [name-substring ...]
"""
import sqlite3
import sys


def main():
    args = sys.argv[1:]
    min_calls = 1
    if "--min-calls" in args:
        i = args.index("--min-calls")
        min_calls = int(args[i + 1])
        del args[i:i + 2]
    db = sqlite3.connect(args[0])
    filt = args[1:]
    rows = db.execute(
        "select name, grid_x, grid_y, grid_z, workgroup_x, lds_size, vgpr_count, accum_vgpr_count, sgpr_count, "
        "count(*), sum(duration), avg(duration), min(duration), max(duration) from kernels "
        "group by name, grid_x, grid_y, grid_z, workgroup_x, lds_size order by sum(duration) desc").fetchall()
    total = sum(r[10] for r in rows)
    print(f"{'kernel':44s} {'grid(threads)':>20s} {'wg':>5s} {'lds':>6s} {'vgpr/agpr/sgpr':>14s} "
          f"{'calls':>7s} {'total_ms':>9s} {'avg_us':>8s} {'min_us':>8s} {'max_us':>8s} {'pct':>6s}")
    for (name, gx, gy, gz, wg, lds, vg, ag, sg, n, tot, avg, mn, mx) in rows:
        if n < min_calls or (filt and not any(f in name for f in filt)):
            continue
        short = name.replace("seedk::", "").replace("unsigned short", "bf16").replace("(LinArgs)", "")
        short = short.replace("(AttnArgs)", "").replace("void ", "").split("(")[0]
        print(f"{short[:44]:44s} {f'{gx}x{gy}x{gz}':>20s} {wg:5d} {lds:6d} {f'{vg}/{ag}/{sg}':>14s} "
              f"{n:7d} {tot / 1e6:9.2f} {avg / 1e3:8.2f} {mn / 1e3:8.2f} {mx / 1e3:8.2f} {100 * tot / total:6.2f}")


if __name__ == "__main__":
    main()
