"""Summaries of rocprofv3 result databases (the SQLite files rocprofv3 writes
with its default output format).

    python -m paper_2608_02474_amd.rocpd_summary trace  RESULTS.db
        per (kernel, grid size): dispatches, average / min / max microseconds
    python -m paper_2608_02474_amd.rocpd_summary counter RESULTS.db COUNTER
        per (kernel, grid size): dispatches and the average counter value

Grouping by grid size separates dispatches of one kernel at different
problem sizes (for example the all-token first step from the cached steps).
"""
from __future__ import annotations

import re
import sqlite3
import sys


def short_name(n: str) -> str:
    n = re.sub(r"\(.*", "", n)
    return n.replace("void ", "").strip()


def trace_rows(db: str):
    c = sqlite3.connect(db)
    q = ("select name, grid_x * grid_y * grid_z, count(*), avg(duration), min(duration), "
         "max(duration), sum(duration) from kernels group by name, grid_x, grid_y, grid_z "
         "order by sum(duration) desc")
    return [(short_name(r[0]), r[1], r[2], r[3] / 1e3, r[4] / 1e3, r[5] / 1e3, r[6] / 1e3)
            for r in c.execute(q)]


def counter_rows(db: str, counter: str):
    c = sqlite3.connect(db)
    q = ("select kernel_name, grid_size, count(*), avg(value) from counters_collection "
         "where counter_name = ? group by kernel_name, grid_size order by avg(value) desc")
    return [(short_name(r[0]), r[1], r[2], r[3]) for r in c.execute(q, (counter,))]


def main(argv):
    if len(argv) >= 2 and argv[0] == "trace":
        print(f"{'kernel':58s} {'grid threads':>12s} {'calls':>5s} {'avg us':>10s} "
              f"{'min us':>10s} {'max us':>10s} {'total us':>11s}")
        for n, g, k, avg, mn, mx, tot in trace_rows(argv[1]):
            print(f"{n[:58]:58s} {g:12d} {k:5d} {avg:10.1f} {mn:10.1f} {mx:10.1f} {tot:11.1f}")
        return 0
    if len(argv) >= 3 and argv[0] == "counter":
        print(f"{'kernel':58s} {'grid threads':>12s} {'calls':>5s} {argv[2] + ' (KiB)':>16s}")
        for n, g, k, v in counter_rows(argv[1], argv[2]):
            print(f"{n[:58]:58s} {g:12d} {k:5d} {v:16.1f}")
        return 0
    print(__doc__)
    return 2


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
