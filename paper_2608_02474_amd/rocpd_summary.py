"""Summaries of rocprofv3 result databases (the SQLite files rocprofv3 writes
with its default output format).

    python -m paper_2608_02474_amd.rocpd_summary trace  RESULTS.db
        per (kernel, grid size): dispatches, average / min / max microseconds
    python -m paper_2608_02474_amd.rocpd_summary counter RESULTS.db COUNTER
        per (kernel, grid size): dispatches and the average counter value
    python -m paper_2608_02474_amd.rocpd_summary traffic FETCH.db WRITE.db \
            COPY_FETCH.db COPY_WRITE.db KEY=KERNEL_SUBSTRING@GRID[+KERNEL_SUBSTRING@GRID...]@SOURCE ...
        HBM bytes per call of each named (kernel, grid) or sum of them (a call
        made of several launches), calibrated with the
        counters of a copy of known size (the hbm_copy module: 1 GiB read and
        1 GiB written), as JSON records keyed KEY carrying the sha256 of SOURCE
        (the kernel's source file, so that a stale record can be recognised)

Grouping by grid size separates dispatches of one kernel at different
problem sizes (for example the all-token first step from the cached steps).
"""
from __future__ import annotations

import hashlib
import json
import re
import sqlite3
import sys

COPY_BYTES = 1 << 30  # what the hbm_copy module reads and writes by default


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


def counter_of(db: str, counter: str, substring: str, grid: int) -> float:
    c = sqlite3.connect(db)
    q = ("select avg(value) from counters_collection where counter_name = ? and "
         "kernel_name like ? and grid_size = ?")
    v = c.execute(q, (counter, f"%{substring}%", grid)).fetchone()[0]
    if v is None:
        raise SystemExit(f"no {counter} dispatch of *{substring}* with grid {grid} in {db}")
    return float(v)


def copy_counter(db: str, counter: str) -> float:
    """Counter of the largest single dispatch in the calibration run (the copy)."""
    c = sqlite3.connect(db)
    q = "select max(value) from counters_collection where counter_name = ?"
    return float(c.execute(q, (counter,)).fetchone()[0])


def traffic(fetch_db, write_db, copy_fetch_db, copy_write_db, specs):
    ff = COPY_BYTES / 1024.0 / copy_counter(copy_fetch_db, "FETCH_SIZE")
    wf = COPY_BYTES / 1024.0 / copy_counter(copy_write_db, "WRITE_SIZE")
    out = {}
    for spec in specs:
        key, rest = spec.split("=", 1)
        parts, source = rest.rsplit("@", 1)
        f = w = 0.0
        grids = []
        for part in parts.split("+"):
            sub, grid = part.rsplit("@", 1)
            f += counter_of(fetch_db, "FETCH_SIZE", sub, int(grid))
            w += counter_of(write_db, "WRITE_SIZE", sub, int(grid))
            grids.append(int(grid))
        out[key] = {"fetch_kib": round(f, 1), "write_kib": round(w, 1),
                    "fetch_factor": round(ff, 4), "write_factor": round(wf, 4),
                    "bytes_per_launch": int(round((f * ff + w * wf) * 1024)),
                    "grid_threads": grids[0] if len(grids) == 1 else grids,
                    "source_sha256": hashlib.sha256(open(source, "rb").read()).hexdigest()}
    return out


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
    if len(argv) >= 6 and argv[0] == "traffic":
        print(json.dumps(traffic(*argv[1:5], argv[5:]), indent=1))
        return 0
    print(__doc__)
    return 2


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
