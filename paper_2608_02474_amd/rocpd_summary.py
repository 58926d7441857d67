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
    python -m paper_2608_02474_amd.rocpd_summary mfma PATTERN RUN.db [RUN.db ...]
        per (kernel, grid size) matching PATTERN: shader clock, MFMA-busy
        fraction, MFMA work issued, vector instructions per MFMA, wait and LDS
        bank-conflict fractions from counter runs (each with --kernel-trace
        for the durations), then every raw counter average

Grouping by grid size separates dispatches of one kernel at different
problem sizes (for example the all-token first step from the cached steps).
`--skip-first N` (any mode) leaves out the first N dispatches of every
(kernel, grid size), in dispatch order: a launch of the cached block's
all-token first step that has the grid of a cached step's launch (the
attention's 256 key ranges) then does not enter the cached step's figures.
"""
from __future__ import annotations

import hashlib
import json
import re
import sqlite3
import sys

COPY_BYTES = 1 << 30  # what the hbm_copy module reads and writes by default
SKIP = 0  # dispatches left out at the start of every (kernel, grid size)


def _order_column(c, view: str) -> str:
    """A column of `view` that orders dispatches in time."""
    cols = [d[0] for d in c.execute(f"select * from {view} limit 0").description]
    for name in ("start", "dispatch_id", "id"):
        if name in cols:
            return name
    raise SystemExit(f"no ordering column (start, dispatch_id, id) in {view}: {cols}")


def _kernels(c) -> str:
    """The kernels view, less the first SKIP dispatches of every (kernel, grid)."""
    if SKIP <= 0:
        return "kernels"
    o = _order_column(c, "kernels")
    return (f"(select * from (select *, row_number() over (partition by name, grid_x, grid_y, grid_z "
            f"order by {o}) as skip_rn from kernels) where skip_rn > {SKIP})")


def _counters(c) -> str:
    """The counters view, less the first SKIP dispatches of every (kernel, grid, counter)."""
    if SKIP <= 0:
        return "counters_collection"
    o = _order_column(c, "counters_collection")
    return (f"(select * from (select *, row_number() over (partition by kernel_name, grid_size, counter_name "
            f"order by {o}) as skip_rn from counters_collection) where skip_rn > {SKIP})")


def short_name(n: str) -> str:
    n = re.sub(r"\(.*", "", n)
    return n.replace("void ", "").strip()


def trace_rows(db: str):
    c = sqlite3.connect(db)
    q = ("select name, grid_x * grid_y * grid_z, count(*), avg(duration), min(duration), "
         f"max(duration), sum(duration) from {_kernels(c)} group by name, grid_x, grid_y, grid_z "
         "order by sum(duration) desc")
    return [(short_name(r[0]), r[1], r[2], r[3] / 1e3, r[4] / 1e3, r[5] / 1e3, r[6] / 1e3)
            for r in c.execute(q)]


def counter_rows(db: str, counter: str):
    c = sqlite3.connect(db)
    q = (f"select kernel_name, grid_size, count(*), avg(value) from {_counters(c)} "
         "where counter_name = ? group by kernel_name, grid_size order by avg(value) desc")
    return [(short_name(r[0]), r[1], r[2], r[3]) for r in c.execute(q, (counter,))]


def counter_of(db: str, counter: str, substring: str, grid: int) -> float:
    c = sqlite3.connect(db)
    q = (f"select avg(value) from {_counters(c)} where counter_name = ? and "
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


def dispatch_durations(db: str):
    """{(kernel, grid threads): average duration in ns} from the kernel trace
    of a run (empty if the run recorded none)."""
    c = sqlite3.connect(db)
    try:
        q = (f"select name, grid_x * grid_y * grid_z, avg(duration) from {_kernels(c)} "
             "group by name, grid_x, grid_y, grid_z")
        return {(short_name(r[0]), r[1]): r[2] for r in c.execute(q)}
    except sqlite3.Error:
        return {}


def counter_table(dbs, pattern: str = ""):
    """Average value per dispatch of every counter in the given runs, per
    (kernel, grid threads) whose name contains `pattern`, with the average
    dispatch duration: {(kernel, grid): {"calls": n, "dur_ns": t, COUNTER: v}}."""
    out = {}
    for db in dbs:
        dur = dispatch_durations(db)
        c = sqlite3.connect(db)
        q = (f"select kernel_name, grid_size, counter_name, count(*), avg(value) from {_counters(c)} "
             "where kernel_name like ? group by kernel_name, grid_size, counter_name")
        for name, grid, counter, n, v in c.execute(q, (f"%{pattern}%",)):
            key = (short_name(name), grid)
            rec = out.setdefault(key, {"calls": n})
            rec[counter] = float(v)
            if key in dur:
                rec.setdefault("dur_ns", dur[key])
    return out


def mfma_summary(dbs, pattern: str = "", simds: int = 1024, xcds: int = 8):
    """Per-dispatch MFMA evidence of the kernels matching `pattern`.
    GRBM_GUI_ACTIVE is summed over the 8 XCDs (each counts its own busy
    cycles), SQ_VALU_MFMA_BUSY_CYCLES over the 1024 SIMDs:
      sclk        GRBM_GUI_ACTIVE / 8 / duration (GHz), the shader clock while it ran
      mfma_busy   SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 x 1024 SIMDs):
                  the fraction of the SIMDs' cycles their MFMA pipe was busy
      peak_frac   mfma_busy x sclk / 2.4 GHz: the same against the nominal clock
      bf16_tflop  SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 (the MFMA work issued)
      valu/mfma   SQ_INSTS_VALU / SQ_INSTS_MFMA (vector instructions per MFMA)
      coexec      SQ_VALU_MFMA_COEXEC_CYCLES / SQ_VALU_MFMA_BUSY_CYCLES
      wait        SQ_WAIT_ANY / SQ_WAVE_CYCLES and SQ_WAIT_INST_ANY / SQ_WAVE_CYCLES
      lds_bank    SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE"""
    rows = []
    for (name, grid), r in sorted(counter_table(dbs, pattern).items(), key=lambda kv: -kv[1].get("dur_ns", 0)):
        g = r.get("GRBM_GUI_ACTIVE")
        d = r.get("dur_ns")
        busy = r.get("SQ_VALU_MFMA_BUSY_CYCLES")
        ratio = lambda a, b: (r[a] / r[b]) if r.get(a) is not None and r.get(b) else None
        sclk = g / xcds / d if g and d else None
        mb = busy / (g / xcds * simds) if busy is not None and g else None
        rows.append({"kernel": name, "grid": grid, "calls": r["calls"], "dur_us": d / 1e3 if d else None,
                     "sclk_ghz": sclk, "mfma_busy": mb,
                     "peak_frac": mb * sclk / 2.4 if mb is not None and sclk else None,
                     "bf16_tflop": r["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512 / 1e12
                     if r.get("SQ_INSTS_VALU_MFMA_MOPS_BF16") is not None else None,
                     "valu_per_mfma": ratio("SQ_INSTS_VALU", "SQ_INSTS_MFMA"),
                     "coexec": ratio("SQ_VALU_MFMA_COEXEC_CYCLES", "SQ_VALU_MFMA_BUSY_CYCLES"),
                     "wait_any": ratio("SQ_WAIT_ANY", "SQ_WAVE_CYCLES"),
                     "wait_inst": ratio("SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES"),
                     "lds_bank": ratio("SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE"),
                     "raw": {k: v for k, v in r.items() if k not in ("calls", "dur_ns")}})
    return rows


def main(argv):
    global SKIP
    if "--skip-first" in argv:
        i = argv.index("--skip-first")
        SKIP = int(argv[i + 1])
        argv = argv[:i] + argv[i + 2:]
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
    if len(argv) >= 3 and argv[0] == "mfma":
        pattern, dbs = argv[1], argv[2:]
        cols = ("dur_us", "sclk_ghz", "mfma_busy", "peak_frac", "bf16_tflop", "valu_per_mfma", "coexec",
                "wait_any", "wait_inst", "lds_bank")
        print(f"{'kernel':44s} {'grid':>9s} " + " ".join(f"{c:>13s}" for c in cols))
        rows = mfma_summary(dbs, pattern)
        for r in rows:
            vals = " ".join(f"{r[c]:13.4f}" if r[c] is not None else f"{'-':>13s}" for c in cols)
            print(f"{r['kernel'][:44]:44s} {r['grid']:9d} {vals}")
        print("\nraw counters per dispatch (averages):")
        for r in rows:
            print(f"{r['kernel'][:44]:44s} {r['grid']:9d} " +
                  " ".join(f"{k}={v:.6g}" for k, v in sorted(r["raw"].items())))
        return 0
    if len(argv) >= 6 and argv[0] == "traffic":
        print(json.dumps(traffic(*argv[1:5], argv[5:]), indent=1))
        return 0
    print(__doc__)
    return 2


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
