"""Summaries of rocprofv3 result databases (SQLite, ROCm 7).

  python -m paper_2608_12703_amd.profsum kernels RESULTS.db [--calls N] [--command CMD]
      per-kernel dispatch count, mean / min / max duration and share of GPU time
      (--calls: divide the totals by this many verify steps)
  python -m paper_2608_12703_amd.profsum step RESULTS.db --marker NAME [--which I]
      the kernels of one step: from the I-th dispatch whose name contains NAME to the
      next one (negative I counts from the end)
  python -m paper_2608_12703_amd.profsum traffic --fetch FETCH.db --write WRITE.db
          --kernel NAME --calib-mib MIB --out OUT.json [--command CMD]
      HBM bytes per dispatch of one kernel from a FETCH_SIZE run and a WRITE_SIZE run,
      each scaled by what the same counter reads for a plain copy of MIB MiB captured in
      the same run (the largest copyBuffer dispatch)
  python -m paper_2608_12703_amd.profsum counters RESULTS.db [RESULTS.db ...]
          [--kernel SUBSTR ...] [--command CMD]
      per kernel, the mean per dispatch of every counter collected (several --pmc runs may
      be given); with SQ_INSTS_VALU_MFMA_MOPS_BF16 also the bf16 matrix rate (512 flop per
      count over the dispatch's duration) against the dense bf16 peak
"""
from __future__ import annotations

import argparse
import json
import sqlite3
import sys

from .roofline import kernel_source_hash


def kernel_table(db: str, calls: int | None = None) -> str:
    cur = sqlite3.connect(db).cursor()
    rows = cur.execute("select name, count(*), avg(end - start), min(end - start), max(end - start), "
                       "sum(end - start) from kernels group by name order by sum(end - start) desc").fetchall()
    total = sum(r[5] for r in rows) or 1
    out = [f"{'kernel':70s} {'calls':>7s} {'mean us':>9s} {'min us':>9s} {'max us':>9s} {'share':>6s}"
           + (f" {'us/step':>9s}" if calls else "")]
    for name, n, avg, mn, mx, tot in rows:
        line = f"{name[:70]:70s} {n:7d} {avg / 1e3:9.2f} {mn / 1e3:9.2f} {mx / 1e3:9.2f} {100 * tot / total:5.1f}%"
        if calls:
            line += f" {tot / 1e3 / calls:9.1f}"
        out.append(line)
    return "\n".join(out)


def step_table(db: str, marker: str, which: int) -> str:
    """Kernels of one step: the dispatches from the `which`-th dispatch whose name contains
    `marker` (negative counts from the end) up to the next one, summed per kernel name
    in order of first appearance."""
    cur = sqlite3.connect(db).cursor()
    rows = cur.execute("select name, start, end from kernels order by start").fetchall()
    idx = [i for i, r in enumerate(rows) if marker in r[0]]
    i0 = idx[which]
    nxt = [i for i in idx if i > i0]
    i1 = nxt[0] if nxt else len(rows)
    agg = {}
    for name, st, en in rows[i0:i1]:
        e = agg.setdefault(name, [0.0, 0])
        e[0] += (en - st) / 1e3
        e[1] += 1
    total = sum(v[0] for v in agg.values())
    out = [f"{'kernel':70s} {'calls':>6s} {'us':>9s} {'share':>6s}"]
    for name, (us, n) in agg.items():
        out.append(f"{name[:70]:70s} {n:6d} {us:9.1f} {100 * us / total:5.1f}%")
    out.append(f"{'sum of kernel durations':70s} {'':6s} {total:9.1f}")
    return "\n".join(out)


def _counter(db: str, kernel: str):
    cur = sqlite3.connect(db).cursor()
    vals = [r[0] for r in cur.execute("select value from counters_collection where kernel_name like ?",
                                      (f"%{kernel}%",))]
    copies = [r[0] for r in cur.execute("select value from counters_collection where kernel_name like "
                                        "'%copyBuffer%'")]
    if not vals or not copies:
        raise SystemExit(f"{db}: no dispatches of {kernel!r} or of the calibration copy")
    return sum(vals) / len(vals), len(vals), max(copies)


def traffic(fetch_db: str, write_db: str, kernel: str, calib_mib: int, command: str) -> dict:
    f_kib, f_n, f_copy = _counter(fetch_db, kernel)
    w_kib, w_n, w_copy = _counter(write_db, kernel)
    known_kib = calib_mib * 1024.0
    f_scale, w_scale = known_kib / f_copy, known_kib / w_copy
    return {"kernel": kernel, "source_sha256": kernel_source_hash(),
            "fetch_kib_per_dispatch": round(f_kib, 1), "write_kib_per_dispatch": round(w_kib, 1),
            "dispatches": [f_n, w_n],
            "calibration": {"copy_mib": calib_mib, "fetch_kib": f_copy, "write_kib": w_copy,
                            "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4)},
            "hbm_bytes_per_launch": int(round((f_kib * f_scale + w_kib * w_scale) * 1024)),
            "command": command}


N_XCD, N_SIMD = 8, 1024


def counter_table(dbs, kernels=None) -> str:
    """Mean value per dispatch of each counter, per kernel name (matching `kernels`)."""
    from .roofline import BF16_MFMA_PEAK
    per = {}      # kernel -> counter -> [sum, n]
    dur = {}      # kernel -> [sum ns, n] (dispatch durations of the counter runs)
    for db in dbs:
        cur = sqlite3.connect(db).cursor()
        rows = cur.execute("select kernel_name, counter_name, value, dispatch_id, duration "
                           "from counters_collection").fetchall()
        seen = set()
        for name, cname, val, disp, du in rows:
            if kernels and not any(k in name for k in kernels):
                continue
            e = per.setdefault(name, {}).setdefault(cname, [0.0, 0])
            e[0] += float(val)
            e[1] += 1
            if (db, disp) not in seen and du:
                seen.add((db, disp))
                d = dur.setdefault(name, [0.0, 0])
                d[0] += float(du)
                d[1] += 1
    out = []
    for name in sorted(per, key=lambda n: -dur.get(n, [0, 1])[0]):
        cs = per[name]
        d = dur.get(name)
        mean_ns = d[0] / d[1] if d and d[1] else 0.0
        out.append(f"{name[:100]}")
        if mean_ns:
            out.append(f"    mean duration under the counters {mean_ns / 1e3:.2f} us ({d[1]} dispatches)")
        for cname in sorted(cs):
            tot, n = cs[cname]
            out.append(f"    {cname:36s} {tot / n:16.1f}")
        if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in cs and mean_ns:
            tot, n = cs["SQ_INSTS_VALU_MFMA_MOPS_BF16"]
            flops = tot / n * 512
            rate = flops / (mean_ns * 1e-9)
            out.append(f"    bf16 matrix work {flops / 1e9:.2f} GFLOP per dispatch -> {rate / 1e12:.1f} TFLOP/s "
                       f"= {100 * rate / BF16_MFMA_PEAK:.1f}% of the dense bf16 peak")
        if "SQ_VALU_MFMA_BUSY_CYCLES" in cs and "GRBM_GUI_ACTIVE" in cs and mean_ns:
            # GRBM_GUI_ACTIVE sums the 8 XCDs over the counter window (the dispatch plus a
            # few microseconds around it: a lower bound on the busy fraction of a short
            # kernel); the busy cycles sum the 1024 SIMDs (256 CUs x 4)
            busy = cs["SQ_VALU_MFMA_BUSY_CYCLES"][0] / cs["SQ_VALU_MFMA_BUSY_CYCLES"][1]
            xcd_cycles = cs["GRBM_GUI_ACTIVE"][0] / cs["GRBM_GUI_ACTIVE"][1] / N_XCD
            out.append(f"    matrix pipes busy {100 * busy / (xcd_cycles * N_SIMD):.1f}% of the SIMD cycles of "
                       f"the counter window ({xcd_cycles:.0f} cycles per XCD)")
        if "SQ_WAIT_INST_ANY" in cs and "SQ_WAVE_CYCLES" in cs:
            wait = cs["SQ_WAIT_INST_ANY"][0] / max(cs["SQ_WAVE_CYCLES"][0], 1.0)
            out.append(f"    waves waiting on a dependency {100 * wait:.1f}% of their cycles")
    return "\n".join(out)


def main(argv=None):
    p = argparse.ArgumentParser(prog="profsum")
    sub = p.add_subparsers(dest="cmd", required=True)
    k = sub.add_parser("kernels")
    k.add_argument("db")
    k.add_argument("--calls", type=int)
    k.add_argument("--command", default="")
    st = sub.add_parser("step")
    st.add_argument("db")
    st.add_argument("--marker", required=True)
    st.add_argument("--which", type=int, default=-2)
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--kernel", required=True)
    t.add_argument("--calib-mib", type=int, required=True)
    t.add_argument("--out", required=True)
    t.add_argument("--command", default="")
    c = sub.add_parser("counters")
    c.add_argument("dbs", nargs="+")
    c.add_argument("--kernel", action="append")
    c.add_argument("--command", default="")
    a = p.parse_args(argv)
    if a.cmd == "counters":
        if a.command:
            print(f"command: {a.command}\n")
        print(counter_table(a.dbs, a.kernel))
        return
    if a.cmd == "kernels":
        if a.command:
            print(f"command: {a.command}\n")
        print(kernel_table(a.db, a.calls))
    elif a.cmd == "step":
        print(step_table(a.db, a.marker, a.which))
    else:
        rec = traffic(a.fetch, a.write, a.kernel, a.calib_mib, a.command)
        with open(a.out, "w") as fh:
            json.dump(rec, fh, indent=1)
        json.dump(rec, sys.stdout, indent=1)
        print()


if __name__ == "__main__":
    main()
