"""Summarise rocprofv3 CSV output (kernel-trace stats and --pmc counters).

    python -m paper_1906_11367_amd.profsum --stats DIR [--pmc NAME=DIR ...]
        [--copy-fetch DIR --copy-write DIR] [--kernel SUBSTR] [--json OUT]
        [--warmup W --steps S [--settle T]]

--stats   a rocprofv3 --kernel-trace --stats --output-format csv directory
--warmup, --steps, --settle
          the traced bench.py run made W warmup steps, then two passes of
          `settle` untimed steps (bench.py: 60) followed by S timed steps:
          each kernel's average is taken over the dispatches of the timed
          steps only (from the per-dispatch trace), as bench.py times them.
--pmc     counter directories (one rocprofv3 --pmc pass each)
--copy-*  passes over a plain elementwise kernel that reads and writes a known
          number of bytes: FETCH_SIZE / WRITE_SIZE of the kernels above are
          scaled by (known bytes / counted bytes) of that kernel.
--derived utilisation per kernel from SQ counters (MI355X: 8 XCDs, 1024
          SIMDs; GRBM_GUI_ACTIVE sums the XCDs' active cycles):
            cycles     = GRBM_GUI_ACTIVE / 8
            VALU busy  = 4 * SQ_ACTIVE_INST_VALU / (1024 * cycles)
                         (a wave64 VALU instruction occupies its SIMD 4 cycles)
            MFMA busy  = SQ_VALU_MFMA_BUSY_CYCLES / (1024 * cycles)
            wait share = SQ_WAIT_ANY / SQ_WAVE_CYCLES (wave cycles spent waiting)
            LDS conflict = SQ_LDS_BANK_CONFLICT / SQ_ACTIVE_INST_LDS
Prints a Markdown table per kernel (average duration, calls, counters per
dispatch); --json writes the HBM bytes per launch of the kernels whose name
contains --kernel.
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import json
import os

COPY_BYTES = 256 << 20      # the calibration kernel reads and writes 256 MiB
XCDS, SIMDS = 8, 1024       # MI355X: 8 XCDs, 256 CUs x 4 SIMDs


def _csv(dir_, suffix):
    files = glob.glob(os.path.join(dir_, "**", f"*{suffix}"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no *{suffix} under {dir_}")
    with open(files[0]) as f:
        return list(csv.DictReader(f))


def short(name):
    return name.replace("void ", "").split("(")[0]


def counters(dir_):
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in _csv(dir_, "counter_collection.csv"):
        agg[short(r["Kernel_Name"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
    return {k: {c: sum(v) / len(v) for c, v in d.items()} for k, d in agg.items()}


def stats(dir_, warmup=0, steps=0, settle=0):
    if not steps:
        out = {}
        for r in _csv(dir_, "kernel_stats.csv"):
            out[short(r["Name"])] = {"calls": int(r["Calls"]), "avg_us": float(r["AverageNs"]) / 1e3,
                                     "total_us": float(r["TotalDurationNs"]) / 1e3,
                                     "pct": float(r["Percentage"])}
        return out
    per = collections.defaultdict(list)
    for r in _csv(dir_, "kernel_trace.csv"):
        per[short(r["Kernel_Name"])].append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    total_steps = warmup + 2 * (settle + steps)
    out = {}
    for k, d in per.items():
        d.sort()
        launches = len(d) // total_steps
        if launches == 0 or len(d) % total_steps:     # not launched once per step: keep every dispatch
            kept = d
        else:
            a1 = (warmup + settle) * launches
            a2 = (warmup + 2 * settle + steps) * launches
            kept = d[a1:a1 + steps * launches] + d[a2:a2 + steps * launches]
        durs = [(e - s) / 1e3 for s, e in kept]
        out[k] = {"calls": len(durs), "avg_us": sum(durs) / len(durs), "total_us": sum(durs)}
    tot = sum(v["total_us"] for v in out.values())
    for v in out.values():
        v["pct"] = 100.0 * v["total_us"] / tot
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--stats")
    ap.add_argument("--pmc", nargs="*", default=[])
    ap.add_argument("--copy-fetch")
    ap.add_argument("--copy-write")
    ap.add_argument("--kernel")
    ap.add_argument("--json")
    ap.add_argument("--source-hash")
    ap.add_argument("--warmup", type=int, default=0)
    ap.add_argument("--steps", type=int, default=0)
    ap.add_argument("--settle", type=int, default=60)
    ap.add_argument("--derived", action="store_true")
    a = ap.parse_args()
    fetch_f = write_f = None
    if a.copy_fetch:
        c = counters(a.copy_fetch)
        k = [v for n, v in c.items() if "elementwise" in n and v.get("FETCH_SIZE", 0) > 0]
        fetch_f = COPY_BYTES / (max(v["FETCH_SIZE"] for v in k) * 1024.0)
    if a.copy_write:
        c = counters(a.copy_write)
        k = [v for n, v in c.items() if "elementwise" in n and v.get("WRITE_SIZE", 0) > 0]
        write_f = COPY_BYTES / (max(v["WRITE_SIZE"] for v in k) * 1024.0)
    merged = collections.defaultdict(dict)
    for spec in a.pmc:
        name, d = spec.split("=", 1)
        for k, v in counters(d).items():
            merged[k].update(v)
    st = stats(a.stats, a.warmup, a.steps, a.settle) if a.stats else {}
    names = sorted(set(st) | set(merged), key=lambda n: -st.get(n, {}).get("total_us", 0))
    if fetch_f:
        print(f"calibration: FETCH_SIZE x {fetch_f:.4f}, WRITE_SIZE x {write_f:.4f} "
              f"(plain elementwise kernel, {COPY_BYTES >> 20} MiB read + written)\n")
    print("| kernel | calls | avg us | % | counters per dispatch |")
    print("|---|---|---|---|---|")
    result = {}
    for n in names:
        s = st.get(n, {})
        c = merged.get(n, {})
        extra = ", ".join(f"{k}={v:.4g}" for k, v in sorted(c.items()))
        if fetch_f and "FETCH_SIZE" in c and "WRITE_SIZE" in c:
            rd = c["FETCH_SIZE"] * 1024 * fetch_f
            wr = c["WRITE_SIZE"] * 1024 * write_f
            extra += f"; HBM read {rd / 1e6:.1f} MB, write {wr / 1e6:.1f} MB"
            if a.kernel and a.kernel in n:
                result[n] = rd + wr
        print(f"| {n[:70]} | {s.get('calls', '')} | {s.get('avg_us', 0):.2f} | {s.get('pct', 0):.1f} | {extra} |")
    if a.derived:
        print()
        print("| kernel | VALU instr / wave | VALU busy | MFMA busy | LDS instr / wave | LDS conflict | wait share |")
        print("|---|---|---|---|---|---|---|")
        for n in names:
            c = merged.get(n, {})
            if not c.get("SQ_WAVES") or not c.get("GRBM_GUI_ACTIVE") or n.startswith("at::"):
                continue
            cyc = c["GRBM_GUI_ACTIVE"] / XCDS
            w = c["SQ_WAVES"]
            valu = 4 * c.get("SQ_ACTIVE_INST_VALU", 0) / (SIMDS * cyc)
            mfma = c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) / (SIMDS * cyc)
            lds_c = c.get("SQ_LDS_BANK_CONFLICT", 0) / max(c.get("SQ_ACTIVE_INST_LDS", 0), 1)
            wait = c.get("SQ_WAIT_ANY", 0) / max(c.get("SQ_WAVE_CYCLES", 0), 1)
            print(f"| {n[:70]} | {c.get('SQ_INSTS_VALU', 0) / w:.0f} | {100 * valu:.1f} % | {100 * mfma:.1f} % | "
                  f"{c.get('SQ_INSTS_LDS', 0) / w:.0f} | {lds_c:.2f} | {100 * wait:.1f} % |")
    if a.json and result:
        with open(a.json, "w") as f:
            json.dump({"source_hash": a.source_hash, "kernels": {k: v for k, v in result.items()},
                       "hbm_bytes_per_launch": sum(result.values()),
                       "fetch_factor": fetch_f, "write_factor": write_f}, f, indent=1)


if __name__ == "__main__":
    main()
