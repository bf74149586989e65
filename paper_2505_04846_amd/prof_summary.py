"""Turns rocprofv3 output into the committed profile summaries.

    python -m paper_2505_04846_amd.prof_summary stats  DIR  OUT.md  --title T --command C
    python -m paper_2505_04846_amd.prof_summary traffic FETCH_DIR WRITE_DIR --kernel NAME
        --match SUBSTRING --workload W --sources a.hip,b.h --command C [--json profiles/traffic.json]
    python -m paper_2505_04846_amd.prof_summary counters DIR [DIR ...] --out OUT.md
        --match SUBSTRING --title T --command C [--command C ...]

`stats` renders run_kernel_stats.csv of a `rocprofv3 --kernel-trace --stats` run as a markdown
table.  `traffic` reads two `rocprofv3 --pmc` runs (FETCH_SIZE, then WRITE_SIZE; KiB per
dispatch) of a program that first copied 256 MiB device to device (bench.py
--copy-calibration): the copy's readings give the scale of each counter (known bytes / reading),
and the scaled per-dispatch HBM bytes of the kernels whose name contains SUBSTRING are recorded
in traffic.json under (kernel, workload, source hash) -- bench.py reports them only while the
kernel sources are unchanged.  `counters` renders `rocprofv3 --pmc` runs of MFMA, clock, LDS and
L2 counters as raw means and derived figures (clock, MFMA busy fraction, executed FLOP/s).
"""

import argparse
import csv
import glob
import hashlib
import json
import os
import statistics

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
COPY_BYTES = 256 << 20


def _csv(d, name):
    hits = glob.glob(os.path.join(d, "**", name), recursive=True)
    if not hits:
        raise SystemExit(f"no {name} under {d}")
    with open(hits[0]) as f:
        return list(csv.DictReader(f))


def source_sha(names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2505_04846_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stats(args):
    rows = _csv(args.dir, "run_kernel_stats.csv")
    lines = [f"# {args.title}", "", "Command:", "", "```", args.command, "```", "",
             "| kernel | calls | avg (us) | min (us) | max (us) | share |",
             "|---|---:|---:|---:|---:|---:|"]
    for r in rows:
        name = r["Name"].replace("(anonymous namespace)::", "").replace("|", "/")
        if len(name) > 90:
            name = name[:87] + "..."
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['Percentage']):.1f}% |")
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")


def _per_dispatch(rows, counter, match):
    """(calibration reading, mean reading of the matching kernel, its dispatch count).  The
    calibration copies are the first three copy dispatches of the program (bench.py issues
    them before anything else)."""
    rows = sorted((r for r in rows if r["Counter_Name"] == counter),
                  key=lambda r: int(r["Dispatch_Id"]))
    copy = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]][:3]
    kern = [float(r["Counter_Value"]) for r in rows if match in r["Kernel_Name"]]
    if len(copy) < 3 or not kern:
        raise SystemExit(f"{counter}: calibration copies {len(copy)}, matching dispatches {len(kern)}")
    return statistics.median(copy), statistics.mean(kern), len(kern)


def traffic(args):
    fc, fk, n1 = _per_dispatch(_csv(args.fetch_dir, "run_counter_collection.csv"), "FETCH_SIZE",
                               args.match)
    wc, wk, n2 = _per_dispatch(_csv(args.write_dir, "run_counter_collection.csv"), "WRITE_SIZE",
                               args.match)
    f_scale = COPY_BYTES / (fc * 1024.0)
    w_scale = COPY_BYTES / (wc * 1024.0)
    rec = {
        "kernel": args.kernel, "workload": args.workload,
        "source_sha": source_sha(args.sources.split(",")),
        "hbm_bytes_per_launch": fk * 1024.0 * f_scale + wk * 1024.0 * w_scale,
        "read_bytes_per_launch": fk * 1024.0 * f_scale,
        "write_bytes_per_launch": wk * 1024.0 * w_scale,
        "fetch_scale": f_scale, "write_scale": w_scale, "dispatches": [n1, n2],
        "command": args.command,
    }
    recs = []
    if os.path.exists(args.json):
        with open(args.json) as f:
            recs = [r for r in json.load(f)
                    if not (r["kernel"] == rec["kernel"] and r["workload"] == rec["workload"])]
    recs.append(rec)
    with open(args.json, "w") as f:
        json.dump(recs, f, indent=1)
    print(json.dumps(rec))


def _agent(d):
    """(XCD count, SIMD count, CU count) of the GPU agent of a rocprofv3 run."""
    for r in _csv(d, "*agent_info.csv"):
        if r.get("Agent_Type", "").upper().endswith("GPU") or r.get("Name", "").startswith("gfx"):
            return int(r["Num_Xcc"]), int(r["Simd_Count"]), int(r["Cu_Count"])
    raise SystemExit(f"no GPU agent in {d}")


def counters(args):
    """Derived MFMA / clock / LDS / L2 figures of the dispatches matching --match, from one or
    more `rocprofv3 --pmc` runs (each run's counters are averaged over its matching dispatches;
    every run must have collected GRBM_GUI_ACTIVE, which sums the busy cycles of all XCDs)."""
    merged, durs = {}, []
    n_xcc = n_simd = n_cu = None
    for d in args.dirs:
        n_xcc, n_simd, n_cu = _agent(d)
        rows = [r for r in _csv(d, "*counter_collection.csv") if args.match in r["Kernel_Name"]]
        if not rows:
            raise SystemExit(f"no dispatch of {args.match} in {d}")
        per = {}
        for r in rows:
            per.setdefault(r["Dispatch_Id"], {})[r["Counter_Name"]] = float(r["Counter_Value"])
            per[r["Dispatch_Id"]]["_ns"] = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        disp = list(per.values())
        for name in disp[0]:
            if not name.startswith("_"):
                merged.setdefault(name, []).append(statistics.mean(x[name] for x in disp))
        durs += [x["_ns"] * 1e-9 for x in disp]
    c = {k: statistics.mean(v) for k, v in merged.items()}
    dur = statistics.mean(durs)
    lines = [f"# {args.title}", "", "Commands (one `rocprofv3 --pmc` run each):", "", "```"]
    lines += args.command + ["```", "", f"Dispatches of `{args.match}`: mean duration "
                             f"{dur * 1e3:.3f} ms.", "", "| counter | mean per dispatch |",
                             "|---|---:|"]
    lines += [f"| `{k}` | {v:.6g} |" for k, v in sorted(c.items())]
    lines += ["", "Derived (per dispatch; XCDs and SIMDs from the run's agent record: "
              f"{n_xcc} and {n_simd}):", ""]
    cyc = c.get("GRBM_GUI_ACTIVE", 0.0) / n_xcc  # busy cycles of one XCD
    if cyc:
        ghz = cyc / dur / 1e9
        note = (" (above the 2.4 GHz peak: for a dispatch this short the counter also holds cycles "
                "outside it, so no clock is derived)" if ghz > 2.4 else "")
        lines.append(f"- clock: GRBM_GUI_ACTIVE / {n_xcc} / duration = {ghz:.3f} GHz{note}")
    if cyc and "SQ_VALU_MFMA_BUSY_CYCLES" in c:
        lines.append(f"- MFMA busy: SQ_VALU_MFMA_BUSY_CYCLES / (cycles x {n_simd} SIMDs) = "
                     f"{c['SQ_VALU_MFMA_BUSY_CYCLES'] / (cyc * n_simd):.3f}")
    mops = sum(c.get(k, 0.0) for k in ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_VALU_MFMA_MOPS_F16"))
    if mops:
        lines.append(f"- executed matrix FLOP/s: MOPS x 512 / duration = {mops * 512 / dur / 1e12:.1f} "
                     f"TFLOP/s ({mops * 512:.4g} FLOP per dispatch)")
    if c.get("SQ_INSTS_MFMA"):
        m = c["SQ_INSTS_MFMA"]
        if "SQ_INSTS_VALU" in c:
            lines.append(f"- other VALU instructions per MFMA: {(c['SQ_INSTS_VALU'] - m) / m:.2f}")
        if "SQ_INSTS_LDS" in c:
            lines.append(f"- LDS instructions per MFMA: {c['SQ_INSTS_LDS'] / m:.3f}")
    if c.get("SQ_WAVE_CYCLES"):
        w = c["SQ_WAVE_CYCLES"]
        if "SQ_WAIT_ANY" in c:
            lines.append(f"- waves waiting: SQ_WAIT_ANY / SQ_WAVE_CYCLES = {c['SQ_WAIT_ANY'] / w:.3f}")
        if "SQ_ACTIVE_INST_ANY" in c:
            lines.append(f"- waves issuing: SQ_ACTIVE_INST_ANY / SQ_WAVE_CYCLES = "
                         f"{c['SQ_ACTIVE_INST_ANY'] / w:.3f}")
    if "TA_TA_BUSY_sum" in c:
        # GRBM_GUI_ACTIVE over-counts short dispatches under the profiler, so the busy cycles
        # are also set against the dispatch's duration at the 2.4 GHz peak clock (a lower bound
        # on the busy fraction at any lower clock)
        per_cu = c["TA_TA_BUSY_sum"] / n_cu
        lines.append(f"- texture-address units: {per_cu:.4g} busy cycles per CU; over the "
                     f"dispatch's duration at 2.4 GHz: {per_cu / (dur * 2.4e9):.3f}")
    if "TCC_HIT_sum" in c and "TCC_MISS_sum" in c:
        h, mi = c["TCC_HIT_sum"], c["TCC_MISS_sum"]
        lines.append(f"- L2 hit rate: {h / (h + mi):.3f} ({mi:.4g} misses)")
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines[-8:]))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("dir")
    a.add_argument("out")
    a.add_argument("--title", required=True)
    a.add_argument("--command", required=True)
    b = sub.add_parser("traffic")
    b.add_argument("fetch_dir")
    b.add_argument("write_dir")
    b.add_argument("--kernel", required=True)
    b.add_argument("--match", required=True)
    b.add_argument("--workload", required=True)
    b.add_argument("--sources", required=True)
    b.add_argument("--command", required=True)
    b.add_argument("--json", default=os.path.join(ROOT, "profiles", "traffic.json"))
    c = sub.add_parser("counters")
    c.add_argument("dirs", nargs="+")
    c.add_argument("--out", required=True)
    c.add_argument("--match", required=True)
    c.add_argument("--title", required=True)
    c.add_argument("--command", action="append", required=True)
    args = ap.parse_args()
    {"stats": stats, "traffic": traffic, "counters": counters}[args.cmd](args)


if __name__ == "__main__":
    main()
