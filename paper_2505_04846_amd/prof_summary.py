"""Turns rocprofv3 output into the committed profile summaries.

    python -m paper_2505_04846_amd.prof_summary stats  DIR  OUT.md  --title T --command C
    python -m paper_2505_04846_amd.prof_summary traffic FETCH_DIR WRITE_DIR --kernel NAME
        --match SUBSTRING --workload W --sources a.hip,b.h --command C [--json profiles/traffic.json]

`stats` renders run_kernel_stats.csv of a `rocprofv3 --kernel-trace --stats` run as a markdown
table.  `traffic` reads two `rocprofv3 --pmc` runs (FETCH_SIZE, then WRITE_SIZE; KiB per
dispatch) of a program that first copied 256 MiB device to device (bench.py
--copy-calibration): the copy's readings give the scale of each counter (known bytes / reading),
and the scaled per-dispatch HBM bytes of the kernels whose name contains SUBSTRING are recorded
in traffic.json under (kernel, workload, source hash) -- bench.py reports them only while the
kernel sources are unchanged.
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
    args = ap.parse_args()
    (stats if args.cmd == "stats" else traffic)(args)


if __name__ == "__main__":
    main()
