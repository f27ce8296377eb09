"""Condense rocprofv3 CSV output of ``bench.py`` runs into the short text summaries kept under
``profiles/``, and the per-launch HBM traffic record ``bench.py`` reports.

    python -m paper_2509_23722_amd.rocprof_summary --trace DIR [--fetch DIR --write DIR \\
        --copy-fetch DIR --copy-write DIR --kernel NAME] [--sq DIR ...] --workload NAME \\
        [--tag TAG] [--what TEXT] --commands FILE --out-dir profiles

Each DIR is a rocprofv3 ``-d`` output directory holding ``*_kernel_stats.csv`` (kernel trace) or
``*_counter_collection.csv`` (``--pmc``). HBM bytes: FETCH_SIZE and WRITE_SIZE (KiB per
dispatch) of the kernel, each scaled by the ratio between the bytes a plain device copy of
known size moves and what the same counter reads for that copy (``bench.py
--copy-calibration``, 1 GiB read + 1 GiB written per launch).
"""
import argparse
import csv
import glob
import hashlib
import json
import os
from collections import defaultdict

HERE = os.path.dirname(os.path.abspath(__file__))
COPY_BYTES = 1 << 30


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("octo.hip", "octo_sim.hpp", "octo_device.hpp"):
        with open(os.path.join(HERE, "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def short(name):
    name = name.replace("octo::", "")
    return name.split("(")[0].replace("void ", "").strip()


def one(pattern):
    files = sorted(glob.glob(pattern))
    if not files:
        raise SystemExit(f"no file matches {pattern}")
    return files[0]


def kernel_stats(d):
    rows = list(csv.DictReader(open(one(os.path.join(d, "*kernel_stats.csv")))))
    return [(short(r["Name"]), int(r["Calls"]), float(r["AverageNs"]), float(r["MinNs"]),
             float(r["MaxNs"]), float(r["Percentage"])) for r in rows]


def counters(d):
    """{kernel: {counter: mean value per dispatch}} and dispatch counts."""
    rows = list(csv.DictReader(open(one(os.path.join(d, "*counter_collection.csv")))))
    acc = defaultdict(lambda: defaultdict(list))
    for r in rows:
        acc[short(r["Kernel_Name"])][r["Counter_Name"]].append(float(r["Counter_Value"]))
    return {k: {c: (sum(v) / len(v), len(v)) for c, v in cs.items()} for k, cs in acc.items()}


def copy_factor(d, counter):
    c = counters(d)
    vals = [cs[counter][0] for k, cs in c.items() if "copyBuffer" in k or "elementwise" in k]
    kib = max(vals)
    return COPY_BYTES / (kib * 1024.0), kib


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", required=True)
    for k in ("fetch", "write", "copy-fetch", "copy-write"):
        ap.add_argument("--" + k)
    ap.add_argument("--sq", action="append", default=[])
    ap.add_argument("--kernel", help="short name of the dominant kernel")
    ap.add_argument("--workload", required=True)
    ap.add_argument("--tag", help="file name tag (default: the workload)")
    ap.add_argument("--what", default="one `bench.py --headline-only` run: every simulation "
                    "kernel dispatch is a headline-call one (the first call of a run also builds "
                    "the cached MERGE and static-schedule tables)")
    ap.add_argument("--commands", required=True, help="text file with the commands that ran")
    ap.add_argument("--out-dir", default="profiles")
    args = ap.parse_args()
    cmds = open(args.commands).read().strip()
    tag = args.tag or args.workload

    stats = kernel_stats(args.trace)
    lines = [f"# Kernel trace: simulation kernels, {args.workload}", "",
             f"rocprofv3 kernel-trace statistics of {args.what}.", "", "Commands:", "", "```",
             cmds, "```", "",
             "| kernel | calls | average us | min us | max us | % of GPU time |",
             "|---|---:|---:|---:|---:|---:|"]
    for name, calls, avg, mn, mx, pct in stats:
        lines.append(f"| {name} | {calls} | {avg / 1e3:.1f} | {mn / 1e3:.1f} | {mx / 1e3:.1f} "
                     f"| {pct:.2f} |")
    with open(os.path.join(args.out_dir, f"kernel_trace_{tag}.md"), "w") as f:
        f.write("\n".join(lines) + "\n")

    if args.sq:
        lines = [f"# SQ counters per dispatch, {args.workload}", "", "Commands:", "", "```",
                 cmds, "```", ""]
        for d in args.sq:
            c = counters(d)
            names = sorted({n for cs in c.values() for n in cs})
            lines += ["| kernel | " + " | ".join(names) + " |",
                      "|---|" + "---:|" * len(names)]
            for k, cs in c.items():
                if "copyBuffer" in k:
                    continue
                lines.append(f"| {k} | " + " | ".join(
                    f"{cs[n][0]:.4g}" if n in cs else "" for n in names) + " |")
            lines.append("")
        with open(os.path.join(args.out_dir, f"sq_counters_{tag}.md"), "w") as f:
            f.write("\n".join(lines) + "\n")
    if args.fetch and args.write and args.copy_fetch and args.copy_write and args.kernel:
        traffic_summary(args, cmds, tag)


def traffic_summary(args, cmds, tag):
    ff, fkib_copy = copy_factor(args.copy_fetch, "FETCH_SIZE")
    wf, wkib_copy = copy_factor(args.copy_write, "WRITE_SIZE")
    fetch, write = counters(args.fetch), counters(args.write)
    lines = [f"# HBM traffic per dispatch, {args.workload}", "",
             "FETCH_SIZE and WRITE_SIZE (KiB per dispatch, mean over the run's dispatches), "
             "each in a rocprofv3 `--pmc` run of its own, scaled by the copy calibration: a "
             f"plain 1 GiB device copy reads {fkib_copy:.0f} KiB by FETCH_SIZE (factor "
             f"{ff:.4f}) and writes {wkib_copy:.0f} KiB by WRITE_SIZE (factor {wf:.4f}).", "",
             "Commands:", "", "```", cmds, "```", "",
             "| kernel | dispatches | FETCH KiB | WRITE KiB | HBM MB (scaled) |",
             "|---|---:|---:|---:|---:|"]
    rec = None
    for k in fetch:
        if "copyBuffer" in k:
            continue
        fk, n = fetch[k].get("FETCH_SIZE", (0.0, 0))
        wk = write.get(k, {}).get("WRITE_SIZE", (0.0, 0))[0]
        mb = (fk * 1024 * ff + wk * 1024 * wf) / 1e6
        lines.append(f"| {k} | {n} | {fk:.1f} | {wk:.1f} | {mb:.2f} |")
        if k == args.kernel:
            rec = {"kernel": k, "kernel_source_sha": kernel_source_hash(),
                   "hbm_bytes_per_launch": int(fk * 1024 * ff + wk * 1024 * wf),
                   "fetch_kib": fk, "write_kib": wk, "fetch_factor": ff, "write_factor": wf,
                   "workload": args.workload}
    with open(os.path.join(args.out_dir, f"hbm_traffic_{tag}.md"), "w") as f:
        f.write("\n".join(lines) + "\n")
    if rec is None:
        raise SystemExit(f"kernel {args.kernel} not in the counter runs")
    with open(os.path.join(args.out_dir, f"traffic_{tag}.json"), "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")

if __name__ == "__main__":
    main()
