"""Short text summaries of rocprofv3 CSV output (kernel statistics and HBM
byte counters), as kept beside the library's measurements.

    python -m paper_2412_00119_amd.profsum stats  <rocprof dir> [--command CMD]
    python -m paper_2412_00119_amd.profsum traffic --fetch <dir> --write <dir>
        --kernel REGEX --source FILE --calib-bytes N [--command CMD]
    python -m paper_2412_00119_amd.profsum counters <dir> [<dir> ...] --kernel REGEX
        [--command CMD ...]

`stats` turns `*_kernel_stats.csv` into a table of kernels (calls, average,
min, max, share of GPU time).  `traffic` reads the per-dispatch FETCH_SIZE and
WRITE_SIZE counters (KiB per dispatch, from two separate `--pmc` runs), finds
the calibration copy (the largest `copyBuffer` dispatch, a plain
device-to-device copy of N bytes each way), derives the factor that maps each
counter onto the copy's known bytes, and reports the scaled bytes per launch
of the kernels matching REGEX with the SHA-256 of their source file and device
compile flags, so that a reader can tell whether the figure still describes the
current kernel.
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import os
import re
import sys


def _one(pattern: str) -> str:
    hits = sorted(glob.glob(pattern, recursive=True))
    if not hits:
        sys.exit(f"no file matches {pattern}")
    return hits[0]


def short_name(name: str) -> str:
    name = re.sub(r"\(anonymous namespace\)::", "", name)
    m = re.match(r"(?:void )?([\w:<>, ]+?)\(", name)
    return (m.group(1) if m else name).strip()


def stats(args) -> None:
    path = _one(os.path.join(args.dir, "**", "*kernel_stats.csv"))
    rows = list(csv.DictReader(open(path)))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    print("# rocprofv3 kernel statistics\n")
    if args.command:
        print(f"Command:\n\n    {args.command}\n")
    print("| kernel | calls | avg us | min us | max us | total ms | % GPU time |")
    print("|---|---:|---:|---:|---:|---:|---:|")
    for r in rows:
        print(f"| {short_name(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
              f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
              f"{float(r['TotalDurationNs']) / 1e6:.3f} | {float(r['Percentage']):.2f} |")


def _per_dispatch(dirname: str, counter: str):
    path = _one(os.path.join(dirname, "**", "*counter_collection.csv"))
    vals = collections.defaultdict(float)
    names = {}
    for r in csv.DictReader(open(path)):
        if r["Counter_Name"] != counter:
            continue
        d = int(r["Dispatch_Id"])
        vals[d] += float(r["Counter_Value"])
        names[d] = r["Kernel_Name"]
    return [(d, names[d], vals[d]) for d in sorted(vals)]


def traffic(args) -> None:
    out = {}
    for counter, dirname in (("FETCH_SIZE", args.fetch), ("WRITE_SIZE", args.write)):
        rows = _per_dispatch(dirname, counter)
        copies = [v for _, n, v in rows if "copyBuffer" in n]
        if not copies:
            sys.exit(f"{counter}: no calibration copy dispatch in {dirname}")
        calib_kib = max(copies)
        factor = args.calib_bytes / (calib_kib * 1024.0)
        ker = [v for _, n, v in rows if re.search(args.kernel, n)]
        if not ker:
            sys.exit(f"{counter}: no dispatch of {args.kernel} in {dirname}")
        out[counter] = (factor, calib_kib, sum(ker) / len(ker), len(ker))
    from paper_2412_00119_amd.build import kernel_fingerprint
    sha = kernel_fingerprint(args.source)
    fetch_f, fetch_c, fetch_kib, n_f = out["FETCH_SIZE"]
    write_f, write_c, write_kib, n_w = out["WRITE_SIZE"]
    fetch_b = fetch_kib * 1024.0 * fetch_f
    write_b = write_kib * 1024.0 * write_f
    print(f"# HBM traffic of `{args.kernel}`\n")
    if args.command:
        print("Commands (one `--pmc` counter per run):\n")
        for c in args.command:
            print(f"    {c}")
        print()
    print("| counter | calibration copy (KiB read by the counter) | factor | kernel KiB per dispatch "
          "(mean) | dispatches | bytes per launch |")
    print("|---|---:|---:|---:|---:|---:|")
    print(f"| FETCH_SIZE | {fetch_c:.0f} | {fetch_f:.3f} | {fetch_kib:.1f} | {n_f} | {fetch_b:.4g} |")
    print(f"| WRITE_SIZE | {write_c:.0f} | {write_f:.3f} | {write_kib:.1f} | {n_w} | {write_b:.4g} |")
    print(f"\ncalibration copy: {args.calib_bytes} bytes read and {args.calib_bytes} bytes written\n")
    print(f"kernel_source: {os.path.relpath(args.source)}")
    print(f"kernel_build_sha256: {sha}")
    print(f"fetch_bytes_per_launch: {fetch_b:.6g}")
    print(f"write_bytes_per_launch: {write_b:.6g}")
    print(f"traffic_bytes_per_launch: {fetch_b + write_b:.6g}")


def counters(args) -> None:
    """Mean value per dispatch of every counter in the given --pmc runs, per
    kernel matching REGEX, with the ratios that read them."""
    table = collections.defaultdict(lambda: collections.defaultdict(list))
    dur = collections.defaultdict(list)
    for d in args.dirs:
        path = _one(os.path.join(d, "**", "*counter_collection.csv"))
        per = collections.defaultdict(float)
        meta = {}
        for r in csv.DictReader(open(path)):
            if not re.search(args.kernel, r["Kernel_Name"]):
                continue
            key = (int(r["Dispatch_Id"]), r["Counter_Name"])
            per[key] += float(r["Counter_Value"])
            meta[int(r["Dispatch_Id"])] = (short_name(r["Kernel_Name"]),
                                           int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
        for (disp, cname), v in per.items():
            table[meta[disp][0]][cname].append(v)
        for disp, (kname, ns) in meta.items():
            dur[kname].append(ns)
    print("# rocprofv3 counters per dispatch\n")
    if args.command:
        print("Commands (one `--pmc` pass per run):\n")
        for c in args.command:
            print(f"    {c}")
        print()
    for kname in sorted(table):
        cs = table[kname]
        print(f"## {kname}\n")
        print("| counter | dispatches | mean per dispatch |")
        print("|---|---:|---:|")
        mean = {}
        for cname in sorted(cs):
            vals = cs[cname]
            mean[cname] = sum(vals) / len(vals)
            print(f"| {cname} | {len(vals)} | {mean[cname]:.6g} |")
        print()
        derived = []
        simds = 256 * 4
        dur_cycles = (sum(dur[kname]) / len(dur[kname])) * 2.4 if dur[kname] else 0.0   # ns x 2.4 GHz
        mfma = mean.get("SQ_INSTS_MFMA", 0.0)
        if "SQ_INSTS_VALU" in mean:
            valu = mean["SQ_INSTS_VALU"] - mfma   # SQ_INSTS_VALU counts the MFMAs too
            derived.append(("VALU instructions (MFMA excluded) per SIMD", valu / simds))
            if dur_cycles:
                derived.append(("VALU issue cycles (4 per wave64 instruction) / dispatch cycles at 2.4 GHz",
                                4 * valu / simds / dur_cycles))
            if mfma:
                derived.append(("VALU instructions per MFMA", valu / mfma))
        if "SQ_VALU_MFMA_BUSY_CYCLES" in mean and mfma:
            derived.append(("MFMA busy cycles per MFMA", mean["SQ_VALU_MFMA_BUSY_CYCLES"] / mfma))
            if dur_cycles:
                derived.append(("MFMA busy cycles per SIMD / dispatch cycles at 2.4 GHz",
                                mean["SQ_VALU_MFMA_BUSY_CYCLES"] / simds / dur_cycles))
        if "SQ_INSTS_LDS" in mean and mfma:
            derived.append(("LDS instructions per MFMA", mean["SQ_INSTS_LDS"] / mfma))
        if "SQ_WAIT_INST_LDS" in mean and "SQ_WAVE_CYCLES" in mean and mean["SQ_WAVE_CYCLES"]:
            derived.append(("waves waiting on LDS / wave cycles",
                            mean["SQ_WAIT_INST_LDS"] / mean["SQ_WAVE_CYCLES"]))
        if "SQ_WAIT_ANY" in mean and "SQ_WAVE_CYCLES" in mean and mean["SQ_WAVE_CYCLES"]:
            derived.append(("waves waiting on anything / wave cycles", mean["SQ_WAIT_ANY"] / mean["SQ_WAVE_CYCLES"]))
        if "SQ_ACTIVE_INST_VALU" in mean and "SQ_WAVE_CYCLES" in mean and mean["SQ_WAVE_CYCLES"]:
            derived.append(("waves issuing VALU / wave cycles", mean["SQ_ACTIVE_INST_VALU"] / mean["SQ_WAVE_CYCLES"]))
        if "SQ_LDS_BANK_CONFLICT" in mean and "SQ_INSTS_LDS" in mean and mean["SQ_INSTS_LDS"]:
            derived.append(("LDS bank-conflict cycles per LDS instruction",
                            mean["SQ_LDS_BANK_CONFLICT"] / mean["SQ_INSTS_LDS"]))
        if derived:
            print("| ratio | value |")
            print("|---|---:|")
            for name, v in derived:
                print(f"| {name} | {v:.4g} |")
            print()
        if dur[kname]:
            print(f"mean dispatch duration under the counters: {sum(dur[kname]) / len(dur[kname]) / 1e3:.2f} us "
                  f"(counter collection serialises dispatches; the ratios over dispatch cycles use it)\n")


def main(argv=None) -> None:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("--command", default="")
    t = sub.add_parser("traffic")
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--kernel", required=True)
    t.add_argument("--source", required=True)
    t.add_argument("--calib-bytes", type=float, required=True)
    t.add_argument("--command", action="append", default=[])
    c = sub.add_parser("counters")
    c.add_argument("dirs", nargs="+")
    c.add_argument("--kernel", required=True)
    c.add_argument("--command", action="append", default=[])
    args = ap.parse_args(argv)
    {"stats": stats, "traffic": traffic, "counters": counters}[args.cmd](args)


if __name__ == "__main__":
    main()
