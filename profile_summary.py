"""Markdown summaries of rocprofv3 runs of bench.py, for profiles/.

Three modes (each prints one summary with the command it summarises):

  traffic  HBM traffic per kernel: four ``rocprofv3 --pmc ... --output-format csv``
           folders, FETCH_SIZE and WRITE_SIZE of ``copy_calib.py`` (1 GiB read and 1 GiB
           written per dispatch) and of the bench command; optionally a
           ``--kernel-trace --stats`` folder of the same command for durations. Per kernel:
           dispatches, calibrated bytes read and written, achieved HBM GB/s and fraction
           of 8 TB/s. The lines
               traffic_bytes_per_launch attend_full <bytes>
               source_sha256 <file> <hash>
           are what bench.py reads back (it trusts the figure only while the hashed
           sources are unchanged): the V^T pre-pass, fast path and fixup of one
           full-cache attention.
  trace    kernel time per kernel from a ``--kernel-trace --stats`` folder.
  mfma     ``--pmc MfmaUtil MfmaFlopsBF16 --kernel-trace`` folder: MFMA busy share and
           executed bf16 MFMA work per kernel.

    python profile_summary.py traffic --copy-fetch D1 --copy-write D2 --fetch D3 --write D4 \\
        [--trace D5] --workload NAME --command "..." > profiles/hbm_traffic__NAME.md
    python profile_summary.py trace --trace D --workload NAME --command "..."
    python profile_summary.py mfma --counters D --workload NAME --command "..."
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import os
import re
import sys
from collections import defaultdict

ROOT = os.path.dirname(os.path.abspath(__file__))
SOURCES = ["paper_2609_39329_amd/csrc/attention_kernels.hpp",
           "paper_2609_39329_amd/csrc/attention.hip", "paper_2609_39329_amd/csrc/stats.hip",
           "paper_2609_39329_amd/csrc/solve.hip"]
PEAK_GBS = 8000.0
LIB_KERNEL = re.compile(r"pkv::|^_ZN3pkv")
COPY_KERNEL = re.compile(r"copy|elementwise", re.I)
COPY_BYTES = float(1 << 30)


def demangle_args(m: str) -> str:
    """Template arguments of a mangled name the profiler left undemangled (bf16 types):
    'Li128ELb1E' -> '128, true', 'DF16b' -> '__bf16', 'f' -> 'float'."""
    out, i = [], 0
    while i < len(m) and m[i] != "E":
        if m.startswith("Lb0E", i) or m.startswith("Lb1E", i):
            out.append("true" if m[i + 2] == "1" else "false")
            i += 4
        elif m[i] == "L":
            j = m.index("E", i)
            out.append(m[i + 2:j].replace("n", "-"))
            i = j + 1
        elif m.startswith("DF16b", i):
            out.append("__bf16")
            i += 5
        else:
            out.append({"f": "float", "d": "double", "i": "int"}.get(m[i], m[i]))
            i += 1
    return ", ".join(out)


def short(name: str) -> str:
    """'void pkv::(anonymous namespace)::foo<1, true>(pkv::P)' -> 'foo<1, true>'."""
    mm = re.match(r"_ZN3pkv12_GLOBAL__N_1(\d+)", name)
    if mm:  # _ZN3pkv12_GLOBAL__N_1 <len> <name> [I <args> E] E ...
        k = mm.end()
        base = name[k:k + int(mm.group(1))]
        rest = name[k + int(mm.group(1)):]
        return base + (f"<{demangle_args(rest[1:])}>" if rest.startswith("I") else "")
    n = name[5:] if name.startswith("void ") else name
    depth, cut = 0, len(n)
    for i, ch in enumerate(n):  # drop the parameter list (the first '(' outside '<>')
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0 and not n.startswith("(anonymous", i):
            cut = i
            break
    n = n[:cut]
    return re.sub(r"(pkv::)?\(anonymous namespace\)::|pkv::", "", n)


def read_counter(folder: str, counter: str):
    """{kernel name: [value per dispatch]} (counter in KiB, summed over XCDs)."""
    files = glob.glob(os.path.join(folder, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        sys.exit(f"no counter_collection.csv under {folder}")
    per = defaultdict(dict)
    for f in files:
        with open(f, newline="") as fh:
            for row in csv.DictReader(fh):
                if row["Counter_Name"] != counter:
                    continue
                key = (f, row["Dispatch_Id"])
                per[row["Kernel_Name"]][key] = per[row["Kernel_Name"]].get(key, 0.0) + float(
                    row["Counter_Value"])
    return {k: list(v.values()) for k, v in per.items()}


def read_durations(folder: str):
    """{kernel name: (calls, average ns)} from a --stats kernel_stats.csv."""
    files = glob.glob(os.path.join(folder, "**", "*kernel_stats.csv"), recursive=True)
    out = {}
    for f in files:
        with open(f, newline="") as fh:
            for row in csv.DictReader(fh):
                out[row["Name"]] = (int(row["Calls"]), float(row["AverageNs"]))
    return out


def calibration(folder: str, counter: str) -> float:
    vals = [v for k, vs in read_counter(folder, counter).items() if COPY_KERNEL.search(k)
            for v in vs]
    if not vals:
        sys.exit(f"no copy dispatch in {folder}")
    reading = max(vals)  # the 1 GiB copy is the largest dispatch of the calibration run
    return COPY_BYTES / (reading * 1024.0), reading


def mean(v):
    return sum(v) / len(v)


def hashes() -> None:
    for s in SOURCES:
        with open(os.path.join(ROOT, s), "rb") as fh:
            print(f"    source_sha256 {s} {hashlib.sha256(fh.read()).hexdigest()}")


def trace_mode(a) -> None:
    files = glob.glob(os.path.join(a.trace, "**", "*kernel_stats.csv"), recursive=True)
    if not files:
        sys.exit(f"no kernel_stats.csv under {a.trace}")
    rows = [r for f in files for r in csv.DictReader(open(f, newline=""))]
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    print(f"# Kernel trace: {a.workload}\n")
    print("Command (run on the MI355X box from /tmp with TMPDIR=/tmp):\n")
    print(f"    rocprofv3 --kernel-trace --stats --output-format csv -d <trace> -o p -- {a.command}")
    print(f"    python profile_summary.py trace --trace <trace> --workload {a.workload} --command '...'\n")
    print("Sources:\n")
    hashes()
    print("\n| kernel | calls | total us | avg us | % |\n|---|---|---|---|---|")
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        t = float(r["TotalDurationNs"])
        if t < 1e-4 * total:
            continue
        print(f"| `{short(r['Name'])}` | {int(r['Calls'])} | {t / 1e3:,.0f} | "
              f"{float(r['AverageNs']) / 1e3:,.2f} | {100 * t / total:.2f} |")


def mfma_mode(a) -> None:
    util = read_counter(a.counters, "MfmaUtil")
    flops = read_counter(a.counters, "MfmaFlopsBF16")
    files = glob.glob(os.path.join(a.counters, "**", "*counter_collection.csv"), recursive=True)
    dur = defaultdict(list)
    for f in files:
        seen = set()
        for row in csv.DictReader(open(f, newline="")):
            key = (row["Kernel_Name"], row["Dispatch_Id"])
            if key in seen:
                continue
            seen.add(key)
            dur[row["Kernel_Name"]].append(int(row["End_Timestamp"]) - int(row["Start_Timestamp"]))
    print(f"# MFMA utilisation per kernel: {a.workload}\n")
    print("Command (run on the MI355X box from /tmp with TMPDIR=/tmp):\n")
    print(f"    rocprofv3 --pmc MfmaUtil MfmaFlopsBF16 --kernel-trace --output-format csv -d <counters> -o p -- {a.command}")
    print(f"    python profile_summary.py mfma --counters <counters> --workload {a.workload} --command '...'\n")
    print("`MfmaUtil`: share of SIMD cycles with the MFMA pipe busy (duration-weighted mean over "
          "dispatches). `MfmaFlopsBF16`: bf16 MFMA work the hardware executed (the split-bf16 fp32 "
          "products execute several bf16 products per algorithmic one; fp32 MFMA is not counted). "
          "Durations are those of the counter run (dispatches serialised by the profiler).\n")
    print("Sources:\n")
    hashes()
    print("\n| kernel | dispatches | MfmaUtil % | bf16 MFMA FLOP / dispatch | duration us | "
          "executed bf16 TFLOP/s |\n|---|---|---|---|---|---|")
    ks = [k for k in util if LIB_KERNEL.search(k) and k in flops and mean(flops[k]) > 0]
    for k in sorted(ks, key=lambda k: -mean(dur[k]) * len(dur[k])):
        d = dur[k]
        w = sum(u * t for u, t in zip(util[k], d)) / max(sum(d), 1)
        fl = mean(flops[k])
        print(f"| `{short(k)}` | {len(d)} | {w:.1f} | {fl:.4g} | {mean(d) / 1e3:,.1f} | "
              f"{fl / (mean(d) * 1e-9) / 1e12:,.0f} |")


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("mode", choices=("traffic", "trace", "mfma"))
    for x in ("copy-fetch", "copy-write", "fetch", "write", "counters"):
        ap.add_argument(f"--{x}")
    ap.add_argument("--trace")
    ap.add_argument("--workload", required=True)
    ap.add_argument("--command", required=True, help="the bench command that was profiled")
    ap.add_argument("--teacher-psplit", action="store_true",
                    help="the workload's full-cache pass forms P V from a two-term P")
    a = ap.parse_args()
    if a.mode == "trace":
        return trace_mode(a)
    if a.mode == "mfma":
        return mfma_mode(a)
    if not (a.copy_fetch and a.copy_write and a.fetch and a.write):
        sys.exit("traffic needs --copy-fetch, --copy-write, --fetch and --write")

    sf, rf = calibration(a.copy_fetch, "FETCH_SIZE")
    sw, rw = calibration(a.copy_write, "WRITE_SIZE")
    fetch = read_counter(a.fetch, "FETCH_SIZE")
    write = read_counter(a.write, "WRITE_SIZE")
    dur = read_durations(a.trace) if a.trace else {}

    print(f"# HBM traffic per kernel: {a.workload}\n")
    print("Counters FETCH_SIZE and WRITE_SIZE (KiB per dispatch, summed over the XCDs), each from "
          "a run of its own, scaled by what the same counter reads for a plain 1 GiB copy.\n")
    print("## Sources these counters belong to\n")
    hashes()
    print("\n## Commands\n")
    print("Run on the MI355X box from /tmp with TMPDIR=/tmp; one counter per pass:\n")
    print("    rocprofv3 --pmc FETCH_SIZE --output-format csv -d <copy-fetch> -o p -- "
          "python -u /root/repo/copy_calib.py")
    print("    rocprofv3 --pmc WRITE_SIZE --output-format csv -d <copy-write> -o p -- "
          "python -u /root/repo/copy_calib.py")
    print(f"    rocprofv3 --pmc FETCH_SIZE --output-format csv -d <fetch> -o p -- {a.command}")
    print(f"    rocprofv3 --pmc WRITE_SIZE --output-format csv -d <write> -o p -- {a.command}")
    if a.trace:
        print(f"    rocprofv3 --kernel-trace --stats --output-format csv -d <trace> -o p -- {a.command}")
    print("    python profile_summary.py traffic --copy-fetch <copy-fetch> --copy-write <copy-write> "
          "--fetch <fetch> --write <write>" + (" --trace <trace>" if a.trace else "")
          + f" --workload {a.workload} --command '...'")
    print("\n## Calibration (plain copy, 1,073,741,824 bytes read and written)\n")
    print("| counter | reading per dispatch | scale (bytes / KiB read) |\n|---|---|---|")
    print(f"| FETCH_SIZE | {rf:,.0f} KiB | {sf * 1024:.1f} |")
    print(f"| WRITE_SIZE | {rw:,.0f} KiB | {sw * 1024:.1f} |")

    print("\n## Library kernels\n")
    hdr = "| kernel | dispatches | read MB / dispatch | written MB / dispatch |"
    sep = "|---|---|---|---|"
    if dur:
        hdr += " avg µs | HBM GB/s | % of 8 TB/s |"
        sep += "---|---|---|"
    print(hdr + "\n" + sep)
    totals = {}
    for k in sorted(set(fetch) | set(write), key=lambda k: -mean(fetch.get(k, [0.0]))):
        if not LIB_KERNEL.search(k):
            continue
        fb = mean(fetch[k]) * 1024.0 * sf if k in fetch else 0.0
        wb = mean(write[k]) * 1024.0 * sw if k in write else 0.0
        totals[short(k)] = fb + wb
        line = f"| `{short(k)}` | {len(fetch.get(k, write.get(k, [])))} | {fb / 1e6:,.1f} | {wb / 1e6:,.1f} |"
        if dur:
            if k in dur:
                us = dur[k][1] / 1e3
                gbs = (fb + wb) / (dur[k][1] * 1e-9) / 1e9
                line += f" {us:,.1f} | {gbs:,.0f} | {100 * gbs / PEAK_GBS:.1f} |"
            else:
                line += " – | – | – |"
        print(line)

    # the full-cache pass: the teacher's fast path and its fixup (one dispatch each per
    # layer or reference chunk: no other call uses these instantiations; a chunk's pass
    # carries its own entries; the teacher reads its contiguous cache's V as stored, so no
    # V^T pre-pass belongs to it), with split key ranges the merge (its largest dispatch),
    # and for fp32 inputs the fp32 kernel over the cache
    ps = "true" if a.teacher_psplit else "false"
    pats = [r"attn_combine_kernel<\d+, (true|false)>",
            rf"attn_bf16_kernel<\d+, false, {ps}, (false|true), (false|true), (false|true), false, 0, "
            r"(false|true)>",
            r"attn_f32_kernel<\d+, false, (false|true), false, false>"]
    def largest(k):
        f = max(fetch.get(k, [0.0])) * 1024.0 * sf
        w = max(write.get(k, [0.0])) * 1024.0 * sw
        return f + w
    full = [k for k in set(fetch) | set(write)
            if LIB_KERNEL.search(k) and any(re.fullmatch(pt, short(k)) for pt in pats)]
    if full:
        print("\n## One full-cache attention launch (fast path, fixup and, where present, the merge)\n")
        for k in sorted(full, key=short):
            print(f"- `{short(k)}`: {largest(k) / 1e6:,.1f} MB")
        print(f"\n    traffic_bytes_per_launch attend_full {sum(largest(k) for k in full):.0f}")

if __name__ == "__main__":
    main()
