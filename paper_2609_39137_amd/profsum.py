"""Summaries of rocprofv3 CSV output for the ``profiles/`` folder.

Two commands, both run on the CPU over files a profiled run wrote:

``stats``: a ``*_kernel_stats.csv`` of ``rocprofv3 --kernel-trace --stats``
becomes a short markdown table (calls, average/min/max duration, share).

``counters``: per-dispatch means of the fused router kernel's counters from
one ``--pmc`` pass (MFMA busy cycles, wait cycles, LDS bank conflicts).

``traffic``: the ``*_counter_collection.csv`` of a ``FETCH_SIZE`` pass and of
a ``WRITE_SIZE`` pass over ``bench.py --pmc-pass`` become the HBM bytes per
launch of the fused router kernel.  Both counters are read in KiB per
dispatch.  The pass also runs one device-to-device copy of known size; the
ratio of what each counter reports for that copy to its true size is the
calibration factor, and the router kernel's readings are divided by it.  The
result is written as JSON (read by ``bench.py`` as ``roofline.traffic``, and
only while the router sources still hash to the recorded value) plus a
markdown note.

    python -m paper_2609_39137_amd.profsum stats CSV --cmd "..." --out profiles/X.md
    python -m paper_2609_39137_amd.profsum traffic --fetch CSV --write CSV --copy-bytes N \\
        --workload NAME --variant V --cmd-fetch "..." --cmd-write "..." --out profiles/Y
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import statistics
import sys

_PKG = os.path.dirname(os.path.abspath(__file__))
# the fused router kernel's instantiations (16x16 and 32x32 MFMA tilings)
ROUTER_KERNELS = ("router16_kernel", "router32_kernel")


def _is_router(name: str) -> bool:
    return any(k in name for k in ROUTER_KERNELS)


def router_source_hash() -> str:
    """Hash of the sources that define the fused router kernel (a counter summary is valid only for them)."""
    h = hashlib.sha256()
    for f in ("router.hip", "epilogue.h", "common.h"):
        with open(os.path.join(_PKG, "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _short(name: str, n: int = 90) -> str:
    name = name.replace("idb::(anonymous namespace)::", "").replace("idb::", "")
    return name if len(name) <= n else name[: n - 3] + "..."


def stats_markdown(csv_path: str, cmd: str, title: str, top: int = 10) -> str:
    rows = list(csv.DictReader(open(csv_path)))
    lines = [f"# {title}", "", "Command:", "", "```", cmd, "```", "",
             "| kernel | calls | avg us | min us | max us | share % |", "|---|---:|---:|---:|---:|---:|"]
    for r in rows[:top]:
        lines.append(f"| `{_short(r['Name'])}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    return "\n".join(lines) + "\n"


def _counter_rows(csv_path: str, counter: str):
    out = []
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] == counter:
            out.append((r["Kernel_Name"], float(r["Counter_Value"])))
    return out


def _calibrated(csv_path: str, counter: str, copy_bytes: int):
    rows = _counter_rows(csv_path, counter)
    router = [v for n, v in rows if _is_router(n)]
    copies = [v for n, v in rows if not _is_router(n) and "copy" in n.lower()]
    if not router or not copies:
        raise SystemExit(f"{csv_path}: no {counter} readings for the router kernel or the calibration copy")
    copy_kib = max(copies)
    factor = copy_kib * 1024.0 / copy_bytes
    kib = statistics.mean(router)
    return {"counter": counter, "router_kib_per_dispatch": kib, "router_dispatches": len(router),
            "copy_kib": copy_kib, "copy_bytes": copy_bytes, "factor": factor,
            "router_bytes": kib * 1024.0 / factor}


def traffic(args) -> None:
    f = _calibrated(args.fetch, "FETCH_SIZE", args.copy_bytes)
    w = _calibrated(args.write, "WRITE_SIZE", args.copy_bytes)
    total = f["router_bytes"] + w["router_bytes"]
    d = {"workload": args.workload, "variant": args.variant, "source_sha256": router_source_hash(),
         "hbm_bytes_per_launch": round(total), "fetch": f, "write": w,
         "cmd_fetch": args.cmd_fetch, "cmd_write": args.cmd_write}
    with open(args.out + ".json", "w") as fh:
        json.dump(d, fh, indent=1)
    md = [f"# HBM traffic of the fused router kernel, {args.workload} (variant {args.variant})", "",
          "Counters in KiB per dispatch; the calibration is a device-to-device copy of "
          f"{args.copy_bytes} bytes in the same run.", "",
          "| counter | router KiB/dispatch | dispatches | copy KiB | factor | router bytes (calibrated) |",
          "|---|---:|---:|---:|---:|---:|"]
    for c in (f, w):
        md.append(f"| {c['counter']} | {c['router_kib_per_dispatch']:.1f} | {c['router_dispatches']} | "
                  f"{c['copy_kib']:.1f} | {c['factor']:.4f} | {c['router_bytes']:.4g} |")
    md += ["", f"Total HBM bytes per launch: {total:.4g}", "", "Commands:", "", "```", args.cmd_fetch,
           args.cmd_write, "```", "", f"Router sources hash: `{d['source_sha256']}`", ""]
    with open(args.out + ".md", "w") as fh:
        fh.write("\n".join(md))
    print(json.dumps({"hbm_bytes_per_launch": d["hbm_bytes_per_launch"], "fetch_factor": f["factor"],
                      "write_factor": w["factor"]}))


def counters(args) -> None:
    """Per-dispatch means of the fused router kernel's counters in one --pmc pass."""
    per = {}
    for r in csv.DictReader(open(args.csv)):
        if _is_router(r["Kernel_Name"]):
            per.setdefault(r["Counter_Name"], {}).setdefault(r["Dispatch_Id"], 0.0)
            per[r["Counter_Name"]][r["Dispatch_Id"]] += float(r["Counter_Value"])
    if not per:
        raise SystemExit(f"{args.csv}: no readings for the router kernel")
    mean = {c: statistics.mean(v.values()) for c, v in per.items()}
    n = max(len(v) for v in per.values())
    md = [f"# {args.title}", "", "Command:", "", "```", args.cmd, "```", "",
          f"Per-dispatch values (mean over {n} dispatches of the fused router kernel), summed over the chip.", "",
          "| counter | per dispatch |", "|---|---:|"]
    for c in sorted(mean):
        md.append(f"| {c} | {mean[c]:.4g} |")
    if "SQ_VALU_MFMA_BUSY_CYCLES" in mean and "SQ_INSTS_VALU_MFMA_MOPS_BF16" not in mean:
        md += ["", f"MFMA busy cycles per SIMD ({args.simds} SIMDs): "
               f"{mean['SQ_VALU_MFMA_BUSY_CYCLES'] / args.simds:.4g}"]
    if "SQ_WAIT_INST_ANY" in mean and "SQ_WAVE_CYCLES" in mean:
        md.append(f"Share of wave cycles waiting for an instruction to issue: "
                  f"{mean['SQ_WAIT_INST_ANY'] / mean['SQ_WAVE_CYCLES']:.3f}")
    if "SQ_WAIT_INST_LDS" in mean and "SQ_WAVE_CYCLES" in mean:
        md.append(f"Share of wave cycles waiting on LDS: {mean['SQ_WAIT_INST_LDS'] / mean['SQ_WAVE_CYCLES']:.3f}")
    md.append("")
    with open(args.out, "w") as fh:
        fh.write("\n".join(md))


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="action", required=True)
    a = sub.add_parser("stats")
    a.add_argument("csv")
    a.add_argument("--cmd", required=True)
    a.add_argument("--title", default="Kernel statistics")
    a.add_argument("--out", required=True)
    b = sub.add_parser("traffic")
    b.add_argument("--fetch", required=True)
    b.add_argument("--write", required=True)
    b.add_argument("--copy-bytes", type=int, required=True)
    b.add_argument("--workload", required=True)
    b.add_argument("--variant", type=int, required=True)
    b.add_argument("--cmd-fetch", required=True)
    b.add_argument("--cmd-write", required=True)
    b.add_argument("--out", required=True, help="output path without extension (.json and .md are written)")
    c = sub.add_parser("counters")
    c.add_argument("csv")
    c.add_argument("--cmd", required=True)
    c.add_argument("--title", default="Hardware counters")
    c.add_argument("--simds", type=int, default=1024)
    c.add_argument("--out", required=True)
    args = ap.parse_args(argv)
    if args.action == "stats":
        with open(args.out, "w") as fh:
            fh.write(stats_markdown(args.csv, args.cmd, args.title))
    elif args.action == "counters":
        counters(args)
    else:
        traffic(args)
    return 0


if __name__ == "__main__":
    sys.exit(main())
