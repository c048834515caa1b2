"""Summaries of rocprofv3 CSV output for the ``profiles/`` folder.

Three commands, all run on the CPU over files a profiled run wrote:

``stats``: a ``*_kernel_stats.csv`` of ``rocprofv3 --kernel-trace --stats``
becomes a short markdown table (calls, average/min/max duration, share).

``counters``: per-dispatch means of one kernel family's counters from one
``--pmc`` pass (MFMA busy cycles and instruction counts, wait cycles, LDS
bank conflicts).

``traffic``: the ``*_counter_collection.csv`` of a ``FETCH_SIZE`` pass and of
a ``WRITE_SIZE`` pass over ``bench.py --pmc-pass`` become the HBM bytes per
launch of the fused router kernel, the slice merge and the selection from
given scores.  Both counters are read in KiB per dispatch.  The pass runs one
device-to-device copy of known size before the counted launches; the ratio
of what each counter reports for that copy to its true size is the
calibration factor, and the kernels' readings are divided by it.  The result
is written as JSON (read by ``bench.py`` as ``roofline.traffic``, and only
while the router sources still hash to the recorded value) plus a markdown
note.

    python -m paper_2609_39137_amd.profsum stats CSV --cmd "..." --out profiles/X.md
    python -m paper_2609_39137_amd.profsum traffic --fetch CSV --write CSV --copy-bytes N \\
        --workload NAME --variant V --cmd-fetch "..." --cmd-write "..." --out profiles/Y
    python -m paper_2609_39137_amd.profsum counters CSV --family router --cmd "..." --out profiles/Z.md
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
    """Hash of the sources of the counted kernels (fused router, slice merge with the update, selection from
    given scores): a counter summary is valid only for them."""
    h = hashlib.sha256()
    for f in ("router.hip", "epilogue.h", "common.h", "controller_block.h", "select.hip"):
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


# kernel families whose HBM bytes the counter passes report: the fused
# router kernel, the slice merge (with the update in its last workgroup) and
# the unfused selection from given scores
FAMILIES = {
    "router": ROUTER_KERNELS,
    "merge": ("router_merge_tile_kernel", "router_merge_kernel"),
    "select": ("select_reg_kernel", "select_kernel"),
}


def _family(name: str):
    for fam, keys in FAMILIES.items():
        if any(k in name for k in keys):
            return fam
    return None


def stats_json(csv_path: str, cmd: str) -> dict:
    """Average duration per kernel family (the launch-weighted mean over its instantiations) of a kernel trace."""
    fam = {}
    for r in csv.DictReader(open(csv_path)):
        f = _family(r["Name"])
        if f is None:
            continue
        calls, total = fam.get(f, (0, 0.0))
        fam[f] = (calls + int(r["Calls"]), total + float(r["TotalDurationNs"]))
    return {"source_sha256": router_source_hash(), "cmd": cmd,
            "kernels": {f: {"calls": c, "avg_us": t / c / 1e3} for f, (c, t) in fam.items()}}


def _counter_rows(csv_path: str, counter: str):
    """(dispatch id, kernel name, value) of one counter, values summed over a dispatch's rows."""
    per = {}
    for r in csv.DictReader(open(csv_path)):
        if r["Counter_Name"] == counter:
            key = int(r["Dispatch_Id"])
            name, v = per.get(key, (r["Kernel_Name"], 0.0))
            per[key] = (name, v + float(r["Counter_Value"]))
    return sorted((k, n, v) for k, (n, v) in per.items())


def _calibrated(csv_path: str, counter: str, copy_bytes: int):
    """Per-family mean of a byte counter over the dispatches after the calibration copy, calibrated by it."""
    rows = _counter_rows(csv_path, counter)
    copies = [(k, v) for k, n, v in rows if _family(n) is None and "copy" in n.lower()]
    if not copies:
        raise SystemExit(f"{csv_path}: no {counter} reading for the calibration copy")
    copy_id, copy_kib = max(copies, key=lambda c: c[1])
    factor = copy_kib * 1024.0 / copy_bytes
    out = {"counter": counter, "copy_kib": copy_kib, "copy_bytes": copy_bytes, "factor": factor, "kernels": {}}
    for fam in FAMILIES:
        vals = [v for k, n, v in rows if k > copy_id and _family(n) == fam]
        if vals:
            kib = statistics.mean(vals)
            out["kernels"][fam] = {"kib_per_dispatch": kib, "dispatches": len(vals), "bytes": kib * 1024.0 / factor}
    if "router" not in out["kernels"]:
        raise SystemExit(f"{csv_path}: no {counter} readings for the router kernel after the calibration copy")
    return out


def traffic(args) -> None:
    f = _calibrated(args.fetch, "FETCH_SIZE", args.copy_bytes)
    w = _calibrated(args.write, "WRITE_SIZE", args.copy_bytes)
    kern = {}
    for fam in f["kernels"]:
        if fam in w["kernels"]:
            kern[fam] = {"fetch_bytes": round(f["kernels"][fam]["bytes"]), "write_bytes": round(w["kernels"][fam]["bytes"]),
                         "hbm_bytes_per_launch": round(f["kernels"][fam]["bytes"] + w["kernels"][fam]["bytes"]),
                         "dispatches": f["kernels"][fam]["dispatches"]}
    d = {"workload": args.workload, "variant": args.variant, "source_sha256": router_source_hash(),
         "hbm_bytes_per_launch": kern["router"]["hbm_bytes_per_launch"], "kernels": kern,
         "fetch_factor": f["factor"], "write_factor": w["factor"], "copy_bytes": args.copy_bytes,
         "cmd_fetch": args.cmd_fetch, "cmd_write": args.cmd_write}
    with open(args.out + ".json", "w") as fh:
        json.dump(d, fh, indent=1)
    md = [f"# HBM traffic per launch, {args.workload} (router variant {args.variant})", "",
          "FETCH_SIZE and WRITE_SIZE are read in KiB per dispatch, over the dispatches after a device-to-device "
          f"copy of {args.copy_bytes} bytes in the same run; each is divided by the ratio it reports for that "
          f"copy (FETCH_SIZE {f['factor']:.4f}, WRITE_SIZE {w['factor']:.4f}).", "",
          "| kernel | dispatches | fetched bytes | written bytes | HBM bytes per launch |", "|---|---:|---:|---:|---:|"]
    names = {"router": "fused router kernel", "merge": "slice merge + update", "select": "select from scores"}
    for fam, k in kern.items():
        md.append(f"| {names[fam]} | {k['dispatches']} | {k['fetch_bytes']:.4g} | {k['write_bytes']:.4g} | "
                  f"{k['hbm_bytes_per_launch']:.4g} |")
    md += ["", "Commands:", "", "```", args.cmd_fetch, args.cmd_write, "```", "",
           f"Router sources hash: `{d['source_sha256']}`", ""]
    with open(args.out + ".md", "w") as fh:
        fh.write("\n".join(md))
    print(json.dumps({"kernels": kern, "fetch_factor": f["factor"], "write_factor": w["factor"]}))


def counters(args) -> None:
    """Per-dispatch means of the fused router kernel's counters in one --pmc pass."""
    per = {}
    for r in csv.DictReader(open(args.csv)):
        if _family(r["Kernel_Name"]) == args.family:
            per.setdefault(r["Counter_Name"], {}).setdefault(r["Dispatch_Id"], 0.0)
            per[r["Counter_Name"]][r["Dispatch_Id"]] += float(r["Counter_Value"])
    if not per:
        raise SystemExit(f"{args.csv}: no readings for the {args.family} kernel")
    mean = {c: statistics.mean(v.values()) for c, v in per.items()}
    n = max(len(v) for v in per.values())
    md = [f"# {args.title}", "", "Command:", "", "```", args.cmd, "```", "",
          f"Per-dispatch values (mean over {n} dispatches of the {args.family} kernel), summed over the chip.", "",
          "| counter | per dispatch |", "|---|---:|"]
    for c in sorted(mean):
        md.append(f"| {c} | {mean[c]:.4g} |")
    md.append("")
    if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in mean and mean["SQ_INSTS_VALU_MFMA_MOPS_BF16"] > 0:
        md.append(f"bf16 MFMA flops per dispatch (512 per MOPS unit): {512 * mean['SQ_INSTS_VALU_MFMA_MOPS_BF16']:.4g}")
    if "SQ_VALU_MFMA_BUSY_CYCLES" in mean and mean["SQ_VALU_MFMA_BUSY_CYCLES"] > 0:
        md.append(f"MFMA busy cycles per SIMD ({args.simds} SIMDs): "
                  f"{mean['SQ_VALU_MFMA_BUSY_CYCLES'] / args.simds:.4g}")
    if "SQ_WAIT_INST_ANY" in mean and "SQ_WAVE_CYCLES" in mean:
        md.append(f"Share of wave cycles waiting for an instruction to issue: "
                  f"{mean['SQ_WAIT_INST_ANY'] / mean['SQ_WAVE_CYCLES']:.3f}")
    if "SQ_WAIT_INST_LDS" in mean and "SQ_WAVE_CYCLES" in mean:
        md.append(f"Share of wave cycles waiting on LDS: {mean['SQ_WAIT_INST_LDS'] / mean['SQ_WAVE_CYCLES']:.3f}")
    if "TCC_HIT_sum" in mean and "TCC_MISS_sum" in mean and mean["TCC_HIT_sum"] + mean["TCC_MISS_sum"] > 0:
        md.append(f"L2 hit rate: {mean['TCC_HIT_sum'] / (mean['TCC_HIT_sum'] + mean['TCC_MISS_sum']):.3f}")
    if args.units:
        # instruction counters count wave instructions; a wave has 64 lanes
        for c in sorted(mean):
            if c.startswith("SQ_INSTS_"):
                md.append(f"{c} per {args.unit_name}: {mean[c] / args.units:.4g} wave instructions, "
                          f"{64 * mean[c] / args.units:.4g} lane operations")
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
    a.add_argument("--json", default=None, help="also write per-family average durations (read by bench.py)")
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
    c.add_argument("--family", default="router", choices=sorted(FAMILIES))
    c.add_argument("--units", type=float, default=0.0, help="work units per dispatch (e.g. T*E scores)")
    c.add_argument("--unit-name", default="unit")
    c.add_argument("--out", required=True)
    args = ap.parse_args(argv)
    if args.action == "stats":
        with open(args.out, "w") as fh:
            fh.write(stats_markdown(args.csv, args.cmd, args.title))
        if args.json:
            with open(args.json, "w") as fh:
                json.dump(stats_json(args.csv, args.cmd), fh, indent=1)
    elif args.action == "counters":
        counters(args)
    else:
        traffic(args)
    return 0


if __name__ == "__main__":
    sys.exit(main())
