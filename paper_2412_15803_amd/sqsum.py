"""Summarise rocprofv3 SQ counter runs per kernel into a markdown table.

    python -m paper_2412_15803_amd.sqsum --pmc <dir of one --pmc run> [--pmc <dir> ...] \
        --command "<rocprofv3 command>" [--command ...] --title "<title>" --out profiles/<name>.md

Every counter is averaged over a kernel's dispatches.  Derived figures, for
MI355X (8 XCDs, 256 CUs, 1024 SIMDs; a wave64 VALU instruction occupies its
SIMD for 4 cycles):
- clock = GRBM_GUI_ACTIVE / 8 XCDs / dispatch duration;
- VALU busy = 4 * SQ_INSTS_VALU / (1024 * GRBM_GUI_ACTIVE / 8);
- MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (1024 * GRBM_GUI_ACTIVE / 8).
"""

from __future__ import annotations

import argparse
import collections
import csv
import glob
import os
import re
import statistics


def _short(name):
    m = re.search(r"(\w+_kernel(?:<[^>]*>)?)", name)
    return m.group(1) if m else name


def collect(dirs, split=None):
    """{kernel: {counter: mean over dispatches, 'us': mean duration, 'n': dispatches}}.

    `split` maps a kernel's short name to [(label, count), ...]: its
    dispatches in each run, in launch order, are divided into consecutive
    groups reported as separate columns "kernel label"."""
    split = split or {}
    per = collections.defaultdict(lambda: collections.defaultdict(list))
    durs = collections.defaultdict(dict)
    for d in dirs:
        for f in sorted(glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)):
            with open(f, newline="") as fh:
                rows = list(csv.DictReader(fh))
            sums = collections.defaultdict(float)
            when = {}
            for r in rows:
                if "wq::" not in r["Kernel_Name"]:
                    continue
                name, did = _short(r["Kernel_Name"]), int(r["Dispatch_Id"])
                sums[(name, did, r["Counter_Name"])] += float(r["Counter_Value"])
                when[(name, did)] = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
            # Each kernel's dispatches of this run in launch order, relabelled by `split`.
            label = {}
            for name in {k[0] for k in when}:
                ids = sorted(did for (n, did) in when if n == name)
                groups = split.get(name)
                if not groups:
                    for did in ids:
                        label[(name, did)] = name
                    continue
                i = 0
                for lab, count in groups:
                    for did in ids[i:i + count]:
                        label[(name, did)] = f"{name} {lab}"
                    i += count
                for did in ids[i:]:
                    label[(name, did)] = f"{name} (rest)"
            for (name, did), us in when.items():
                durs[label[(name, did)]][(f, did)] = us
            for (name, did, c), v in sums.items():
                per[label[(name, did)]][c].append(v)
    out = {}
    for k, cs in per.items():
        out[k] = {c: statistics.mean(v) for c, v in cs.items()}
        out[k]["us"] = statistics.mean(durs[k].values())
        out[k]["n"] = len(durs[k])
    return out


def _parse_split(items):
    out = {}
    for item in items or []:
        kernel, groups = item.split("=", 1)
        out[kernel] = [(g.rsplit(":", 1)[0], int(g.rsplit(":", 1)[1])) for g in groups.split(",")]
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--pmc", action="append", required=True)
    ap.add_argument("--command", action="append", required=True)
    ap.add_argument("--title", required=True)
    ap.add_argument("--split", action="append",
                    help="KERNEL=LABEL:COUNT,LABEL:COUNT: report a kernel's dispatches of each run, in launch "
                         "order, as separate columns")
    ap.add_argument("--out", required=True)
    a = ap.parse_args()
    res = collect(a.pmc, _parse_split(a.split))
    lines = [f"# {a.title}", "", "Commands (each from /tmp with TMPDIR=/tmp, one MI355X):", "", "```"]
    lines += a.command
    lines += ["```", "", "Summary: `python -m paper_2412_15803_amd.sqsum` over the runs above.", ""]
    names = sorted(res)
    counters = sorted({c for k in names for c in res[k] if c not in ("us", "n")})
    lines.append("| Figure | " + " | ".join(f"`{k}`" for k in names) + " |")
    lines.append("|---|" + "---|" * len(names))

    def row(label, fn):
        vals = []
        for k in names:
            try:
                vals.append(fn(res[k]))
            except (KeyError, ZeroDivisionError):
                vals.append("—")
        lines.append(f"| {label} | " + " | ".join(vals) + " |")

    row("dispatches (per run)", lambda r: str(r["n"] // max(1, len(a.pmc))))
    row("duration avg (us)", lambda r: f"{r['us']:.1f}")
    row("clock (GHz)", lambda r: f"{r['GRBM_GUI_ACTIVE'] / 8 / (r['us'] * 1e3):.2f}")
    row("VALU busy", lambda r: f"{4 * r['SQ_INSTS_VALU'] / (1024 * r['GRBM_GUI_ACTIVE'] / 8):.0%}")
    row("MFMA busy", lambda r: f"{r['SQ_VALU_MFMA_BUSY_CYCLES'] / (1024 * r['GRBM_GUI_ACTIVE'] / 8):.0%}")
    for c in counters:
        row(c, lambda r, c=c: f"{r[c]:,.0f}")
    with open(a.out, "w") as fh:
        fh.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
