"""Summarise rocprofv3 output for one kernel into a short markdown file.

    python -m paper_2412_15803_amd.profsum --kernel grouped_m1_kernel \
        --trace <dir with *_kernel_trace.csv> --fetch <dir of a --pmc FETCH_SIZE run> \
        --write <dir of a --pmc WRITE_SIZE run> --algo-bytes N --copy-mib C \
        --command "<the rocprofv3 command>" --out profiles/<name>.md

Durations come from the kernel trace.  HBM traffic per launch is FETCH_SIZE
and WRITE_SIZE (KiB per dispatch) scaled by what the same counters read for a
plain device copy of C MiB in the same run (its true traffic is C MiB read and
C MiB written).  The summary records the library's source hash; bench.py
reports the traffic figure only while the sources still match it.
"""

from __future__ import annotations

import argparse
import csv
import glob
import os
import statistics

from .build import STEP_KERNEL_SOURCES, source_hash


def _rows(directory, pattern):
    out = []
    for f in sorted(glob.glob(os.path.join(directory, "**", pattern), recursive=True)):
        with open(f, newline="") as fh:
            out.extend(csv.DictReader(fh))
    return out


def _counter(directory, name):
    """[(kernel name, grid size, value)] for one counter, one entry per
    dispatch, in dispatch order."""
    rows = [r for r in _rows(directory, "*counter_collection.csv") if r["Counter_Name"] == name]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    return [(r["Kernel_Name"], int(r["Grid_Size"]), float(r["Counter_Value"])) for r in rows]


def _copy_value(entries):
    copies = [v for name, _, v in entries if "copy" in name.lower()]
    if not copies:
        raise SystemExit("no copy kernel found in the counter run (bench.py --copy-probe-mib)")
    return max(copies)


def _durations(trace_dir, kernel, skip=0, take=0):
    """Durations (us) of the kernel's launches in start order; with skip/take
    only launches [skip, skip + take) of them (take 0: all after skip)."""
    trace = [r for r in _rows(trace_dir, "*kernel_trace.csv") if kernel in r["Kernel_Name"]]
    if not trace:
        raise SystemExit(f"kernel {kernel!r} not in the trace")
    trace.sort(key=lambda r: int(r["Start_Timestamp"]))
    sel = trace[skip:skip + take] if take else trace[skip:]
    if not sel:
        raise SystemExit(f"no launches of {kernel!r} left after skipping {skip}")
    return [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in sel]


def _traffic(fetch, write, f_scale, w_scale, kernel, skip=0, take=0):
    """Mean scaled fetch and write bytes per dispatch of the kernel; with
    skip/take only its dispatches [skip, skip + take) in dispatch order."""
    kf = [v for name, _, v in fetch if kernel in name]
    kw = [v for name, _, v in write if kernel in name]
    kf = kf[skip:skip + take] if take else kf[skip:]
    kw = kw[skip:skip + take] if take else kw[skip:]
    if not kf or not kw:
        raise SystemExit(f"kernel {kernel!r} not in the counter runs")
    return kf, kw, statistics.mean(kf) * f_scale * 1024.0, statistics.mean(kw) * w_scale * 1024.0


def summarise(args):
    durs = _durations(args.trace, args.kernel, args.skip, args.take)
    med = statistics.median(durs)
    fetch = _counter(args.fetch, "FETCH_SIZE")
    write = _counter(args.write, "WRITE_SIZE")
    copy_kib = args.copy_mib * 1024.0
    f_scale = copy_kib / _copy_value(fetch)
    w_scale = copy_kib / _copy_value(write)
    kf, kw, fetch_b, write_b = _traffic(fetch, write, f_scale, w_scale, args.kernel, args.counter_skip,
                                        args.counter_take)
    traffic = fetch_b + write_b
    avg = statistics.mean(durs)
    others = []
    for k in args.also or ():
        d = _durations(args.trace, k)
        _, _, fb, wb = _traffic(fetch, write, f_scale, w_scale, k)
        others.append(f"| other kernel `{k}`: launches, avg duration (us), scaled fetch + write bytes | "
                      f"{len(d)}, {statistics.mean(d):.2f}, {fb:,.0f} + {wb:,.0f} |")
    names = tuple(args.sources.split(",")) if args.sources else STEP_KERNEL_SOURCES
    src_hash = source_hash(names)
    lines = [
        f"# {args.title}",
        "",
        "Commands (each from /tmp with TMPDIR=/tmp, one MI355X):",
        "",
        "```",
        *args.command,
        "```",
        "",
        "| Figure | Value |",
        "|---|---|",
        f"| kernel | `{args.kernel}` |",
        f"| launches summarised | {len(durs)}"
        + (f" (the kernel's launches {args.skip}..{args.skip + len(durs) - 1} in start order: {args.select})"
           if args.skip or args.take else "") + " |",
        f"| duration median / avg / min / max (us) | {med:.2f} / {avg:.2f} / {min(durs):.2f} / {max(durs):.2f} |",
        f"| algorithmic bytes per launch | {args.algo_bytes:,} |",
        f"| achieved (algorithmic bytes / median duration) | {args.algo_bytes / (med * 1e3):.1f} GB/s"
        f" = {args.algo_bytes / (med * 1e3) / 8000:.4f} of 8 TB/s |",
        f"| achieved (algorithmic bytes / avg duration) | {args.algo_bytes / (avg * 1e3):.1f} GB/s |",
        f"| FETCH_SIZE per launch (raw KiB, mean of {len(kf)}"
        + (f": the kernel's dispatches {args.counter_skip}..{args.counter_skip + len(kf) - 1} of each counter run"
           if args.counter_skip or args.counter_take else "") + f") | {statistics.mean(kf):,.1f} |",
        f"| WRITE_SIZE per launch (raw KiB, mean of {len(kw)}) | {statistics.mean(kw):,.1f} |",
        f"| copy calibration: FETCH_SIZE / WRITE_SIZE of a {args.copy_mib} MiB copy (raw KiB) | "
        f"{_copy_value(fetch):,.1f} / {_copy_value(write):,.1f} |",
        f"| scale factors applied (fetch / write) | {f_scale:.4f} / {w_scale:.4f} |",
        f"| HBM traffic per launch, scaled (fetch + write bytes) | {fetch_b:,.0f} + {write_b:,.0f} = {traffic:,.0f} |",
        f"| traffic / algorithmic bytes | {traffic / args.algo_bytes:.4f} |",
        *([f"| flops per launch; achieved (flops / avg duration) | {args.flops:,} ; "
           f"{args.flops / (avg * 1e-6) / 1e12:.1f} TFLOP/s |"] if args.flops else []),
        *others,
        "",
        "Machine-readable (read by bench.py; valid only for this source hash):",
        "",
        "```",
        f"source_hash: {src_hash}",
        f"source_files: {','.join(names)}",
        f"traffic_bytes_per_launch: {traffic:.0f}",
        f"avg_duration_us: {avg:.3f}",
        f"median_duration_us: {med:.3f}",
        f"launches_summarised: {len(durs)}",
        "```",
        "",
    ]
    with open(args.out, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))


def parse_summary(path):
    """The machine-readable block of a summary written above as a dict of
    strings, or None (no file, or no source hash and traffic in it)."""
    try:
        with open(path) as fh:
            text = fh.read()
    except OSError:
        return None
    vals = {}
    for line in text.splitlines():
        if ":" in line and not line.startswith("|"):
            k, _, v = line.partition(":")
            vals[k.strip()] = v.strip()
    if "source_hash" not in vals or "traffic_bytes_per_launch" not in vals:
        return None
    return vals


def parse_traffic(path):
    """(source_hash, traffic bytes per launch) from a summary written above, or None."""
    vals = parse_summary(path)
    if vals is None:
        return None
    return vals["source_hash"], float(vals["traffic_bytes_per_launch"])


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--kernel", required=True, help="substring of the kernel name")
    ap.add_argument("--trace", required=True)
    ap.add_argument("--fetch", required=True)
    ap.add_argument("--write", required=True)
    ap.add_argument("--algo-bytes", type=int, required=True)
    ap.add_argument("--copy-mib", type=int, required=True)
    ap.add_argument("--command", action="append", required=True)
    ap.add_argument("--title", default="Kernel trace and HBM traffic")
    ap.add_argument("--also", action="append", help="another kernel to list (durations and traffic)")
    ap.add_argument("--flops", type=int, default=0, help="flops per launch, for a matrix-core kernel")
    ap.add_argument("--sources", default=None,
                    help="comma-separated csrc/ files whose hash marks the summary (default: the step kernel's)")
    ap.add_argument("--skip", type=int, default=0, help="leave out the kernel's first N launches (warm-up)")
    ap.add_argument("--take", type=int, default=0, help="then summarise only the next N launches (0: all)")
    ap.add_argument("--select", default="", help="what the selected launches are, for the summary")
    ap.add_argument("--counter-skip", type=int, default=0, help="leave out the kernel's first N dispatches of the counter runs")
    ap.add_argument("--counter-take", type=int, default=0, help="then use only the next N dispatches (0: all)")
    ap.add_argument("--out", required=True)
    summarise(ap.parse_args())


if __name__ == "__main__":
    main()
