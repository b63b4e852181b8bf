"""Vector ALUs against matrix cores for small batches, in one process.

    python -m paper_2412_15803_amd.small_batch_compare            # timings
    rocprofv3 --kernel-trace --output-format csv -d OUT -o trace -- \
        python3 -m paper_2412_15803_amd.small_batch_compare
    python -m paper_2412_15803_amd.small_batch_compare --summarise OUT --out profiles/small_batch_paths.md

For each shape and batch size M, the same wq_gemv calls run once through the
vector-ALU kernel (WQ_SMALL_BATCH_VECTOR=1, read by the library at every
call) and once through the default path (matrix cores from M = 3 on).
Calls rotate over copies of random codes and scales totalling >= 1 GiB, so
every call streams its weights from HBM.
"""

from __future__ import annotations

import argparse
import csv
import glob
import os
import statistics

SHAPES = ((28672, 4096), (4096, 14336), (128256, 4096))
BATCHES = (4, 8, 16)
CALLS = 40


def run():
    import torch

    from . import workloads as wl
    from . import wq

    dev = torch.device("cuda:0")
    gen = torch.Generator(device=dev)
    gen.manual_seed(11)
    for n, k in SHAPES:
        r = max(1, -(-(1 << 30) // wl.ideal_bytes(n, k, 1)))
        ws = []
        for _ in range(r):
            p = torch.randint(-2**31, 2**31 - 1, (n, k // 8), dtype=torch.int32, device=dev, generator=gen)
            s = (torch.rand((n, k // 32), device=dev, generator=gen) * 0.01 + 0.001).to(torch.float16)
            ws.append((p, s))
        for m in BATCHES:
            x = torch.randn((m, k), device=dev, generator=gen).to(torch.float16)
            y = torch.empty((m, n), dtype=torch.float16, device=dev)
            for path in ("vector", "default"):
                if path == "vector":
                    os.environ["WQ_SMALL_BATCH_VECTOR"] = "1"
                else:
                    os.environ.pop("WQ_SMALL_BATCH_VECTOR", None)
                for i in range(3):
                    wq.wq_gemv(*ws[i % r], x, y)
                torch.cuda.synchronize()
                a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                a.record()
                for i in range(CALLS):
                    wq.wq_gemv(*ws[i % r], x, y)
                e.record()
                torch.cuda.synchronize()
                us = a.elapsed_time(e) * 1e3 / CALLS
                print(f"{n}x{k} M={m:2d} {path:7s}: {us:8.2f} us per call (events, host launch included)", flush=True)
        del ws
        torch.cuda.empty_cache()
    os.environ.pop("WQ_SMALL_BATCH_VECTOR", None)


def _schedule():
    """(shape, M, path, launches per call) in the order run() issues them."""
    out = []
    for n, k in SHAPES:
        for m in BATCHES:
            for path in ("vector", "default"):
                per_call = -(-m // 8) if path == "vector" else -(-m // 16)
                out.append(((n, k), m, path, per_call))
    return out


def summarise(trace_dir, out):
    """Kernel durations per (shape, M, path) from a rocprofv3 kernel trace of
    run(): the small-batch launches, in dispatch order, follow run()'s fixed
    order (3 warm-up and CALLS timed calls per case)."""
    rows = []
    for f in glob.glob(os.path.join(trace_dir, "**", "*kernel_trace.csv"), recursive=True):
        with open(f, newline="") as fh:
            rows.extend(csv.DictReader(fh))
    launches = [r for r in rows if "gemv_mb_kernel" in r["Kernel_Name"] or "gemm_mfma_kernel" in r["Kernel_Name"]]
    launches.sort(key=lambda r: int(r["Start_Timestamp"]))
    lines = ["# Small batches: vector-ALU kernel against matrix-core kernel", "",
             "Commands (from /tmp with TMPDIR=/tmp and PYTHONPATH=<repo>, one MI355X):", "", "```",
             "rocprofv3 --kernel-trace --output-format csv -d <out> -o trace -- "
             "python3 -m paper_2412_15803_amd.small_batch_compare",
             "python -m paper_2412_15803_amd.small_batch_compare --summarise <out> --out profiles/small_batch_paths.md",
             "```", "",
             f"Per case: {CALLS} timed wq_gemv calls after 3 warm-up calls, rotating over >= 1 GiB of weight copies. "
             "Kernel time per call = sum of its launches (the vector path runs 8 batch rows per launch). "
             "The default path is the vector kernel at M = 2 and the matrix-core kernel from M = 3 on.", "",
             "| Shape N x K | M | Path | Kernel | Launches per call | Kernel us per call (avg) | GB/s |",
             "|---|---|---|---|---|---|---|"]
    i = 0
    for (n, k), m, path, per_call in _schedule():
        count = (3 + CALLS) * per_call
        seg = launches[i:i + count]
        i += count
        if len(seg) < count:
            raise SystemExit("trace has fewer small-batch launches than run() issues")
        timed = seg[3 * per_call:]
        durs = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in timed]
        per = sum(durs) / CALLS
        kname = timed[0]["Kernel_Name"].split("(")[0].split("::")[-1]
        if "<" not in kname:
            kname = "gemv_mb_kernel" if "gemv_mb_kernel" in timed[0]["Kernel_Name"] else "gemm_mfma_kernel"
        ideal = n * k // 2 + n * (k // 32) * 2 + 2 * m * k + 2 * m * n
        lines.append(f"| {n}x{k} | {m} | {path} | `{kname}` | {per_call} | {per:.2f} | {ideal / (per * 1e3):.1f} |")
    lines.append("")
    with open(out, "w") as fh:
        fh.write("\n".join(lines))
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--summarise", metavar="TRACE_DIR")
    ap.add_argument("--out", default="profiles/small_batch_paths.md")
    args = ap.parse_args()
    if args.summarise:
        summarise(args.summarise, args.out)
    else:
        run()


if __name__ == "__main__":
    main()
