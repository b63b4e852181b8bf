#!/usr/bin/env python3
"""Benchmark: one decode step of 4-bit linears at batch 1 on one MI355X.

Workload: a 3B-class decode step -- 28 layers x (qkv 5120x3072, o 3072x3072,
gate_up 16384x3072, down 3072x8192) + lm_head 128256x3072, all symmetric
4-bit with groups of 32 and fp16 scales, fp16 activations, M = 1: 113 linears
and 1,809,859,072 bytes of weights, scales, x and y per step.  Weights are
seeded N(0, 0.02^2), generated and packed on the device; x ~ N(0, 1) per
linear.  A step is one wq_decode_linears call over all 113 linears, with every
input already resident in HBM.

Prints ONE JSON line: value = achieved GB/s of algorithmic bytes per step.
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

HBM_PEAK_GBS = 8000.0
ROOT = os.path.dirname(os.path.abspath(__file__))
# rocprofv3 summary of the step kernel (duration, FETCH_SIZE / WRITE_SIZE);
# its traffic figure is used only while the library sources still match.
STEP_PROFILE = os.path.join(ROOT, "profiles", "grouped_m1_3b_step.md")
METRIC = "achieved HBM GB/s (% of peak) & µs per decode step of 4-bit linears, batch 1"


def parse_args():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--seed", type=int, default=1234)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="approximate CPU time budget of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--chained", action="store_true",
                    help="also time the step with every linear reading its predecessor's output")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (for scaling HBM counters)")
    ap.add_argument("--attention-only", action="store_true",
                    help="time only the paged decode-attention shapes (for profiling its kernels)")
    ap.add_argument("--attention-config", type=int, default=None,
                    help="with --attention-only: time only this entry of ATTN_CONFIGS")
    ap.add_argument("--attention-eager", action="store_true",
                    help="with --attention-only: launch every call from the host (no HIP graph)")
    ap.add_argument("--dependent-only", action="store_true",
                    help="time only the dependent decode step (for profiling the fused kernels)")
    ap.add_argument("--dependent-ctx", type=int, default=0,
                    help="with --dependent-only: cached tokens per layer for attention (0: linears only)")
    ap.add_argument("--dependent-eager", action="store_true",
                    help="with --dependent-only: the persistent chain (WQ_FUSED_PERSISTENT=1) launched from the host")
    ap.add_argument("--prefill-only", action="store_true",
                    help="time only the prefill GEMM shapes (for profiling its kernel)")
    ap.add_argument("--prefill-config", type=int, default=None,
                    help="with --prefill-only: time only this entry of PREFILL_CONFIGS")
    ap.add_argument("--step-batches", type=str, default=None,
                    help="time only the 3B-class step at these comma-separated batch sizes (for counters)")
    ap.add_argument("--layers-only", action="store_true",
                    help="time only the one-call-per-layer figures (for profiling their launches)")
    ap.add_argument("--stream-only", action="store_true",
                    help="time only the streaming-read probe")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-shape figures (single linears, small batches, 8B-class step)")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def build_step(seed, device):
    import torch

    from paper_2412_15803_amd import workloads as wl
    from paper_2412_15803_amd import wq

    plan = wl.decode_step_linears(base_seed=seed)
    lins = []
    total_bytes = 0
    for lin, ws, xs in plan:
        w = wl.weights_device(ws, lin.n, lin.k, device)
        packed = torch.empty((lin.n, lin.k // 8), dtype=torch.int32, device=device)
        scales = torch.empty((lin.n, lin.k // 32), dtype=torch.float16, device=device)
        wq.wq_pack(w, packed, scales)
        del w
        x = wl.x_device(xs, 1, lin.k, device)
        y = torch.empty((1, lin.n), dtype=torch.float16, device=device)
        lins.append((packed, scales, x, y))
        total_bytes += wl.ideal_bytes(lin.n, lin.k, 1)
    torch.cuda.synchronize()
    return plan, lins, total_bytes


def chained_step(lins):
    """The same 113 linears with every x taken from the previous linear's y
    (a slice of it), as in a real decode where each linear consumes its
    predecessor's output: every linear then depends on the one before."""
    out = []
    prev_y = None
    for packed, scales, x, y in lins:
        k = x.shape[1]
        if prev_y is not None and prev_y.shape[1] >= k:
            x = prev_y[:, :k]
        out.append((packed, scales, x, y))
        prev_y = y
    return out


def time_steps(lins, arr, steps, warmup, m=1):
    """Milliseconds per step over `steps` back-to-back wq_decode_linears
    calls after `warmup` untimed ones, from events on the launch stream."""
    import torch

    from paper_2412_15803_amd import wq

    for _ in range(warmup):
        wq.wq_decode_linears(lins, m=m, _array=arr)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(steps):
        wq.wq_decode_linears(lins, m=m, _array=arr)
    end.record()
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def step_graph(lins, arr, m=1, per_graph=10):
    """A HIP graph of `per_graph` wq_decode_linears calls of the step on a
    side stream.  The call is made once on that stream first, so its plan is
    resident and the graph holds only the kernel launches; one replay is
    checked bit for bit against that eager call.  Returns (graph, calls)."""
    import torch

    from paper_2412_15803_amd import wq

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        wq.wq_decode_linears(lins, m=m, _array=arr, stream=s)
    s.synchronize()
    eager = [y.clone() for *_, y in lins]
    for *_, y in lins:
        y.fill_(float("nan"))
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        for _ in range(per_graph):
            wq.wq_decode_linears(lins, m=m, _array=arr, stream=s)
    graph.replay()
    torch.cuda.synchronize()
    for (*_, y), ref in zip(lins, eager):
        if not torch.equal(y.view(torch.int16), ref.view(torch.int16)):
            raise RuntimeError("graph replay of the decode step differs from the eager call")
    return graph, per_graph


def step_spread(lins, arr, steps, rounds=5):
    """Five rounds, each one eager run of `steps` back-to-back calls and one
    run of the same number of calls replayed from a HIP graph, alternated so
    that neither form gets the cooler start: per-step times (ms) of both."""
    import torch

    from paper_2412_15803_amd import wq

    graph, per = step_graph(lins, arr)
    reps = max(1, steps // per)
    eager, replay = [], []
    for _ in range(rounds):
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            wq.wq_decode_linears(lins, _array=arr)
        e.record()
        torch.cuda.synchronize()
        eager.append(a.elapsed_time(e) / steps)
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            graph.replay()
        e.record()
        torch.cuda.synchronize()
        replay.append(a.elapsed_time(e) / (reps * per))
    del graph
    return eager, replay


def _spread(ms_list, nbytes):
    v = sorted(ms_list)
    med = v[len(v) // 2]
    return {"runs": len(v), "us_median": round(med * 1e3, 2), "us_range": [round(v[0] * 1e3, 2), round(v[-1] * 1e3, 2)],
            "GB_s_median": round(nbytes / (med * 1e-3) / 1e9, 1)}


def cpu_model():
    """The host CPU's model name from /proc/cpuinfo (or the platform's)."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.lower().startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def blas_threads():
    """NumPy's BLAS library and its thread count (threadpoolctl, else the
    usual environment variables)."""
    try:
        from threadpoolctl import threadpool_info

        info = [d for d in threadpool_info() if d.get("user_api") == "blas"]
        if info:
            return {"library": info[0].get("internal_api"), "threads": info[0].get("num_threads")}
    except Exception:
        pass
    for var in ("OPENBLAS_NUM_THREADS", "OMP_NUM_THREADS", "MKL_NUM_THREADS"):
        if os.environ.get(var):
            return {"library": None, "threads": int(os.environ[var]), "from": var}
    return {"library": None, "threads": None}


def cpu_baseline(seed, budget_s):
    """The oracle GEMV (as it stands) on a bounded prefix of the same step:
    layer 0's four linears and the lm_head first, then further layers until
    the time budget is spent.  Inputs are random packed words and scales of
    the same shapes (the GEMV's cost does not depend on the values)."""
    import numpy as np

    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import oracle
    from paper_2412_15803_amd import workloads as wl

    plan = wl.decode_step_linears(base_seed=seed)
    order = plan[:4] + [plan[-1]] + plan[4:-1]
    done_bytes = 0
    done = []
    t_total = 0.0
    for lin, ws, xs in order:
        p = wl.random_words_host(ws, lin.n, lin.k)
        s = wl.random_scales_host(ws + 1, lin.n, lin.k)
        x = wl.x_host(xs, 1, lin.k)
        t0 = time.perf_counter()
        oracle.gemv(p, s, x, lin.n, lin.k)
        t_total += time.perf_counter() - t0
        done_bytes += wl.ideal_bytes(lin.n, lin.k, 1)
        done.append(lin.name)
        if t_total >= budget_s and len(done) >= 5:
            break
    threaded = cpu_baseline_threads(order, budget_s / 2)
    return {
        "value": round(done_bytes / t_total / 1e9, 4),
        "unit": "GB/s",
        "cores": 1,
        "kind": "oracle",
        "all_cores": threaded,
        "cpu_model": cpu_model(),
        "cores_available": len(os.sched_getaffinity(0)),
        "blas": blas_threads(),
        "sample": f"{len(done)} of 113 linears of the same step ({done[0]} .. {done[-1]}, incl. lm_head), "
                  f"{done_bytes / 1e9:.3f} GB in {t_total:.1f} s; NumPy elementwise + fp64 sums (the oracle's "
                  f"GEMV uses no BLAS call), one thread, baseline not target",
    }


def cpu_baseline_threads(order, budget_s):
    """The same oracle calls spread over one thread per available core
    (NumPy releases the interpreter lock inside its array loops): the linears
    of the same step in order, until the wall-clock budget is spent."""
    import concurrent.futures as cf

    sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
    import oracle
    from paper_2412_15803_amd import workloads as wl

    cores = len(os.sched_getaffinity(0))

    def make(item):
        lin, ws, xs = item
        return (wl.random_words_host(ws, lin.n, lin.k), wl.random_scales_host(ws + 1, lin.n, lin.k),
                wl.x_host(xs, 1, lin.k), lin.n, lin.k)

    def run(args):
        oracle.gemv(*args)
        return wl.ideal_bytes(args[3], args[4], 1)

    done_bytes, done, t_wall = 0, 0, 0.0
    with cf.ThreadPoolExecutor(max_workers=cores) as pool:
        i = 0
        while i < len(order) and t_wall < budget_s:
            batch = list(pool.map(make, order[i:i + cores]))  # inputs are not timed
            t0 = time.perf_counter()
            done_bytes += sum(pool.map(run, batch))
            t_wall += time.perf_counter() - t0
            done += len(batch)
            i += cores
            del batch
    return {
        "value": round(done_bytes / t_wall / 1e9, 4),
        "unit": "GB/s",
        "cores": cores,
        "sample": f"{done} of 113 linears of the same step, {cores} concurrent calls at a time on one thread "
                  f"each, {done_bytes / 1e9:.3f} GB in {t_wall:.1f} s wall",
    }


def random_linear(n, k, gen, device):
    """Random packed codes and scales of one linear (timing inputs: the GEMV's
    cost does not depend on the values)."""
    import torch

    p = torch.randint(-2**31, 2**31 - 1, (n, k // 8), dtype=torch.int32, device=device, generator=gen)
    s = (torch.rand((n, k // 32), device=device, generator=gen) * 0.01 + 0.001).to(torch.float16)
    return p, s


def time_gemv_rotated(n, k, ms_list, gen, device, calls=200, reps=5):
    """Per-call time of wq_gemv on one shape, cold: the calls rotate over
    copies of the weights totalling >= 1 GiB (4x the 256 MB last-level cache)
    and are replayed from a HIP graph, so host launch cost is not counted.
    Returns {M: (us per call, GB/s)} for each M in ms_list."""
    import torch

    from paper_2412_15803_amd import workloads as wl
    from paper_2412_15803_amd import wq

    per = wl.ideal_bytes(n, k, 1)
    r = max(1, -(-(1 << 30) // per))
    ws = [random_linear(n, k, gen, device) for _ in range(r)]
    out = {}
    for m in ms_list:
        x = torch.randn((m, k), device=device, generator=gen).to(torch.float16)
        y = torch.empty((m, n), dtype=torch.float16, device=device)
        side = torch.cuda.Stream(device)
        side.wait_stream(torch.cuda.current_stream(device))
        with torch.cuda.stream(side):
            for i in range(3):
                wq.wq_gemv(*ws[i % r], x, y)
        torch.cuda.current_stream(device).wait_stream(side)
        torch.cuda.synchronize()
        eager = y.clone()
        wq.wq_gemv(*ws[(calls - 1) % r], x, eager)
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(calls):
                wq.wq_gemv(*ws[i % r], x, y)
        times = []
        for _ in range(reps):
            a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            graph.replay()
            e.record()
            torch.cuda.synchronize()
            times.append(a.elapsed_time(e) / calls)
            if not torch.equal(y, eager):
                raise RuntimeError(f"graph replay of wq_gemv {n}x{k} M={m} differs from the eager call")
        ms = sorted(times)[len(times) // 2]
        out[m] = (round(ms * 1e3, 2), round(wl.ideal_bytes(n, k, m) / (ms * 1e-3) / 1e9, 1))
        del graph
    del ws
    torch.cuda.empty_cache()
    return out


def stream_read_ceiling(device, gib=2, calls=10, reps=5):
    """GB/s of the library's plain streaming-read probe (wq_stream_read) over
    a `gib` GiB buffer (8x the 256 MB last-level cache): events around
    `calls` back-to-back reads, median and range of `reps` such runs."""
    import torch

    from paper_2412_15803_amd import wq

    buf = torch.ones(gib << 28, dtype=torch.int32, device=device)
    sink = torch.zeros(1024, dtype=torch.int32, device=device)
    nbytes = buf.numel() * 4
    wq.stream_read(buf, sink)
    torch.cuda.synchronize()
    rates = []
    for _ in range(reps):
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(calls):
            wq.stream_read(buf, sink)
        e.record()
        torch.cuda.synchronize()
        rates.append(nbytes * calls / (a.elapsed_time(e) * 1e-3) / 1e9)
    del buf, sink
    torch.cuda.empty_cache()
    rates.sort()
    med = rates[len(rates) // 2]
    return {"kernel": "stream_read_kernel (wq_stream_read)", "bytes": nbytes, "GB_s_median": round(med, 1),
            "GB_s_range": [round(rates[0], 1), round(rates[-1], 1)], "frac_of_peak": round(med / HBM_PEAK_GBS, 4),
            "method": f"{calls} back-to-back reads of a {gib} GiB buffer per run, {reps} runs"}


def time_layer_calls(shapes, gen, device, calls=200, reps=5):
    """One decode layer's linears (independent, as BASELINE-style per-layer
    configs give them) as ONE wq_decode_linears call, cold: the calls rotate
    over >= 1 GiB of copies of the layer's weights (one descriptor list per
    copy, each plan made resident by an eager pass first) and are replayed
    from a HIP graph, so host launch cost is not counted."""
    import torch

    from paper_2412_15803_amd import workloads as wl
    from paper_2412_15803_amd import wq

    per = sum(wl.ideal_bytes(n, k, 1) for n, k in shapes)
    r = max(1, -(-(1 << 30) // per))
    copies = []
    for _ in range(r):
        lins = []
        for n, k in shapes:
            p, sc = random_linear(n, k, gen, device)
            x = torch.randn((1, k), device=device, generator=gen).to(torch.float16)
            lins.append((p, sc, x, torch.empty((1, n), dtype=torch.float16, device=device)))
        copies.append((lins, wq.make_linear_array(lins, 1)))
    s = torch.cuda.Stream(device)
    s.wait_stream(torch.cuda.current_stream(device))
    with torch.cuda.stream(s):
        for lins, arr in copies:
            wq.wq_decode_linears(lins, m=1, _array=arr, stream=s)
    s.synchronize()
    ref = [y.clone() for lins, _ in copies for *_, y in lins]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        for i in range(calls):
            lins, arr = copies[i % r]
            wq.wq_decode_linears(lins, m=1, _array=arr, stream=s)
    times = []
    for _ in range(reps):
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        graph.replay()
        e.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(e) / calls)
    got = [y for lins, _ in copies for *_, y in lins]
    if not all(torch.equal(g, t) for g, t in zip(got, ref)):
        raise RuntimeError("graph replay of the layer calls differs from the eager calls")
    del graph, copies, ref, got
    torch.cuda.empty_cache()
    times.sort()
    ms = times[len(times) // 2]
    gbs = per / (ms * 1e-3) / 1e9
    return {"us": round(ms * 1e3, 2), "us_range": [round(times[0] * 1e3, 2), round(times[-1] * 1e3, 2)],
            "GB_s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4), "bytes": per, "copies": r}


def layer_configs(device, seed):
    """The 3B- and 8B-class layers (qkv, o, gate_up, down) at batch 1, each
    as one wq_decode_linears call per layer."""
    import torch

    from paper_2412_15803_amd import workloads as wl

    gen = torch.Generator(device=device)
    gen.manual_seed(seed + 11)
    res = {"method": "one wq_decode_linears call per layer (its four linears in one launch), rotated over >= 1 GiB "
                     "of layer copies, replayed from a HIP graph; median of 5 runs of 200 calls"}
    for label, layer in (("3B layer", wl.LLAMA3B_LAYER), ("8B layer", wl.LLAMA8B_LAYER)):
        shapes = [(lin.n, lin.k) for lin in layer]
        res[f"{label} " + ", ".join(f"{lin.name} {lin.n}x{lin.k}" for lin in layer)] = time_layer_calls(shapes, gen,
                                                                                                         device)
    return res


def time_step_batches(shapes, batches, gen, device, steps, warmup):
    """One decode step of the given linear shapes (random codes), timed as one
    wq_decode_linears call per step at each batch size M."""
    import torch

    from paper_2412_15803_amd import workloads as wl
    from paper_2412_15803_amd import wq

    ws = [random_linear(n, k, gen, device) for n, k in shapes]
    out = {}
    for m in batches:
        lins, total = [], 0
        for (n, k), (p, s) in zip(shapes, ws):
            x = torch.randn((m, k), device=device, generator=gen).to(torch.float16)
            lins.append((p, s, x, torch.empty((m, n), dtype=torch.float16, device=device)))
            total += wl.ideal_bytes(n, k, m)
        ms = time_steps(lins, wq.make_linear_array(lins, m), steps, warmup, m=m)
        gbs = total / (ms * 1e-3) / 1e9
        out[m] = {"us": round(ms * 1e3, 2), "GB_s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4),
                  "tokens_per_s": round(m / (ms * 1e-3), 1)}
        del lins
    del ws
    torch.cuda.empty_cache()
    return out


def time_pack(n, k, gen, device, calls=10):
    """wq_pack of an fp32 W[n][k] already on the device: us per call and GB/s
    of its bytes (4 read + 0.5625 written per weight)."""
    import torch

    from paper_2412_15803_amd import wq

    w = torch.randn((n, k), device=device, generator=gen).mul_(0.02)
    packed = torch.empty((n, k // 8), dtype=torch.int32, device=device)
    scales = torch.empty((n, k // 32), dtype=torch.float16, device=device)
    wq.wq_pack(w, packed, scales)
    torch.cuda.synchronize()
    a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(calls):
        wq.wq_pack(w, packed, scales)
    e.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(e) / calls
    nbytes = n * k * 4 + n * k // 2 + n * (k // 32) * 2
    del w, packed, scales
    torch.cuda.empty_cache()
    return [round(ms * 1e3, 2), round(nbytes / (ms * 1e-3) / 1e9, 1)]


def time_attention_rotated(hq, hkv, lens, page, seed, device, calls=256, reps=5, eager=False):
    """Per-call time of wq_paged_attention, cold: the calls rotate over
    per-layer caches totalling >= 1 GiB (each layer's K and V arrays hold the
    same sequences under one shared block table, as in a decode step) and are
    replayed from a HIP graph.  Returns (us per call, GB/s, bytes per call)."""
    import torch

    from paper_2412_15803_amd import attn_workloads as aw
    from paper_2412_15803_amd import wq

    per = aw.attention_bytes(lens, hq, hkv, aw.HEAD_DIM, page)
    r = max(1, -(-(1 << 30) // per))
    need = aw.pages_needed(lens, page)
    k_all, v_all = aw.kv_cache_device(seed, r * need, hkv, page, aw.HEAD_DIM, device=device)
    layers = [(k_all[i * need:(i + 1) * need], v_all[i * need:(i + 1) * need]) for i in range(r)]
    table_np, _ = aw.block_table_host(seed + 1, lens, page)
    table = torch.from_numpy(table_np).to(device)
    lens_t = torch.tensor(lens, dtype=torch.int32, device=device)
    q = aw.q_device(seed + 2, len(lens), hq, aw.HEAD_DIM, device=device)
    out = torch.empty_like(q)
    ml = max(lens)
    ws = wq.paged_workspace(q, ml, hkv)
    scale = aw.default_scale(aw.HEAD_DIM)

    def call(i, dst):
        k, v = layers[i % r]
        wq.paged_attention(q, k, v, table, lens_t, dst, scale, ml, workspace=ws)

    side = torch.cuda.Stream(device)
    side.wait_stream(torch.cuda.current_stream(device))
    with torch.cuda.stream(side):
        for i in range(3):
            call(i, out)
    torch.cuda.current_stream(device).wait_stream(side)
    torch.cuda.synchronize()
    ref = torch.empty_like(out)
    call(calls - 1, ref)
    graph = None
    if not eager:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(calls):
                call(i, out)
    times = []
    for _ in range(reps):
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        if graph is not None:
            graph.replay()
        else:
            for i in range(calls):
                call(i, out)
        e.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(e) / calls)
        if not torch.equal(out, ref):
            raise RuntimeError(f"repeated wq_paged_attention {lens[:2]} differs from the first call")
    ms = sorted(times)[len(times) // 2]
    del graph, layers, k_all, v_all
    torch.cuda.empty_cache()
    return round(ms * 1e3, 2), round(per / (ms * 1e-3) / 1e9, 1), per


def time_dependent_step(lins, device, seed, ctx=4096, steps=20, reps=3, graph=True, persistent=False):
    """The 3B-class step as one token's dependent chain (batch 1), reusing the
    step's packed weights: per layer RMSNorm -> qkv, attention of the 24
    query heads (q = the first 3072 qkv outputs) over a paged cache of `ctx`
    tokens, O + residual, RMSNorm -> gate_up, SiLU-mul -> down + residual;
    then RMSNorm -> lm_head and argmax.  With ctx = 0 the attention is left
    out (O reads the first 3072 qkv outputs) and the 113 linears run as one
    wq_fused_linears call.  The step is replayed from one HIP graph, its
    residual stream reset at the start of every replay; every replay must
    reproduce the eager step's logits and token.

    Returns {us per token, tokens/s, GB/s and fraction of the HBM peak over
    the weights (and cached keys and values) read once per token}."""
    import torch

    from paper_2412_15803_amd import attn_workloads as aw
    from paper_2412_15803_amd import workloads as wl
    from paper_2412_15803_amd import wq

    hid, layers = 3072, wl.LLAMA3B_LAYERS
    gen = torch.Generator(device=device)
    gen.manual_seed(seed + 77)

    def vec(n, lo=None):
        t = torch.rand(n, generator=gen, device=device) + 0.5 if lo else torch.randn(n, generator=gen, device=device)
        return t.to(torch.float16)

    h0, h = vec(hid), torch.empty(hid, dtype=torch.float16, device=device)
    qkv = torch.empty(5120, dtype=torch.float16, device=device)
    attn = torch.empty(hid, dtype=torch.float16, device=device)
    gu = torch.empty(16384, dtype=torch.float16, device=device)
    logits = torch.empty(128256, dtype=torch.float16, device=device)
    token = torch.empty(1, dtype=torch.int32, device=device)
    norm1 = [vec(hid, True) for _ in range(layers)]
    norm2 = [vec(hid, True) for _ in range(layers)]
    norm_f = vec(hid, True)
    eps = 1e-5

    def lin(i, x, y, **kw):
        p, sc = lins[i][0], lins[i][1]
        return dict(packed_w=p, scales=sc, x=x, y=y, eps=eps, **kw)

    R, S = wq.PROLOGUE_RMSNORM, wq.PROLOGUE_SILU_MUL
    per_layer = []
    for l in range(layers):
        b = 4 * l
        qkv_lin = lin(b, h, qkv, prologue=R, norm_weight=norm1[l])
        rest = [lin(b + 1, attn if ctx else qkv[:hid], h, residual=h),
                lin(b + 2, h, gu, prologue=R, norm_weight=norm2[l]),
                lin(b + 3, gu, h, prologue=S, residual=h)]
        per_layer.append((qkv_lin, rest))
    head = lin(4 * layers, h, logits, prologue=R, norm_weight=norm_f)

    step_bytes = sum(wl.ideal_bytes(p.shape[0], p.shape[1] * 8, 1) for p, _, _, _ in lins)
    if ctx:
        need = aw.pages_needed((ctx,), 16)
        k_all, v_all = aw.kv_cache_device(seed + 78, layers * need, 8, 16, aw.HEAD_DIM, device=device)
        caches = [(k_all[i * need:(i + 1) * need], v_all[i * need:(i + 1) * need]) for i in range(layers)]
        table_np, _ = aw.block_table_host(seed + 79, (ctx,), 16)
        table = torch.from_numpy(table_np).to(device)
        lens = torch.tensor([ctx], dtype=torch.int32, device=device)
        ws = wq.paged_workspace(qkv[:hid].view(1, 24, aw.HEAD_DIM), ctx, 8)
        scale = aw.default_scale(aw.HEAD_DIM)
        arrays = [(wq.make_fused_array([a]), wq.make_fused_array(r)) for a, r in per_layer]
        head_arr = wq.make_fused_array([head])
        step_bytes += layers * aw.attention_bytes((ctx,), 24, 8, aw.HEAD_DIM, 16)

        def step():
            h.copy_(h0)
            for l in range(layers):
                wq.wq_fused_linears([per_layer[l][0]], _array=arrays[l][0])
                k, v = caches[l]
                wq.paged_attention(qkv[:hid].view(1, 24, aw.HEAD_DIM), k, v, table, lens,
                                   attn.view(1, 24, aw.HEAD_DIM), scale, ctx, workspace=ws)
                wq.wq_fused_linears(per_layer[l][1], _array=arrays[l][1])
            wq.wq_fused_linears([head], argmax=token, _array=head_arr)
    else:
        chain = [d for a, r in per_layer for d in [a] + r] + [head]
        chain_arr = wq.make_fused_array(chain)

        def step():
            h.copy_(h0)
            wq.wq_fused_linears(chain, argmax=token, _array=chain_arr)

    old_env = os.environ.get("WQ_FUSED_PERSISTENT")
    os.environ["WQ_FUSED_PERSISTENT"] = "1" if persistent else "0"
    side = torch.cuda.Stream(device)
    side.wait_stream(torch.cuda.current_stream(device))
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream(device).wait_stream(side)
    torch.cuda.synchronize()
    wq.wq_fused_check()
    ref_logits, ref_token = logits.clone(), int(token.item())
    g = None
    if graph:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            step()
    times = []
    for _ in range(reps):
        a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            if g is not None:
                g.replay()
            else:
                step()
        e.record()
        torch.cuda.synchronize()
        times.append(a.elapsed_time(e) / steps)
        if int(token.item()) != ref_token or not torch.equal(logits, ref_logits):
            raise RuntimeError("repeated dependent step differs from the first one")
    wq.wq_fused_check()
    if old_env is None:
        os.environ.pop("WQ_FUSED_PERSISTENT", None)
    else:
        os.environ["WQ_FUSED_PERSISTENT"] = old_env
    ms = sorted(times)[len(times) // 2]
    del g
    torch.cuda.empty_cache()
    gbs = step_bytes / (ms * 1e-3) / 1e9
    return {"us_per_token": round(ms * 1e3, 1), "tokens_per_s": round(1e3 / ms, 1), "GB_s": round(gbs, 1),
            "frac": round(gbs / HBM_PEAK_GBS, 4), "bytes_per_token": step_bytes, "token": ref_token,
            "finite_logits": bool(torch.isfinite(ref_logits).all().item())}


MFMA_F16_PEAK_TFLOPS = 2500.0  # MI355X dense fp16 matrix-core peak

PREFILL_CONFIGS = (
    # (label, N, K, M): prompt-sized batches of one linear
    ("3B gate_up 16384x3072, M=2048 prompt tokens", 16384, 3072, 2048),
    ("3B down 3072x8192, M=2048", 3072, 8192, 2048),
    ("3B lm_head 128256x3072, M=2048", 128256, 3072, 2048),
    ("8B gate_up 28672x4096, M=512", 28672, 4096, 512),
)


def time_prefill(n, k, m, gen, device, reps=10):
    """wq_gemv on M rows of x (the tiled matrix-core kernel): device time per
    call from events around `reps` back-to-back calls."""
    import torch

    from paper_2412_15803_amd import wq

    packed, scales = random_linear(n, k, gen, device)
    x = torch.randn((m, k), generator=gen, device=device).to(torch.float16)
    y = torch.empty((m, n), dtype=torch.float16, device=device)
    for _ in range(2):
        wq.wq_gemv(packed, scales, x, y)
    torch.cuda.synchronize()
    a, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        wq.wq_gemv(packed, scales, x, y)
    e.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(e) / reps
    tflops = 2.0 * m * n * k / (ms * 1e-3) / 1e12
    del packed, scales, x, y
    torch.cuda.empty_cache()
    return {"us": round(ms * 1e3, 1), "TFLOP_s": round(tflops, 1), "frac": round(tflops / MFMA_F16_PEAK_TFLOPS, 4)}


def prefill_configs(device, seed, only=None):
    """Prompt processing (M > 64 rows of x): the tiled fp16 matrix-core GEMM
    with the 4-bit weights dequantized per tile; TFLOP/s and the fraction of
    the dense fp16 matrix-core peak.  Also the whole 3B-class step's 113
    linears over a 2048-token prompt."""
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(seed + 31)
    res = {"method": "wq_gemv / wq_decode_linears with M prompt rows, random codes and scales, device time from "
                     "events around back-to-back calls; flops = 2 M N K", "peak_TFLOP_s": MFMA_F16_PEAK_TFLOPS}
    for i, (label, n, k, m) in enumerate(PREFILL_CONFIGS):
        if only is not None and i != only:
            continue
        res[label] = time_prefill(n, k, m, gen, device)
    if only is None:
        from paper_2412_15803_amd import workloads as wl

        m = 2048
        steps3 = [(lin.n, lin.k) for lin in wl.LLAMA3B_LAYER] * 28 + [(wl.LLAMA3B_LM_HEAD.n, wl.LLAMA3B_LM_HEAD.k)]
        flops = sum(2.0 * m * n * k for n, k in steps3)
        got = time_step_batches(steps3, [m], gen, device, 3, 1)[m]
        tflops = flops / (got["us"] * 1e-6) / 1e12
        res["3B step, 113 linears, M=2048 prompt tokens (one wq_decode_linears call)"] = {
            "us": got["us"], "prompt_tokens_per_s": got["tokens_per_s"], "TFLOP_s": round(tflops, 1),
            "frac": round(tflops / MFMA_F16_PEAK_TFLOPS, 4)}
    return res


# Counter summaries of the split kernel, by ATTN_CONFIGS index.
ATTN_PROFILES = {0: "paged_attention_3b_ctx4096.md", 1: "paged_attention_3b_ctx32768.md"}
ATTN_SOURCES = ("wq_attention.hip", "wq_device.h")


def attention_traffic(index):
    """HBM bytes per split-kernel launch from the committed counter summary of
    this attention shape, or None (no summary, or the kernel changed since)."""
    from paper_2412_15803_amd.build import source_hash
    from paper_2412_15803_amd.profsum import parse_traffic

    name = ATTN_PROFILES.get(index)
    got = parse_traffic(os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", name)) if name else None
    if not got or got[0] != source_hash(ATTN_SOURCES):
        return None
    return int(got[1])


ATTN_CONFIGS = (
    # (label, query heads, kv heads, sequence lengths); pages of 16 tokens
    ("3B attention, 1 sequence of 4096 tokens", 24, 8, (4096,)),
    ("3B attention, 1 sequence of 32768 tokens", 24, 8, (32768,)),
    ("3B attention, 16 sequences of 4096 tokens", 24, 8, (4096,) * 16),
    ("8B attention, 1 sequence of 4096 tokens", 32, 8, (4096,)),
    ("8B attention, 1 sequence of 32768 tokens", 32, 8, (32768,)),
)


def attention_configs(device, seed, only=None, eager=False):
    """Decode attention over a paged cache (24 or 32 query heads, 8 kv heads
    of 128, pages of 16 tokens): device time per call, GB/s of cached keys
    and values (plus q, out, table) and the fraction of the HBM peak."""
    how = "launched one by one from the host" if eager else "replayed from a HIP graph (device time per call)"
    res = {"method": "wq_paged_attention calls (split and merge kernels) rotated over >= 1 GiB of per-layer "
                     f"caches sharing one block table, {how}"}
    for i, (label, hq, hkv, lens) in enumerate(ATTN_CONFIGS):
        if only is not None and i != only:
            continue
        us, gbs, per = time_attention_rotated(hq, hkv, lens, 16, seed + 100 + i, device, eager=eager)
        res[label] = {"us": us, "GB_s": gbs, "frac": round(gbs / HBM_PEAK_GBS, 4), "bytes": per,
                      "split_kernel_traffic": attention_traffic(i)}
    return res


def per_config(device, seed):
    """Per-shape figures beside the headline step (the 512 x 512 parity shape,
    the 3B- and 8B-class single linears, small batches, the 8B-class step,
    attention and prefill); none of them is the bench value."""
    import torch

    from paper_2412_15803_amd import workloads as wl

    gen = torch.Generator(device=device)
    gen.manual_seed(seed + 7)
    res = {"method": "single wq_gemv calls rotated over >= 1 GiB of weight copies, replayed from a HIP graph "
                     "(device time per call, host launch excluded); random codes and scales of each shape"}
    res["512x512 M=1"] = time_gemv_rotated(512, 512, [1], gen, device)[1]
    res["wq_pack 8B gate_up 28672x4096 (fp32 in, codes + scales out)"] = time_pack(28672, 4096, gen, device)
    for lin in wl.LLAMA3B_LAYER + (wl.LLAMA3B_LM_HEAD,):
        res[f"3B {lin.name} {lin.n}x{lin.k} M=1"] = time_gemv_rotated(lin.n, lin.k, [1], gen, device)[1]
    for lin in wl.LLAMA8B_LAYER:
        got = time_gemv_rotated(lin.n, lin.k, [1, 4, 8, 16], gen, device)
        for m, v in got.items():
            res[f"8B {lin.name} {lin.n}x{lin.k} M={m}"] = v
    res["unit"] = "[us per call, GB/s]"
    steps3 = [(lin.n, lin.k) for lin in wl.LLAMA3B_LAYER] * 28 + [(wl.LLAMA3B_LM_HEAD.n, wl.LLAMA3B_LM_HEAD.k)]
    steps8 = [(lin.n, lin.k) for lin in wl.LLAMA8B_LAYER] * 32 + [(128256, 4096)]
    for m, v in time_step_batches(steps3, [4, 8, 16], gen, device, 20, 3).items():
        res[f"3B step M={m} (one wq_decode_linears call, 113 linears)"] = v
    for m, v in time_step_batches(steps8, [1, 4, 8, 16], gen, device, 20, 3).items():
        res[f"8B step M={m} (one wq_decode_linears call, 129 linears)"] = v
    res["paged decode attention"] = attention_configs(device, seed)
    res["prefill"] = prefill_configs(device, seed)
    return res


def profiled_step():
    """The committed rocprofv3 summary of the step kernel: HBM bytes per
    launch and its trace statistics, or None when the kernel's sources have
    changed since it was taken."""
    from paper_2412_15803_amd.build import source_hash
    from paper_2412_15803_amd.profsum import parse_summary

    got = parse_summary(STEP_PROFILE)
    if got is None or got.get("source_hash") != source_hash():
        return None
    out = {"summary": os.path.relpath(STEP_PROFILE, ROOT), "traffic": float(got["traffic_bytes_per_launch"])}
    for key in ("median_duration_us", "avg_duration_us", "launches_summarised"):
        if key in got:
            out[key] = float(got[key])
    return out


def copy_probe(mib, device):
    import torch

    n = mib * (1 << 20) // 4
    a = torch.ones(n, dtype=torch.float32, device=device)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    log(f"copy probe: {mib} MiB read + {mib} MiB written")


def main():
    args = parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures the single-GPU decode linears only; runs on more than one GPU are not "
              "part of this build (use --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2412_15803_amd import wq

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    device = torch.device("cuda:0")
    wq.lib()  # fail loudly if the HIP library is missing

    if args.prefill_only:
        if args.copy_probe_mib:
            copy_probe(args.copy_probe_mib, device)
        log("timing the prefill GEMM shapes")
        print(json.dumps({"prefill": prefill_configs(device, args.seed, args.prefill_config)}), flush=True)
        return

    if args.step_batches:
        from paper_2412_15803_amd import workloads as wl

        if args.copy_probe_mib:
            copy_probe(args.copy_probe_mib, device)

        ms = [int(v) for v in args.step_batches.split(",")]
        log(f"timing the 3B-class step at M = {ms}")
        gen = torch.Generator(device=device)
        gen.manual_seed(args.seed + 7)
        steps3 = [(lin.n, lin.k) for lin in wl.LLAMA3B_LAYER] * 28 + [(wl.LLAMA3B_LM_HEAD.n, wl.LLAMA3B_LM_HEAD.k)]
        res = time_step_batches(steps3, ms, gen, device, args.steps, args.warmup)
        print(json.dumps({"3B step batches": res}), flush=True)
        return

    if args.layers_only:
        log("timing one wq_decode_linears call per layer")
        print(json.dumps({"layer_calls": layer_configs(device, args.seed)}), flush=True)
        return

    if args.stream_only:
        log("timing the streaming-read probe")
        print(json.dumps({"stream_read_ceiling": stream_read_ceiling(device)}), flush=True)
        return

    if args.attention_only:
        if args.copy_probe_mib:
            copy_probe(args.copy_probe_mib, device)
        log("timing the paged decode-attention shapes")
        res = attention_configs(device, args.seed, args.attention_config, args.attention_eager)
        print(json.dumps({"paged decode attention": res}), flush=True)
        return

    log("building the 3B-class decode step (113 linears) on the device")
    plan, lins, step_bytes = build_step(args.seed, device)
    if args.dependent_only:
        if args.copy_probe_mib:
            copy_probe(args.copy_probe_mib, device)
        log(f"timing the dependent decode step ({args.dependent_ctx} cached tokens per layer)")
        res = time_dependent_step(lins, device, args.seed, ctx=args.dependent_ctx, steps=args.steps, reps=3,
                                  graph=not args.dependent_eager, persistent=args.dependent_eager)
        print(json.dumps({"dependent_decode_step": res}), flush=True)
        return
    arr = wq.make_linear_array(lins, 1)

    if args.copy_probe_mib:
        copy_probe(args.copy_probe_mib, device)

    log(f"timing {args.steps} steps after {args.warmup} warmup steps")
    # One grouped launch per step: the events on the launch stream around K
    # back-to-back launches give the kernel's average duration.
    ms_per_step = time_steps(lins, arr, args.steps, args.warmup)
    gbs = step_bytes / (ms_per_step * 1e-3) / 1e9
    # Spread: five more runs of K eager calls, alternated with five runs of K
    # calls replayed from a HIP graph.
    eager_runs, graph_runs = step_spread(lins, arr, args.steps)
    spread = {"eager": _spread(eager_runs, step_bytes), "graph": _spread(graph_runs, step_bytes)}
    ms_graph = sorted(graph_runs)[len(graph_runs) // 2]


    ms_chained = None
    if args.chained:
        chained = chained_step(lins)
        ms_chained = time_steps(chained, wq.make_linear_array(chained, 1), args.steps, args.warmup)

    prof = profiled_step()
    roofline = {
        "bound": "hbm",
        "achieved": round(gbs, 1),
        "peak": HBM_PEAK_GBS,
        "unit": "GB/s",
        "frac": round(gbs / HBM_PEAK_GBS, 4),
        "traffic": prof["traffic"] if prof else None,
        "kernel": f"grouped_m1_kernel, one launch per step: {ms_per_step * 1e3:.2f} us per launch, the average over "
                  f"the {args.steps} timed launches from HIP events on the launch stream; "
                  f"{step_bytes / 1e6:.2f} MB algorithmic per launch",
        "profile": prof,
    }

    log("timing the streaming-read probe (achievable-bandwidth context)")
    ceiling = stream_read_ceiling(device)

    log("timing the 3B- and 8B-class layers as one call per layer")
    layers = layer_configs(device, args.seed)

    dependent = None
    if not args.no_configs:
        log("timing the dependent decode step (fused linears and paged attention)")
        dependent = {
            "method": "one token's dependent layer chain (batch 1) with the step's weights; per-linear: one "
                      "launch per linear, replayed from a HIP graph; persistent chain: one cooperative launch of the "
                      "persistent kernel per wq_fused_linears call, launched from the host",
            "linears only, per-linear launches (graph replay; 113 fused linears, one wq_fused_linears call)":
                time_dependent_step(lins, device, args.seed, ctx=0),
            "linears only, persistent chain (WQ_FUSED_PERSISTENT=1, launched from the host)":
                time_dependent_step(lins, device, args.seed, ctx=0, graph=False, persistent=True),
            "with attention over 4096 cached tokens per layer, per-linear launches (graph replay)":
                time_dependent_step(lins, device, args.seed, ctx=4096),
        }

    configs = None
    if not args.no_configs:
        log("timing the per-shape figures (single linears, small batches, 8B-class step)")
        configs = per_config(device, args.seed)

    cpu = None
    if not args.no_cpu_baseline:
        log(f"timing the CPU oracle (~{args.cpu_seconds:.0f} s sample)")
        cpu = cpu_baseline(args.seed, args.cpu_seconds)

    out = {
        "metric": METRIC,
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "us_per_step": round(ms_per_step * 1e3, 2),
        "frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
        "tokens_per_s_upper_bound": round(1e3 / ms_per_step, 1),
        "step_runs": spread,
        "graph_us_per_step": round(ms_graph * 1e3, 2),  # median of the graph runs
        "stream_read_ceiling": ceiling,
        "layer_calls": layers,
        "chained_us_per_step": round(ms_chained * 1e3, 2) if ms_chained else None,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": "3B-class decode step, batch 1: 28 x (qkv 5120x3072, o 3072x3072, gate_up 16384x3072, "
                        "down 3072x8192) + lm_head 128256x3072; int4 g32 fp16 scales; 113 linears",
            "batch_m": 1,
            "linears": len(lins),
            "bytes_per_step": step_bytes,
        },
        "roofline": roofline,
        "cpu_baseline": cpu,
        "dependent_decode_step": dependent,
        "per_config": configs,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
