#!/usr/bin/env python3
"""Benchmark of the weight-streaming read path on one MI355X.

Headline: the batch-1 decode weight sweep of a synthetic Llama-70B-shaped model in bf16 (80 layers,
d 8192, 64 q / 8 kv heads of dim 128, FFN 28672, vocab 128256; 139.0 GB of weights read per token),
fully HBM-resident; one step = one decode token = one persistent launch over every matrix.
`value` is the achieved weight-read rate in GB/s (decimal), counting each weight byte once.
The headline and q4 sweeps (and the protocol) also report the same tokens batched b per weight
pass, on the vector ALUs (bit-identical outputs) and on the matrix cores (b <= 16, within rounding).

Also measured in the same run and reported under "rows" (same JSON line):
  probe        pure-read reference, 1 GiB fp32 -> fp64 sum, HBM-resident and host-mapped
  gemv_f16     4096 x 4096 fp16 GEMV, 32 distinct matrices visited per pass (1 GiB)
  llama8b_q4   decode sweep of the Llama-3-8B shape in 4-bit blocks (4.22 GB per token)
  protocol     the matched protocol's pass: int8 GEMV with fp16 row scales over 12 matrices of
               12288 x 7168 (1.06 GB), as 12 dispatches, as the same 12 dispatches replayed from
               a HIP graph, and as one launch, plus the T-sweep
  endpoints    Alg. 2 over the same set stored as a file: map (pinned pages in place), resident and
               per-use copy (staged from the file pages) rates, and the endpoint it selects
  ordering     the protocol pass ordered against an in-flight framework stream by four mechanisms
               (in-stream, event, host-visible event, host drain): excess ms per pass
  size_sweep   bf16 GEMV with K = 4096 and N = 256 ... 140800 rows, resident and host-mapped
  bus          pinned host -> device copy rate, the ceiling of every host-mapped arm
  copy         1 GiB elementwise read+write pass (calibrates the HBM byte counters; not default)

Usage: python bench.py [--gpus 1] [--steps 16] [--warmup 2] [--rows probe,gemv_f16,...]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12   # B/s, MI355X HBM3E


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


KERNEL_SOURCES = ("paper_2608_12114_amd/csrc/wsr_device.h", "paper_2608_12114_amd/csrc/wsr_kernels.hip",
                  "paper_2608_12114_amd/csrc/wsr_internal.h", "paper_2608_12114_amd/build.py")
PROFILE_OF = {"llama70b_bf16": "k_sweep_bf16_llama70b", "llama8b_q4": "k_sweep_q4_llama8b",
              "probe": "k_probe_1gib", "gemv_f16": "k_gemv16_f16_4096x4096",
              "gemv_f16_one_launch": "k_sweep_f16_32x4096x4096", "protocol": "k_sweep_i8_protocol"}


def kernel_sources_sha256() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    return h.hexdigest()


def profiled_traffic(key):
    """HBM bytes per launch from the committed rocprofv3 counter summary (FETCH_SIZE + WRITE_SIZE,
    each scaled by the copy-kernel calibration), or None when the kernel sources changed since."""
    path = os.path.join(ROOT, "profiles", PROFILE_OF[key] + ".json")
    if not os.path.exists(path):
        return None, "no profile"
    rec = json.load(open(path))
    if rec.get("kernel_source_sha256") != kernel_sources_sha256():
        return None, "kernel changed since the counters were taken"
    return rec.get("traffic_bytes_per_launch"), os.path.relpath(path, ROOT)


def row_roofline(gbps, key, bytes_per_launch):
    """The roofline object of a row: HBM-bound, the row's own rate against the 8 TB/s peak, and the
    HBM bytes per launch its profile measured (null once the kernels changed since)."""
    traffic, src = profiled_traffic(key)
    kernel = None
    path = os.path.join(ROOT, "profiles", PROFILE_OF[key] + ".json")
    if os.path.exists(path):
        kernel = json.load(open(path)).get("kernel")
    return {"bound": "hbm", "achieved": round(gbps, 2), "peak": HBM_PEAK / 1e9, "unit": "GB/s",
            "frac": round(gbps * 1e9 / HBM_PEAK, 4), "traffic": traffic, "traffic_source": src, "kernel": kernel,
            "bytes_per_launch": bytes_per_launch}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=16, help="timed decode tokens of the headline")
    p.add_argument("--warmup", type=int, default=2, help="untimed decode tokens before timing")
    p.add_argument("--workload", default="llama70b_bf16", choices=["llama70b_bf16", "llama8b_q4"])
    p.add_argument("--rows", default="probe,gemv_f16,llama8b_q4,protocol,endpoints,ordering,size_sweep,bus",
                   help="comma list of extra rows ('' for none)")
    p.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle baselines of every row")
    p.add_argument("--no-mapped", action="store_true",
                   help="skip the host-mapped arms of the probe and the size sweep (resident-only profiles)")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="target oracle time of the sample")
    p.add_argument("--passes", type=int, default=4, help="extra timed passes for the spread")
    p.add_argument("--processes", type=int, default=0,
                   help="run the headline in this many child processes, one after another, and report "
                        "the median of their medians (a separate JSON line; no GPU use in this process)")
    return p.parse_args()


# --------------------------------------------------------------------------------------------------
# timing helpers (events on the stream the kernels are launched on)

def timed(fn, reps, stream):
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / 1e3   # seconds


def median_of(fn, reps, passes, stream):
    return float(np.median([timed(fn, reps, stream) for _ in range(passes)]))


def calls_per_region(fn, stream, target_s=3e-3, most=16):
    """Calls to time back to back per event pair so that a region lasts about target_s: a short
    pass timed alone also counts the host's time to plan and launch it."""
    t1 = timed(fn, 1, stream)
    return int(min(most, max(1, -(-target_s // t1))))


# --------------------------------------------------------------------------------------------------
# decode sweep

SWEEPS = {"llama70b_bf16": ("LLAMA_70B", "bf16"), "llama8b_q4": ("LLAMA3_8B", "q4")}


def sweep_workload(name, tokens_needed, stream, wsr, check_rows=16):
    import torch
    from synth import device as dv
    from synth import workloads as wl
    shape = getattr(wl, SWEEPS[name][0])
    fmt = SWEEPS[name][1]
    mats = wl.decode_matrices(shape)
    t0 = time.time()
    inp = dv.SweepInputs(mats, [fmt] * len(mats), tokens=tokens_needed, arena=True)
    log(f"{name}: {len(mats)} matrices, {inp.weight_bytes() / 1e9:.2f} GB generated and resident "
        f"in {time.time() - t0:.1f} s")
    specs = wsr.make_mats(inp.specs())
    ws = torch.zeros(wsr.wsr_sweep_workspace_bytes(specs), dtype=torch.uint8, device="cuda")
    return shape, fmt, mats, inp, specs, ws


def spread(ms, boot=2000, seed=0):
    """Median, interquartile range and a 95 % bootstrap interval of the median over timed passes."""
    a = np.asarray(ms, dtype=np.float64)
    rng = np.random.default_rng(seed)
    meds = np.median(a[rng.integers(0, len(a), size=(boot, len(a)))], axis=1)
    return {"n": len(a), "ms_per_token": [round(float(v), 4) for v in a],
            "median": round(float(np.median(a)), 4),
            "iqr": [round(float(np.percentile(a, 25)), 4), round(float(np.percentile(a, 75)), 4)],
            "ci95_median": [round(float(np.percentile(meds, 2.5)), 4), round(float(np.percentile(meds, 97.5)), 4)]}


def run_sweep(name, steps, warmup, stream, wsr, want_cpu, cpu_seconds, passes=4, warm_seconds=0.0):
    """warmup untimed tokens; with warm_seconds > 0 (rows other than the headline) the untimed
    sweeps go on until that much time has passed, so that a short sweep is not timed while the
    GPU's clocks still rise after the host-side checks of the previous row."""
    import torch
    from synth import workloads as wl
    shape, fmt, mats, inp, specs, ws = sweep_workload(name, max(steps, warmup, 1), stream, wsr)
    bpt = inp.weight_bytes()
    assert bpt == wl.bytes_per_token(shape, fmt)
    t0, warmed = time.perf_counter(), 0
    while warmed < warmup or time.perf_counter() - t0 < warm_seconds:
        n = max(1, min(warmup, steps)) if warmup else steps
        wsr.wsr_decode_sweep(specs, n, ws, ws.numel(), stream)
        torch.cuda.synchronize()
        warmed += n
    warmup = warmed
    torch.cuda.synchronize()
    sec = timed(lambda: wsr.wsr_decode_sweep(specs, steps, ws, ws.numel(), stream), 1, stream)
    per_tok = sec / steps
    # further timed passes of the same length, for the spread (the first pass above is the result)
    pass_ms = [per_tok * 1e3] + [timed(lambda: wsr.wsr_decode_sweep(specs, steps, ws, ws.numel(), stream), 1,
                                       stream) / steps * 1e3 for _ in range(passes)]
    gbps = bpt / per_tok / 1e9
    log(f"{name}: {steps} tokens in {sec * 1e3:.2f} ms -> {per_tok * 1e3:.3f} ms/token, "
        f"{gbps:.1f} GB/s ({gbps * 1e9 / HBM_PEAK * 100:.1f}% of 8 TB/s), {1 / per_tok:.2f} tok/s")
    parity = check_sweep(inp, [0, steps - 1])
    log(f"{name}: parity on sampled rows: worst rel-L2 {parity['worst_rel_l2']:.2e}")
    batched = batch_sweep(name, inp, specs, ws, steps, bpt, stream, wsr,
                          (1, 2, 4, 8) if fmt == wl.Q4 else (1, 2, 4, 8, 16))
    out = {"workload": name, "bytes_per_token": bpt, "footprint_bytes": wl.footprint_bytes(shape, fmt),
           "tokens_timed": steps, "warmup_tokens": warmup, "ms_per_token": per_tok * 1e3,
           "GBps": gbps, "hbm_frac": gbps * 1e9 / HBM_PEAK, "tokens_per_s": 1 / per_tok,
           "launches_per_token": 1, "parity": parity, "passes": spread(pass_ms),
           "roofline": row_roofline(gbps, name, bpt)}
    if batched is not None:
        out["batched"] = batched
    out["batched_matrix_cores"] = mma_sweep(name, inp, specs, ws, steps, bpt, stream, wsr)
    if want_cpu:
        out["cpu_baseline"] = cpu_baseline(inp, bpt, cpu_seconds)
    del specs, ws, inp
    torch.cuda.empty_cache()
    return out


def batch_sweep(name, inp, specs, ws, steps, bpt, stream, wsr, batches=(1, 2, 4, 8, 16)):
    """The same tokens with `batch` of them sharing each pass over the weights (the multi-column
    T-sweep): outputs are compared bit for bit with the token-by-token sweep."""
    import torch
    ref = [y.clone() for y in inp.y]           # the token-by-token outputs of the timed passes
    res = []
    for b in batches:
        if b > steps:
            break
        run = lambda: wsr.wsr_decode_sweep_batched(specs, steps, b, ws, ws.numel(), stream)
        run()
        torch.cuda.synchronize()
        same = all(torch.equal(a, y) for a, y in zip(ref, inp.y))
        calls = calls_per_region(run, stream)
        sec = median_of(run, calls, 3, stream) / calls
        passes = -(-steps // b)
        res.append({"batch": b, "ms_per_pass": sec / passes * 1e3, "tokens_per_s": steps / sec,
                    "hbm_GBps": passes * bpt / sec / 1e9, "logical_weight_GBps": steps * bpt / sec / 1e9,
                    "bitwise_equal_to_token_by_token": bool(same), "calls_per_timed_region": calls})
        log(f"{name}: batch {b:2d}: {steps / sec:8.2f} tok/s, HBM {passes * bpt / sec / 1e9:7.1f} GB/s, "
            f"logical weight rate {steps * bpt / sec / 1e9:8.1f} GB/s, same outputs: {same}")
    del ref
    return res


def mma_sweep(name, inp, specs, ws, steps, bpt, stream, wsr, batches=(1, 2, 4, 8, 16)):
    """Batched decode on the matrix cores: b tokens share one pass over the weights (b <= 16).
    The outputs agree with the token-by-token sweep within rounding; the worst rel-L2 is reported.
    Each timed region holds calls back to back, as a decode loop issues them (about 3 ms)."""
    import torch
    ref = [y.clone() for y in inp.y]           # the token-by-token outputs
    res = []
    for b in batches:
        if b > steps:
            break
        run = lambda: wsr.wsr_decode_sweep_mma(specs, b, ws, ws.numel(), stream)
        run()
        torch.cuda.synchronize()
        worst = 0.0
        for a, y in zip(ref, inp.y):
            d = torch.linalg.vector_norm((y[:b] - a[:b]).double(), dim=1)
            n = torch.linalg.vector_norm(a[:b].double(), dim=1).clamp_min(1e-30)
            worst = max(worst, float((d / n).max()))
        calls = calls_per_region(run, stream)
        sec = median_of(run, calls, 5, stream) / calls
        res.append({"batch": b, "ms_per_pass": sec * 1e3, "tokens_per_s": b / sec, "hbm_GBps": bpt / sec / 1e9,
                    "logical_weight_GBps": b * bpt / sec / 1e9, "worst_rel_l2_vs_token_by_token": worst,
                    "calls_per_timed_region": calls})
        log(f"{name}: matrix cores, batch {b:2d}: {b / sec:8.2f} tok/s, HBM {bpt / sec / 1e9:7.1f} GB/s, "
            f"worst rel-L2 vs token by token {worst:.1e}")
    for a, y in zip(ref, inp.y):               # leave the token-by-token outputs in place
        y.copy_(a)
    del ref
    return res


def check_sweep(inp, tokens, nrows=8):
    """Sampled rows of every matrix (first, last and spread rows) against the oracle."""
    import oracle
    from synth import workloads as wl
    ora = oracle.get()
    worst, n = 0.0, 0
    ys = {}
    for i, m in enumerate(inp.mats):
        rows = np.unique(np.linspace(0, m.M - 1, nrows).astype(np.int64))
        ys[i] = inp.y[i][tokens].cpu().numpy()
        for t_i, t in enumerate(tokens):
            x = inp.host_x(i, t)
            got = ys[i][t_i][rows].astype(np.float64)
            want = []
            for r in rows:
                hw = inp.host_weights(i, int(r), 1)
                want.append(oracle_gemv(ora, inp.fmts[i], hw, x)[0])
            want = np.array(want)
            err = float(np.linalg.norm(got - want) / max(np.linalg.norm(want), 1e-30))
            worst = max(worst, err)
            n += rows.size
    return {"worst_rel_l2": worst, "rows_checked": n, "tokens_checked": list(tokens), "tol": 2e-3,
            "ok": worst <= 2e-3}


def oracle_gemv(ora, fmt, hw, x, threads=1):
    from synth import workloads as wl
    if fmt in (wl.Q4, wl.I8):
        return ora.gemv(dict(fmt=fmt, w=hw[0], s=hw[1]), x, threads)
    return ora.gemv16(hw, x, fmt, threads=threads)


def oracle_threads():
    """Host threads for the oracle's all-core mode: every core this process may run on, capped by
    OMP_NUM_THREADS where that is set lower (a machine may grant the process only a share of its cores).
    Returns (threads used, cores available, the cap's source or None)."""
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count() or 1
    cap = os.environ.get("OMP_NUM_THREADS", "")
    if cap.isdigit() and 0 < int(cap) < avail:
        return int(cap), avail, f"OMP_NUM_THREADS={cap}"
    return avail, avail, None


def core_fields(threads, avail, cap):
    return {"cores": threads, "cores_available": avail, "thread_cap": cap}


def time_until(fn, seconds, max_calls=1 << 30):
    """Calls fn() until `seconds` have passed (at least once); returns (calls, seconds spent)."""
    t0 = time.perf_counter()
    n = 0
    while n < max_calls:
        fn()
        n += 1
        if time.perf_counter() - t0 >= seconds:
            break
    return n, time.perf_counter() - t0


def cpu_baseline(inp, bpt, seconds):
    """The oracle as it stands, all host cores, on the first matrices of token 0 until about
    `seconds` of oracle time; scaled to the whole token."""
    import oracle
    from synth import workloads as wl
    ora = oracle.get()
    threads, avail, cap = oracle_threads()
    spent, nbytes, names = 0.0, 0, []
    for i, m in enumerate(inp.mats):
        hw = inp.host_weights(i)
        x = inp.host_x(i, 0)
        t0 = time.perf_counter()
        oracle_gemv(ora, inp.fmts[i], hw, x, threads)
        spent += time.perf_counter() - t0
        nbytes += wl.matrix_bytes(m.M, m.K, inp.fmts[i])
        names.append(f"L{m.layer}.{m.name}")
        if spent >= seconds:
            break
    rate = nbytes / spent
    log(f"cpu oracle: {nbytes / 1e9:.2f} GB in {spent:.1f} s on {threads} threads -> {rate / 1e9:.2f} GB/s")
    # the second mode: one thread, on the first matrix
    hw = inp.host_weights(0)
    x = inp.host_x(0, 0)
    t0 = time.perf_counter()
    oracle_gemv(ora, inp.fmts[0], hw, x, 1)
    one = time.perf_counter() - t0
    m0 = inp.mats[0]
    rate1 = wl.matrix_bytes(m0.M, m0.K, inp.fmts[0]) / one
    log(f"cpu oracle, one thread: L{m0.layer}.{m0.name} in {one:.2f} s -> {rate1 / 1e9:.2f} GB/s")
    return {"value": rate / 1e9, "unit": "GB/s", **core_fields(threads, avail, cap), "kind": "oracle",
            "single_thread": {"value": rate1 / 1e9, "unit": "GB/s", "cores": 1, "seconds": one,
                              "tokens_per_s": rate1 / bpt,
                              "sample": f"token 0, L{m0.layer}.{m0.name} ({m0.M} x {m0.K})"},
            "tokens_per_s": rate / bpt, "seconds": spent,
            "sample": f"token 0, first {len(names)} matrices in sweep order ({names[0]} .. {names[-1]}), "
                      f"{nbytes / 1e9:.2f} GB of weights, fp64 oracle with OpenMP over rows"}


# --------------------------------------------------------------------------------------------------
# extra rows

def probe_cpu_baseline(host):
    """The oracle's probe sum on the host copy of the first buffer: one thread over the whole
    buffer, and all cores over contiguous parts of it (one ctypes call per thread; ctypes releases
    the GIL), the parts' sums added in order.  On the 2^-23 grid every sum is exact, so both modes
    must give the same value."""
    import oracle
    from concurrent.futures import ThreadPoolExecutor
    ora = oracle.get()
    threads, avail, cap = oracle_threads()
    nb = host.nbytes
    t0 = time.perf_counter()
    s1 = ora.probe_sum(host)
    one = time.perf_counter() - t0
    parts = np.array_split(host, threads)
    with ThreadPoolExecutor(threads) as ex:
        t0 = time.perf_counter()
        sums = list(ex.map(ora.probe_sum, parts))
        allc = time.perf_counter() - t0
    total = 0.0
    for v in sums:
        total += v
    log(f"cpu oracle, probe: one thread {nb / one / 1e9:.2f} GB/s, {threads} threads {nb / allc / 1e9:.2f} GB/s")
    return {"value": nb / allc / 1e9, "unit": "GB/s", **core_fields(threads, avail, cap), "kind": "oracle",
            "seconds": allc, "sums_equal": bool(total == s1),
            "single_thread": {"value": nb / one / 1e9, "unit": "GB/s", "cores": 1, "seconds": one},
            "sample": "the whole 1 GiB buffer (2^28 fp32 values), both modes"}


def row_probe(stream, wsr, mapped=True, want_cpu=True):
    import torch
    import synth
    from synth import device as dv
    from synth import workloads as wl
    n = wl.PROBE_N
    nb = n * 4
    first = synth.grid_f32(n, seed=0, stream=1)
    bufs = [dv.to_device(first)] + [dv.to_device(synth.grid_f32(n, seed=0, stream=1 + k)) for k in range(1, 4)]
    out = torch.zeros(1, dtype=torch.float64, device="cuda")
    ws = torch.zeros(wsr.wsr_probe_workspace_bytes(n), dtype=torch.uint8, device="cuda")
    call = lambda b: wsr.wsr_probe_read(b, n, out, ws, ws.numel(), stream)
    t0 = time.perf_counter()                # untimed for at least 0.5 s, as the other rows are
    while time.perf_counter() - t0 < 0.5:
        for b in bufs:
            call(b)
        torch.cuda.synchronize()
    same = median_of(lambda: call(bufs[0]), 20, 5, stream) / 20
    k = [0]

    def rot():
        call(bufs[k[0] & 3])
        k[0] += 1
    rotated = median_of(rot, 20, 5, stream) / 20
    res = {"bytes": nb, "resident_GBps": nb / rotated / 1e9, "resident_same_buffer_GBps": nb / same / 1e9,
           "resident_us": rotated * 1e6, "hbm_frac": nb / rotated / HBM_PEAK}
    del bufs
    torch.cuda.empty_cache()
    res["roofline"] = row_roofline(res["resident_GBps"], "probe", nb)
    if want_cpu:
        res["cpu_baseline"] = probe_cpu_baseline(first)
    del first
    if not mapped:
        log(f"probe: resident {res['resident_GBps']:.1f} GB/s (same buffer {res['resident_same_buffer_GBps']:.1f})")
        return res
    # host-mapped: the same kernel over pinned host pages read in place across PCIe
    host = torch.empty(nb, dtype=torch.uint8, pin_memory=True)
    synth.grid_f32(n, seed=0, stream=1, out=host.numpy().view(np.float32))
    t_reg = time.perf_counter()
    dev, granted = wsr.wsr_register_host(host, nb, 0)
    res["mapped_register_s"] = time.perf_counter() - t_reg      # setup, outside the rate
    try:
        call(dev)
        mapped = median_of(lambda: call(dev), 2, 3, stream) / 2
        res.update({"mapped_GBps": nb / mapped / 1e9, "mapped_registration": granted})
    finally:
        t_unreg = time.perf_counter()
        wsr.wsr_unregister_host(host)
        res["mapped_unregister_s"] = time.perf_counter() - t_unreg
    log(f"probe: resident {res['resident_GBps']:.1f} GB/s (same buffer {res['resident_same_buffer_GBps']:.1f}), "
        f"host-mapped {res['mapped_GBps']:.1f} GB/s")
    return res


def gemv_cpu_baseline(mats, x, fmt, seconds, what):
    """The oracle's 16-bit GEMV over host matrices (visited in turn) for about `seconds` in each
    mode: one thread, then all cores (OpenMP over rows)."""
    import oracle
    ora = oracle.get()
    threads, avail, cap = oracle_threads()
    out = {}
    for mode, th in (("single_thread", 1), ("all", threads)):
        k = [0]

        def one():
            ora.gemv16(mats[k[0] % len(mats)], x, fmt, threads=th)
            k[0] += 1
        calls, sec = time_until(one, seconds)
        nbytes = sum(mats[i % len(mats)].nbytes for i in range(calls))
        out[mode] = {"value": nbytes / sec / 1e9, "unit": "GB/s", "calls": calls, "seconds": sec,
                     "gemv_per_s": calls / sec}
    log(f"cpu oracle, {what}: one thread {out['single_thread']['value']:.2f} GB/s, "
        f"{threads} threads {out['all']['value']:.2f} GB/s")
    return {"value": out["all"]["value"], "unit": "GB/s", **core_fields(threads, avail, cap), "kind": "oracle",
            "seconds": out["all"]["seconds"], "gemv_per_s": out["all"]["gemv_per_s"],
            "single_thread": dict(out["single_thread"], cores=1),
            "sample": f"{what}, about {seconds:g} s per mode"}


def row_gemv_f16(stream, wsr, want_cpu=True):
    import torch
    import synth
    from synth import device as dv
    from synth import workloads as wl
    cfg = wl.GemvConfig()
    host_W = [synth.normal16((cfg.M, cfg.K), wl.W_SIGMA, "f16", seed=0, stream=1 + b) for b in range(cfg.rotate)]
    host_x = synth.normal16(cfg.K, wl.X_SIGMA, "f16", seed=0, stream=1000)
    Ws = [dv.to_device(W) for W in host_W]
    x = dv.to_device(host_x)
    y = torch.empty((cfg.rotate, cfg.M), dtype=torch.float32, device="cuda")
    bytes_one = cfg.M * cfg.K * 2

    def pass_():
        for b in range(cfg.rotate):
            wsr.wsr_gemv_f16(Ws[b], x, y[b], cfg.M, cfg.K, wsr.WSR_F16, stream)
    t0 = time.perf_counter()                # untimed for at least 0.5 s, as the other rows are
    while time.perf_counter() - t0 < 0.5:
        pass_()
        torch.cuda.synchronize()
    t = median_of(pass_, 1, 15, stream)
    per = t / cfg.rotate
    # the same 32 matrices as one persistent launch
    specs = wsr.make_mats([dict(fmt=1, M=cfg.M, K=cfg.K, w=Ws[b], x=x, y=y[b]) for b in range(cfg.rotate)])
    ws = torch.zeros(wsr.wsr_sweep_workspace_bytes(specs), dtype=torch.uint8, device="cuda")
    wsr.wsr_decode_sweep(specs, 1, ws, ws.numel(), stream)
    # four back-to-back passes per timing, like the 32 dispatches of a pass above
    tf = median_of(lambda: wsr.wsr_decode_sweep(specs, 1, ws, ws.numel(), stream), 4, 15, stream) / 4
    # labelled apart: one matrix dispatched 32 times, so it stays in the 256 MB Infinity Cache
    tw = median_of(lambda: wsr.wsr_gemv_f16(Ws[0], x, y[0], cfg.M, cfg.K, wsr.WSR_F16, stream), cfg.rotate, 15,
                   stream) / cfg.rotate
    res = {"bytes_per_gemv": bytes_one, "us_per_gemv": per * 1e6, "GBps_per_dispatch": bytes_one / per / 1e9,
           "hbm_frac_per_dispatch": bytes_one / per / HBM_PEAK,
           "one_launch_32_matrices_GBps": bytes_one * cfg.rotate / tf / 1e9,
           "one_launch_32_matrices_hbm_frac": bytes_one * cfg.rotate / tf / HBM_PEAK,
           "one_launch_us": tf * 1e6,
           "single_buffer_cache_warm": {"us_per_gemv": tw * 1e6, "GBps": bytes_one / tw / 1e9,
                                        "note": "one 32 MiB matrix repeated: served from the Infinity Cache, not HBM"}}
    log(f"gemv_f16 4096x4096: {per * 1e6:.2f} us/GEMV ({res['GBps_per_dispatch']:.1f} GB/s over 32 dispatches); "
        f"one launch over all 32: {res['one_launch_32_matrices_GBps']:.1f} GB/s; one buffer repeated "
        f"(cache-warm): {tw * 1e6:.2f} us/GEMV")
    res["roofline"] = row_roofline(res["GBps_per_dispatch"], "gemv_f16", bytes_one)
    res["roofline_one_launch"] = row_roofline(res["one_launch_32_matrices_GBps"], "gemv_f16_one_launch",
                                              bytes_one * cfg.rotate)
    if want_cpu:
        res["cpu_baseline"] = gemv_cpu_baseline(host_W, host_x, "f16", 2.0,
                                                f"the 32 rotated {cfg.M} x {cfg.K} fp16 matrices in turn")
    del Ws
    torch.cuda.empty_cache()
    return res


def row_protocol(stream, wsr, warmup_passes=12, passes=31, tokens=16, want_cpu=True):
    """The matched protocol of Sec. 3.1: a pass is one single-token int8 GEMV (fp16 row scales) over
    each of 12 distinct 12288 x 7168 matrices, bracketed by one synchronisation; the first 12
    passes are discarded and the median pass is reported, counting weight bytes once.  Measured as
    12 dispatches per pass (the protocol's form) and as one launch over all 12, plus the
    multi-column T-sweep on the same weights."""
    import torch
    from synth import device as dv
    from synth import workloads as wl
    mats = wl.protocol_matrices()
    inp = dv.SweepInputs(mats, [wl.I8] * len(mats), tokens=tokens)
    nbytes = inp.weight_bytes()
    sp = inp.specs()

    def dispatches():
        for d in sp:
            wsr.wsr_gemv_i8(d["w"], d["scales"], d["x"], d["y"], d["M"], d["K"], stream)
    specs = wsr.make_mats(sp)
    ws = torch.zeros(wsr.wsr_sweep_workspace_bytes(specs), dtype=torch.uint8, device="cuda")
    one = lambda: wsr.wsr_decode_sweep(specs, 1, ws, ws.numel(), stream)
    res = {"matrices": len(mats), "M": wl.PROTOCOL_M, "K": wl.PROTOCOL_K, "bytes_per_pass": nbytes,
           "warmup_passes": warmup_passes, "timed_passes": passes,
           "paper_context_GBps": {"packed_int8_resident": 523, "pure_read_reference": 517,
                                  "note": "another machine (unified memory); context, not a target"}}
    # the 12 dispatches recorded once in a HIP graph and replayed per pass: the same kernels and
    # launch shapes, without the host launching each one
    dispatches()
    torch.cuda.synchronize()
    eager = [d["y"][0].clone() for d in sp]   # a single-token GEMV writes token 0's outputs only
    graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(graph, stream=cap):
            for d in sp:
                wsr.wsr_gemv_i8(d["w"], d["scales"], d["x"], d["y"], d["M"], d["K"], cap)
    torch.cuda.current_stream().wait_stream(cap)
    replay = graph.replay
    replays_ok = True
    for _ in range(3):                     # each replay, with eager work between, gives the eager bits
        for d in sp:
            d["y"][0].fill_(float("nan"))
        replay()
        torch.cuda.synchronize()
        replays_ok &= all(torch.equal(a, d["y"][0]) for a, d in zip(eager, sp))
    # the one-launch pass back to back (8 per event pair): the kernel's own rate, without the host's
    # launch latency that a pass bracketed by its own synchronisation includes
    for _ in range(warmup_passes):
        one()
    t0 = time.perf_counter()                # untimed for at least 0.5 s, as the other rows are
    while time.perf_counter() - t0 < 0.5:
        for _ in range(8):
            one()
        torch.cuda.synchronize()
    res["warmup_seconds_one_launch"] = round(time.perf_counter() - t0, 3)
    b2b = [timed(one, 8, stream) / 8 * 1e3 for _ in range(passes)]
    st = spread(b2b)
    res["one_launch_back_to_back"] = {"median_ms_per_pass": st["median"], "iqr_ms": st["iqr"],
                                      "GBps_at_median": nbytes / (st["median"] * 1e-3) / 1e9,
                                      "hbm_frac": nbytes / (st["median"] * 1e-3) / HBM_PEAK}
    res["roofline"] = row_roofline(res["one_launch_back_to_back"]["GBps_at_median"], "protocol", nbytes)
    log(f"protocol one launch, back to back: median {st['median'] * 1e3:.1f} us/pass, "
        f"{res['one_launch_back_to_back']['GBps_at_median']:.1f} GB/s")
    for name, fn in (("dispatches_12", dispatches), ("one_launch", one), ("graph_12", replay)):
        for _ in range(warmup_passes):
            fn()
        ms = [timed(fn, 1, stream) * 1e3 for _ in range(passes)]
        st = spread(ms)
        res[name] = {"median_ms_per_pass": st["median"], "iqr_ms": st["iqr"], "ci95_ms": st["ci95_median"],
                     "GBps_at_median": nbytes / (st["median"] * 1e-3) / 1e9,
                     "hbm_frac": nbytes / (st["median"] * 1e-3) / HBM_PEAK}
        if name == "graph_12":
            torch.cuda.synchronize()
            res[name]["bitwise_equal_to_dispatches"] = bool(replays_ok) and all(
                torch.equal(a, d["y"][0]) for a, d in zip(eager, sp))
        log(f"protocol {name}: median {st['median'] * 1e3:.1f} us/pass, "
            f"{res[name]['GBps_at_median']:.1f} GB/s ({res[name]['hbm_frac'] * 100:.1f}% of 8 TB/s)")
    wsr.wsr_decode_sweep(specs, tokens, ws, ws.numel(), stream)
    torch.cuda.synchronize()
    res["parity"] = check_sweep(inp, [0, tokens - 1], nrows=4)
    log(f"protocol: parity on sampled rows: worst rel-L2 {res['parity']['worst_rel_l2']:.2e}")
    res["batched"] = batch_sweep("protocol", inp, specs, ws, tokens, nbytes, stream, wsr, (1, 2, 4, 8))
    res["batched_matrix_cores"] = mma_sweep("protocol", inp, specs, ws, tokens, nbytes, stream, wsr)
    if want_cpu:
        res["cpu_baseline"] = cpu_baseline(inp, nbytes, 3.0)
    del specs, ws, inp
    torch.cuda.empty_cache()
    return res


def row_endpoints(stream, wsr, warmup=2, passes=5, stage_mib=64):
    """Alg. 2 (Sec. 8.1) on this machine, over the protocol's working set (12 int8 matrices of
    12288 x 7168 with row scales, 1.06 GB) stored as a file: map and prefault the file, check its
    residency, measure map, resident and per-use copy with the same row loops, check residency
    again, and let the library's selection rank W / B with the 5 % band.  The GPU cannot read an
    unregistered file mapping here and registering existing pages is refused on this platform, so
    the map arm reads the same bytes in place from pinned host pages (Alg. 1's adoption of pages
    that are already device-visible); the copy arm stages from the file pages themselves."""
    import tempfile
    import torch
    import synth
    from synth import device as dv
    from synth import workloads as wl
    mats = wl.protocol_matrices()
    M, K = wl.PROTOCOL_M, wl.PROTOCOL_K
    code_b, scale_b = M * K, M * 2
    per = code_b + scale_b
    W = per * len(mats)
    page = os.sysconf("SC_PAGE_SIZE")
    path = os.path.join(tempfile.gettempdir(), f"wsr_protocol_{os.getpid()}.bin")
    res = {"working_set_bytes": W, "matrices": len(mats), "file": "codes then row scales per matrix"}
    try:
        t0 = time.time()
        with open(path, "wb") as f:
            for m in mats:
                f.write(synth.i8_codes(M, K, seed=wl.SEED, stream=wl.w_stream(m.index)).tobytes())
                f.write(synth.i8_scales(M, seed=wl.SEED, stream=wl.s_stream(m.index)).tobytes())
        fmap = np.memmap(path, dtype=np.uint8, mode="r")
        # step 1: prefault; step 2: residency of the mapped set
        _ = int(fmap[::page].sum())
        r_pages, t_pages = wsr.wsr_host_resident_pages(fmap.ctypes.data, W)
        res["file_written_and_prefaulted_s"] = time.time() - t0
        res["mapped_resident_pages"] = [r_pages, t_pages]
        log(f"endpoints: {W / 1e9:.2f} GB file mapped, {r_pages}/{t_pages} pages resident")
        xs = [dv.to_device(synth.normal16(K, wl.X_SIGMA, "f16", seed=wl.SEED,
                                          stream=wl.x_stream(m.layer, wl.X_SLOTS[m.slot]))) for m in mats]
        ys = {a: [torch.empty(M, dtype=torch.float32, device="cuda") for _ in mats] for a in ("map", "resident", "copy_file", "copy_pinned")}

        def specs(base, arm):
            return wsr.make_mats([dict(fmt=wsr.WSR_I8, M=M, K=K, w=base + i * per, scales=base + i * per + code_b,
                                       x=xs[i], y=ys[arm][i]) for i in range(len(mats))])

        def timed_arm(fn):
            for _ in range(warmup):
                fn()
            torch.cuda.synchronize()
            return float(np.median([timed(fn, 1, stream) for _ in range(passes)]))

        # resident arm: one copy of the file pages into device memory, then the sweep over it
        dev = torch.empty(W, dtype=torch.uint8, device="cuda")
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        dev.copy_(torch.from_numpy(np.asarray(fmap)))
        torch.cuda.synchronize()
        res["one_time_copy_s"] = time.perf_counter() - t1
        sp_dev = specs(dev.data_ptr(), "resident")
        ws = torch.zeros(wsr.wsr_sweep_workspace_bytes(sp_dev), dtype=torch.uint8, device="cuda")
        t_res = timed_arm(lambda: wsr.wsr_decode_sweep(sp_dev, 1, ws, ws.numel(), stream))
        # map arm: the same bytes read in place from pinned host pages, adopted through registration
        pinned = torch.empty((W + page - 1) // page * page, dtype=torch.uint8, pin_memory=True)
        pinned.numpy()[:W] = fmap
        t_reg = time.perf_counter()
        dview, granted = wsr.wsr_register_host(pinned, pinned.numel(), 0)
        res["register_s"] = time.perf_counter() - t_reg           # setup, outside every rate (a1)
        try:
            sp_map = specs(dview, "map")
            t_map = timed_arm(lambda: wsr.wsr_decode_sweep(sp_map, 1, ws, ws.numel(), stream))
            # per-use copy: staged through 2 x stage_mib of device memory, from the file pages and
            # from the pinned pages
            stage = torch.empty(2 * stage_mib << 20, dtype=torch.uint8, device="cuda")
            cs = torch.cuda.Stream()
            sp_cf = specs(fmap.ctypes.data, "copy_file")
            sp_cp = specs(pinned.data_ptr(), "copy_pinned")
            t_cf = timed_arm(lambda: wsr.wsr_sweep_staged(sp_cf, 0, stage, stage.numel(), stream, cs))
            t_cp = timed_arm(lambda: wsr.wsr_sweep_staged(sp_cp, 0, stage, stage.numel(), stream, cs))
            torch.cuda.synchronize()
        finally:
            t_unreg = time.perf_counter()
            wsr.wsr_unregister_host(pinned)
            res["unregister_s"] = time.perf_counter() - t_unreg
        same = all(torch.equal(ys["resident"][i], ys[a][i]) for a in ("map", "copy_file", "copy_pinned")
                   for i in range(len(mats)))
        # step 5: the mapping after one pass of every arm
        r_after, _ = wsr.wsr_host_resident_pages(fmap.ctypes.data, W)
        mapped_resident = r_pages == t_pages
        resident_ok = r_after == t_pages
        rates = {"map": W / t_map, "resident": W / t_res, "copy": W / t_cf}
        res.update({
            "GBps": {"map_pinned_in_place": W / t_map / 1e9, "resident": W / t_res / 1e9,
                     "copy_from_file_pages": W / t_cf / 1e9, "copy_from_pinned": W / t_cp / 1e9},
            "ms_per_pass": {"map": t_map * 1e3, "resident": t_res * 1e3, "copy_file": t_cf * 1e3,
                            "copy_pinned": t_cp * 1e3},
            "one_time_copy_GBps": W / res["one_time_copy_s"] / 1e9,
            "register_granted": granted, "mapped_resident_pages_after": r_after,
            "outputs_bitwise_equal_across_arms": bool(same), "stage_bytes": 2 * stage_mib << 20})
        verdicts = {}
        for theta in (0.02, 0.05, 0.10, 0.20):
            code, times = wsr.wsr_select_endpoint(W, rates["map"], rates["resident"], rates["copy"], theta,
                                                  mapped_resident, resident_ok)
            verdicts[f"{theta:.2f}"] = wsr.ENDPOINT_NAMES[code]
        res["alg2"] = {"theta": 0.05, "choice": verdicts["0.05"], "path_time_ms": dict(zip(("map", "resident", "copy"), times)),
                       "theta_sweep": verdicts, "mapped_resident": mapped_resident, "resident_ok": resident_ok}
        log(f"endpoints: map {W / t_map / 1e9:.1f} GB/s, resident {W / t_res / 1e9:.1f} GB/s, "
            f"copy from file {W / t_cf / 1e9:.1f} GB/s (pinned {W / t_cp / 1e9:.1f}); one-time copy "
            f"{res['one_time_copy_GBps']:.1f} GB/s; Alg. 2 -> {verdicts['0.05']} (theta 2-20 %: "
            f"{sorted(set(verdicts.values()))}); outputs equal: {same}")
        del dev, pinned, stage, ws, fmap
        torch.cuda.empty_cache()
    finally:
        if os.path.exists(path):
            os.remove(path)
    return res


def row_ordering(stream, wsr, depths=(2, 8, 32), steps=20, reps=7, seed=0, workloads=("mm", "small")):
    """Sec. 4.3's ordering hierarchy on HIP.  A step of a decode-like loop: the framework issues D
    matrix products on its stream and then writes the pass's activation; the weight pass (the
    protocol's 1.06 GB of int8, one launch) is ordered after that by one of four mechanisms; the
    framework's next operation reads the pass's output.  Excess = time per step minus that of the
    same loop without the pass, paired within each repetition; arms run in a shuffled order per
    repetition.  The pass alone on an idle GPU is the floor of every excess."""
    import torch
    from synth import device as dv
    from synth import workloads as wl
    mats = wl.protocol_matrices()
    inp = dv.SweepInputs(mats, [wl.I8] * len(mats), tokens=1)
    specs = wsr.make_mats(inp.specs())
    ws = torch.zeros(wsr.wsr_sweep_workspace_bytes(specs), dtype=torch.uint8, device="cuda")
    fs, own = torch.cuda.Stream(), torch.cuda.Stream()
    a = torch.randn(2048, 2048, device="cuda", dtype=torch.bfloat16)
    small = torch.zeros(1 << 14, device="cuda")
    x0 = next(iter(inp.x.values()))[0][0]          # the activation the framework writes
    xsrc = x0.clone()
    acc = torch.zeros(16, device="cuda")
    rng = np.random.default_rng(seed)
    modes = {"none": None, "in-stream": wsr.WSR_ORDER_STREAM, "event": wsr.WSR_ORDER_EVENT,
             "host-visible event": wsr.WSR_ORDER_HOST_EVENT, "host drain": wsr.WSR_ORDER_DRAIN}

    def run(mode, depth, n, work):
        for _ in range(n):
            with torch.cuda.stream(fs):
                if work == "mm":
                    b = a
                    for _ in range(depth):
                        b = torch.mm(b, a)
                else:
                    for _ in range(depth):
                        small.add_(1.0)
                x0.copy_(xsrc)
            if mode is not None:
                wsr.wsr_decode_sweep_ordered(specs, 1, ws, ws.numel(), fs, own, mode)
            with torch.cuda.stream(fs):
                acc.add_(inp.y[0][0, :16])

    pass_alone = median_of(lambda: wsr.wsr_decode_sweep(specs, 1, ws, ws.numel(), stream), 1, 15, stream)
    op_ms = {}
    with torch.cuda.stream(fs):
        op_ms["mm"] = median_of(lambda: torch.mm(a, a), 8, 5, fs) / 8 * 1e3
        op_ms["small"] = median_of(lambda: small.add_(1.0), 64, 5, fs) / 64 * 1e3
    res = {"pass_alone_ms": pass_alone * 1e3, "steps": steps, "repetitions": reps,
           "workloads": {"mm": "bf16 mm 2048 x 2048 x 2048 (GPU-bound: the host enqueues faster than the GPU runs)",
                         "small": "in-place add on 16K floats (launch-bound: the GPU runs as fast as the host enqueues)"},
           "op_gpu_ms": op_ms, "results": {},
           "paper_context_ms": {"in-stream": 0.33, "event": 0.44, "host-visible event": 3.46,
                                "host drain": 5.80, "note": "Apple M5 Max and Metal; another machine"}}
    for work in workloads:
        for depth in depths:
            for m in modes.values():
                run(m, depth, 2, work)
            torch.cuda.synchronize()
            excess = {k: [] for k in modes if k != "none"}
            base = []
            for _ in range(reps):
                order = list(modes)
                rng.shuffle(order)
                t = {}
                for k in order:
                    torch.cuda.synchronize()
                    t0 = time.perf_counter()
                    run(modes[k], depth, steps, work)
                    torch.cuda.synchronize()
                    t[k] = (time.perf_counter() - t0) / steps
                base.append(t["none"] * 1e3)
                for k in excess:
                    excess[k].append((t[k] - t["none"]) * 1e3)
            row = {k: {"median_ms": float(np.median(v)), "iqr_ms": [float(np.percentile(v, 25)), float(np.percentile(v, 75))]}
                   for k, v in excess.items()}
            res["results"][f"{work}/{depth}"] = {"step_without_pass_ms": float(np.median(base)), "excess": row}
            log(f"ordering, {work} x {depth} per step ({np.median(base):.3f} ms without the pass): " +
                ", ".join(f"{k} {v['median_ms']:.3f}" for k, v in row.items()) +
                f" ms (pass alone {pass_alone * 1e3:.3f} ms)")
    del specs, ws, inp, a
    torch.cuda.empty_cache()
    return res


def row_size_sweep(stream, wsr, mapped=True, want_cpu=True):
    """The bf16 matrix-size sweep (Sec. 3.4) in both readings of its shapes: reduction length 4096
    with N output rows, and 4096 output rows with reduction length N, for the 12 sizes of N.  Both
    readings stream the same bytes per matrix, so they share the weight buffers: resident (rotated
    over at least 1 GiB of distinct buffers, and one buffer repeated) and host-mapped (one pinned
    buffer read in place)."""
    import torch
    import synth
    from synth import device as dv
    from synth import workloads as wl
    K0 = wl.SWEEP_K
    maxN = max(wl.SWEEP_N)
    x_rows_host = synth.normal16(K0, wl.X_SIGMA, "bf16", seed=0, stream=2)
    x_rows = dv.to_device(x_rows_host)
    x_cols_host = synth.normal16(maxN, wl.X_SIGMA, "bf16", seed=0, stream=3)
    x_cols = dv.to_device(x_cols_host)
    host = torch.empty(maxN * K0 * 2, dtype=torch.uint8, pin_memory=True)
    synth.normal16(maxN * K0, wl.W_SIGMA, "bf16", seed=0, stream=1, out=host.numpy().view(np.uint16))
    hdev = None
    if mapped:
        hdev, granted = wsr.wsr_register_host(host, host.numel(), 0)
    readings = {"rows": [], "cols": []}    # rows: M = N, K = 4096; cols: M = 4096, K = N
    try:
        for N in wl.SWEEP_N:
            nbytes = N * K0 * 2
            rot = max(1, -(-(1 << 30) // nbytes))   # distinct buffers per pass: at least 1 GiB
            Ws = [torch.empty(N * K0, dtype=torch.int16, device="cuda") for _ in range(rot)]
            for W in Ws:
                W.view(torch.uint8).copy_(host[:nbytes], non_blocking=True)
            for name, M, K, x in (("rows", N, K0, x_rows), ("cols", K0, N, x_cols)):
                y = torch.empty(M, dtype=torch.float32, device="cuda")
                k = [0]

                def res_call():
                    wsr.wsr_gemv_f16(Ws[k[0] % rot], x, y, M, K, wsr.WSR_BF16, stream)
                    k[0] += 1
                res_call()
                reps = max(rot, 8)
                tr = median_of(res_call, reps, 5, stream) / reps
                ts = median_of(lambda: wsr.wsr_gemv_f16(Ws[0], x, y, M, K, wsr.WSR_BF16, stream), 8, 5, stream) / 8
                pt = {"N": N, "M": M, "K": K, "bytes": nbytes, "resident_GBps": nbytes / tr / 1e9,
                      "resident_same_buffer_GBps": nbytes / ts / 1e9, "resident_us": tr * 1e6,
                      "hbm_frac": nbytes / tr / HBM_PEAK}
                if mapped:
                    tm = median_of(lambda: wsr.wsr_gemv_f16(hdev, x, y, M, K, wsr.WSR_BF16, stream), 1, 3, stream)
                    pt["mapped_GBps"] = nbytes / tm / 1e9
                readings[name].append(pt)
                log(f"size sweep {name} M={M:6d} K={K:6d} ({nbytes / 2**20:7.1f} MiB): resident {nbytes / tr / 1e9:7.1f} GB/s, "
                    f"same-buffer {nbytes / ts / 1e9:7.1f}" + (f", host-mapped {pt['mapped_GBps']:6.1f}" if mapped else ""))
            del Ws
            torch.cuda.empty_cache()
    finally:
        if mapped:
            wsr.wsr_unregister_host(host)
    out = {"points": readings["rows"], "crossovers": size_crossovers(readings["rows"], "rows"),
           "transposed": {"points": readings["cols"], "crossovers": size_crossovers(readings["cols"], "cols"),
                          "shape": "M = 4096 output rows, K = N"},
           "shape": "M = N output rows, K = 4096"}
    if want_cpu:
        W = host.numpy().view(np.uint16)
        out["cpu_baseline"] = gemv_cpu_baseline([W.reshape(maxN, K0)], x_rows_host, "bf16", 2.0,
                                                f"the largest matrix, {maxN} x {K0} bf16 (1.15 GB)")
        out["transposed"]["cpu_baseline"] = gemv_cpu_baseline([W.reshape(K0, maxN)], x_cols_host, "bf16", 2.0,
                                                              f"the largest matrix, {K0} x {maxN} bf16 (1.15 GB)")
    del host
    return out


def size_crossovers(pts, name="rows"):
    """The size sweep's three crossovers (Sec. 3.4's matrix-size sweep): (i) dispatch, the smallest
    size whose resident rate reaches half the plateau; (ii) MALL, the smallest size from which the
    single-buffer repeat rate stays within 2 % of the rotated rate (below it the repeated buffer
    is served partly from the 256 MB Infinity Cache); (iii) the first size where a host-mapped pass
    is as fast as a resident one (none expected across PCIe)."""
    plateau = max(p["resident_GBps"] for p in pts)
    disp = next(p for p in pts if p["resident_GBps"] >= 0.5 * plateau)
    mall = None
    for i in range(len(pts)):
        if all(q["resident_same_buffer_GBps"] <= 1.02 * q["resident_GBps"] for q in pts[i:]):
            mall = pts[i]
            break
    best = max(pts, key=lambda p: p["resident_same_buffer_GBps"] / p["resident_GBps"])
    mapped = next((p for p in pts if p.get("mapped_GBps", 0.0) >= p["resident_GBps"]), None)
    out = {"resident_plateau_GBps": plateau,
           "dispatch": {"bytes": disp["bytes"], "N": disp["N"], "resident_GBps": disp["resident_GBps"],
                        "paper_context": "about 23 MB on the paper's machine (Sec. 3.4); context, not a target"},
           "mall": None if mall is None else {"bytes": mall["bytes"], "N": mall["N"]},
           "largest_repeat_gain": {"bytes": best["bytes"],
                                   "same_buffer_over_rotated": best["resident_same_buffer_GBps"] / best["resident_GBps"]},
           "mapped_equals_resident": None if mapped is None else {"bytes": mapped["bytes"], "N": mapped["N"]}}
    if not any("mapped_GBps" in p for p in pts):
        out["mapped_equals_resident"] = "not measured"
    mall_txt = "none" if mall is None else f"{mall['bytes'] / 1e6:.1f} MB"
    mapped_txt = "never" if mapped is None else f"{mapped['bytes'] / 1e6:.1f} MB"
    log(f"size sweep {name}: plateau {plateau:.0f} GB/s; dispatch crossover {disp['bytes'] / 1e6:.1f} MB; "
        f"MALL crossover {mall_txt}; mapped = resident: {mapped_txt}")
    return out


def row_copy(stream):
    """A plain elementwise pass of known size (1 GiB read, 1 GiB written): the calibration kernel
    for the FETCH_SIZE / WRITE_SIZE hardware counters."""
    import torch
    n = 1 << 28
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    torch.neg(a, out=b)
    t = median_of(lambda: torch.neg(a, out=b), 1, 5, stream)
    log(f"copy: 1 GiB read + 1 GiB written in {t * 1e6:.1f} us -> {2 * 4 * n / t / 1e9:.1f} GB/s")
    return {"bytes_read": 4 * n, "bytes_written": 4 * n, "us": t * 1e6, "GBps_rw": 2 * 4 * n / t / 1e9}


def row_bus(stream):
    import torch
    n = 1 << 30
    h = torch.empty(n, dtype=torch.uint8, pin_memory=True)
    d = torch.empty(n, dtype=torch.uint8, device="cuda")
    d.copy_(h, non_blocking=True)
    t = median_of(lambda: d.copy_(h, non_blocking=True), 1, 5, stream)
    log(f"bus: pinned host->device copy {n / t / 1e9:.1f} GB/s")
    return {"h2d_GBps": n / t / 1e9}


# --------------------------------------------------------------------------------------------------

def across_processes(args):
    """The headline measured in separate processes (each its own inputs, warm-up and passes)."""
    import subprocess
    meds, firsts = [], []
    for k in range(args.processes):
        cmd = [sys.executable, os.path.abspath(__file__), "--workload", args.workload, "--rows", "",
               "--no-cpu-baseline", "--steps", str(args.steps), "--warmup", str(args.warmup),
               "--passes", str(args.passes)]
        log(f"process {k + 1}/{args.processes}: {' '.join(cmd[1:])}")
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            sys.stderr.write(r.stdout[-2000:] + r.stderr[-2000:])
            raise SystemExit(r.returncode)
        line = json.loads([l for l in r.stdout.splitlines() if l.startswith("{")][-1])
        meds.append(line["passes"]["median"])
        firsts.append(line["ms_per_step"])
        log(f"process {k + 1}: median {line['passes']['median']:.4f} ms/token over {line['passes']['n']} passes")
    st = spread(meds)
    bpt = None
    from synth import workloads as wl
    shape, fmt = SWEEPS[args.workload]
    bpt = wl.bytes_per_token(getattr(wl, shape), fmt)
    print(json.dumps({"workload": args.workload, "processes": args.processes, "steps": args.steps,
                      "passes_per_process": args.passes + 1, "process_medians_ms": meds,
                      "first_pass_ms": firsts, "median_of_medians_ms": st["median"],
                      "iqr_ms": st["iqr"], "ci95_ms": st["ci95_median"],
                      "GBps_at_median": round(bpt / (st["median"] * 1e-3) / 1e9, 2)}), flush=True)


def measured_ceiling(head_gbps, rows):
    """The second denominator: the streaming-read probe's resident rate measured in this run (the
    pure-read reference), against which the headline and every row's roofline rate are also given
    (`frac_of_probe`, added to each row).  The probe's timed passes are 1 GiB each (two launches),
    where a 70B sweep token is one launch over 139 GB, so a long sweep can pass it slightly."""
    if "probe" not in rows:
        return None
    pc = rows["probe"]["resident_GBps"]
    for key, r in rows.items():
        rl = r.get("roofline") if isinstance(r, dict) else None
        if rl and rl.get("achieved") and key != "probe":
            r["frac_of_probe"] = round(rl["achieved"] / pc, 4)
    return {"GBps": round(pc, 1), "frac": round(head_gbps / pc, 4),
            "source": "rows.probe.resident_GBps: 1 GiB fp32 probe, four buffers rotated, back to back",
            "note": "probe passes are 1 GiB (two launches each); the sweep token is one launch over all its "
                    "bytes, so its ramp and drain weigh less and the fraction can exceed 1"}


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "bench.py measures one GPU: the weight-streaming path has no "
                                   "multi-GPU form here (a sharded run would split rows across GPUs); "
                                   "run with --gpus 1"}))
        sys.exit(2)
    if args.processes > 1:
        return across_processes(args)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    from paper_2608_12114_amd import wsr
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    t_start = time.time()

    head = run_sweep(args.workload, args.steps, args.warmup, stream, wsr, not args.no_cpu_baseline,
                     args.cpu_seconds, args.passes)
    rows = {}
    cpu = not args.no_cpu_baseline
    for r in [r for r in args.rows.split(",") if r]:
        if r == "probe":
            rows[r] = row_probe(stream, wsr, mapped=not args.no_mapped, want_cpu=cpu)
        elif r == "gemv_f16":
            rows[r] = row_gemv_f16(stream, wsr, want_cpu=cpu)
        elif r == "llama8b_q4":
            if args.workload != "llama8b_q4":
                rows[r] = run_sweep("llama8b_q4", 64, 4, stream, wsr, cpu, 3.0, warm_seconds=0.5)
        elif r == "size_sweep":
            rows[r] = row_size_sweep(stream, wsr, mapped=not args.no_mapped, want_cpu=cpu)
        elif r == "protocol":
            rows[r] = row_protocol(stream, wsr, want_cpu=cpu)
        elif r == "endpoints":
            rows[r] = row_endpoints(stream, wsr)
        elif r == "ordering":
            rows[r] = row_ordering(stream, wsr)
        elif r == "bus":
            rows[r] = row_bus(stream)
        elif r == "copy":
            rows[r] = row_copy(stream)
        else:
            raise SystemExit(f"unknown row {r}")

    gbps = head["GBps"]
    probe_ceiling = measured_ceiling(gbps, rows)
    dtype = {"llama70b_bf16": "bf16", "llama8b_q4": "q4+f16"}[args.workload]
    traffic, traffic_src = profiled_traffic(args.workload)
    line = {
        "metric": "achieved GB/s (% of HBM peak) for decode-step GEMV sweep; tokens/s at batch 1",
        "value": round(gbps, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(head["ms_per_token"], 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": dtype, "data": "synthetic",
        "config": {"workload": {"llama70b_bf16": "Llama-70B-shaped bf16 decode weight sweep, batch 1",
                                "llama8b_q4": "Llama-3-8B-shaped q4 decode weight sweep, batch 1"}[args.workload],
                   "layers": {"llama70b_bf16": 80, "llama8b_q4": 32}[args.workload],
                   "bytes_per_token": head["bytes_per_token"], "residency": "HBM",
                   "step": "one decode token: every projection matrix of every layer plus lm_head, one launch"},
        "tokens_per_s": round(head["tokens_per_s"], 3), "hbm_frac": round(head["hbm_frac"], 4),
        "roofline": {"bound": "hbm", "achieved": round(gbps, 2), "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                     "frac": round(head["hbm_frac"], 4), "traffic": traffic, "traffic_source": traffic_src,
                     "kernel": f"k_sweep ({dtype})", "bytes_per_launch": head["bytes_per_token"]},
        "probe_ceiling": probe_ceiling,
        "cpu_baseline": head.get("cpu_baseline"),
        "parity": head["parity"],
        "passes": head["passes"],
        "rows": rows,
        "wall_s": round(time.time() - t_start, 1),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
