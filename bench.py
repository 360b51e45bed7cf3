#!/usr/bin/env python3
"""Benchmark of the MI355X binary-delta matmul.

Prints ONE JSON line.  Headline workload (one "step"): the single-tenant
decode GEMV pair x[1,4096] and x[16,4096] against W_base[4096,4096] with one
packed 4096x4096 sign matrix, bf16 output -- two launches of the decode kernel.
`value` is whole-step HBM throughput in TB/s from algorithmic bytes (W_base +
packed signs + x + y per launch) over the HIP-event time of exactly `--steps`
steps, with all inputs resident in HBM.

Cache defeat: every launch reads its own (W_base, signs) buffer set; sets rotate
over more than twice the 256 MB Infinity Cache, so each launch streams its
operands from HBM.  Steps are replayed from a HIP graph (captured once) so host
launch overhead does not pace the GPU; after the `--warmup` eager steps the
graph is replayed three times untimed (its first launch also uploads it, and
the next one still ran slow coming out of idle), then the timed replay runs
exactly `--steps` steps.

Also reported (same run): the other workloads' throughput (multi-tenant decode,
prefill, LLaMA-7B-shaped 32-layer sweep) under "workloads", the dominant
kernel's roofline fraction, and the fp64 CPU oracle timed on a bounded sample
of the headline workload on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "binary-delta matmul TB/s (decode) & TFLOP/s (prefill), % of MI355X roofline"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 matrix peak, published
F16_PEAK_TFLOPS = 2500.0       # MI355X dense fp16 matrix peak, published
MALL_BYTES = 256 << 20


def algorithmic_bytes(M, N, K, tenants_used, y_bytes=2):
    """W_base + packed signs of the tenants read + x + y (alpha and ids: negligible)."""
    return N * K * 2 + tenants_used * N * (K // 32) * 4 + M * K * 2 + M * N * y_bytes


class Launcher:
    """Pre-marshalled C-ABI calls: each call() only passes stored pointers and the
    current stream to bitdelta_matmul (nothing else runs per call)."""

    def __init__(self, lib):
        self.lib = lib

    def matmul(self, x, w, packed, alpha, tid, y):
        import ctypes
        import torch
        import paper_2609_36800_amd as bd
        M, K = x.shape
        N = w.shape[0]
        T = alpha.numel()
        dt = bd.F16 if x.dtype == torch.float16 else bd.BF16
        args = (x.data_ptr(), M, K, w.data_ptr(), N, packed.data_ptr(), alpha.data_ptr(),
                None if tid is None else tid.data_ptr(), T, dt, y.data_ptr(), dt, bd.PATH_AUTO)
        f = self.lib.bitdelta_matmul_typed

        def call():
            rc = f(*args, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
            if rc != 0:
                raise RuntimeError(f"bitdelta_matmul failed: {rc}")
        return call


def make_sets(count, M, N, K, T, multi, seed, dev, prompts=0, dtype="bf16"):
    import workloads as wl
    sets = []
    for i in range(count):
        d = wl.device_problem(M, N, K, T, multi_tenant=multi, seed=seed + i, device=dev,
                              prompts=prompts, dtype=dtype)
        sets.append(d)
    return sets


def capture(calls, warmup_calls):
    """Run warmup_calls eagerly on the capture stream, then capture `calls`
    once into a HIP graph on it (falls back to eager replay if capture is
    unavailable).  Warming up on that stream lets the library make its
    per-stream workspace before capture, where it cannot allocate."""
    import torch
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        for c in warmup_calls:
            c()
    torch.cuda.synchronize()
    try:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.stream(s):
            g.capture_begin()
            for c in calls:
                c()
            g.capture_end()
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        return g.replay, True, g
    except Exception as e:  # graph capture unavailable: replay eagerly
        print(f"# graph capture failed ({e}); timing eager launches", file=sys.stderr)

        def eager():
            for c in calls:
                c()
        return eager, False, None


def upload(replay, times=3):
    """Untimed replays of a freshly captured graph before it is timed: its
    first launch also uploads the graph to the device (measured 20-130 us
    longer than later replays of the same steps), and the first replay after
    that still ran ~4% slow at the headline's 40 launches (the part coming out
    of idle); from the third on, replays time alike."""
    import torch
    for _ in range(times):
        replay()
    torch.cuda.synchronize()


def timed(replay, reps):
    import torch
    torch.cuda.synchronize()
    st = torch.cuda.Event(enable_timing=True)
    en = torch.cuda.Event(enable_timing=True)
    st.record()
    for _ in range(reps):
        replay()
    en.record()
    torch.cuda.synchronize()
    return st.elapsed_time(en) / 1e3  # seconds


def bench_workload(name, shapes, T, multi, flops_fn, steps, warmup, dev, launcher, seed,
                   rotate=True, prompts=0, dtype="bf16"):
    """Time exactly `steps` steps; a step is one launch per (M, N, K) in `shapes`.

    With rotate, consecutive launches read different buffer sets and the sets
    total more than twice the Infinity Cache.  The `steps` steps are captured
    into one graph and replayed once inside the timed region.
    """
    import numpy as np
    import torch
    est = sum(algorithmic_bytes(M, N, K, T) for (M, N, K) in shapes)
    nrot = max(2, -(-2 * MALL_BYTES // est)) if rotate else 1
    rot_calls, keep, rot_bytes = [], [], []
    for r in range(nrot):
        step_calls, b = [], 0
        for j, (M, N, K) in enumerate(shapes):
            d = make_sets(1, M, N, K, T, multi, seed + 1000 * j + r, dev, prompts, dtype)[0]
            y = torch.empty((M, N), dtype=d["x"].dtype, device=dev)
            used = 1 if d["tenant_ids"] is None else len(np.unique(d["tenant_ids"].cpu().numpy()))
            b += algorithmic_bytes(M, N, K, used)
            keep.append((d, y))
            step_calls.append(launcher.matmul(d["x"], d["w"], d["packed"], d["alpha"],
                                              d["tenant_ids"], y))
        rot_calls.append(step_calls)
        rot_bytes.append(b)
    calls = [c for i in range(steps) for c in rot_calls[i % nrot]]
    warm = [c for i in range(max(1, warmup)) for c in rot_calls[i % nrot]]
    replay, graphed, graph = capture(calls, warm)
    upload(replay)
    secs = timed(replay, 1)
    # the same graph replayed again: spread over repeats (the first timed replay
    # above is the one reported, exactly `steps` steps)
    reps = [secs] + [timed(replay, 1) for _ in range(REPEATS - 1)]
    total_bytes = sum(rot_bytes[i % nrot] for i in range(steps))
    sec_per_step = secs / steps
    flops = sum(flops_fn(*s) for s in shapes)
    res = {
        "workload": name, "steps": steps, "graphed": graphed, "buffer_sets": nrot * len(shapes),
        "ms_per_step": sec_per_step * 1e3, "bytes_per_step": total_bytes / steps,
        "TBps": total_bytes / secs / 1e12,
        "TFLOPs": flops * steps / secs / 1e12,
        "launches_per_step": len(shapes),
        "avg_launch_us": secs / (steps * len(shapes)) * 1e6,
        "repeats": spread([r / (steps * len(shapes)) * 1e6 for r in reps], "avg_launch_us"),
    }
    del keep, calls, warm, rot_calls, graph
    torch.cuda.empty_cache()
    return res


REPEATS = 5


def spread(values, what):
    """median / min / max of repeated measurements (the paper reports
    repeatability over five trials)."""
    import statistics
    return {"of": what, "n": len(values), "median": statistics.median(values),
            "min": min(values), "max": max(values)}


def hbm_roofline(bytes_per_launch, us_per_launch, kernel):
    gbs = bytes_per_launch / (us_per_launch * 1e-6) / 1e9
    return {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": gbs / HBM_PEAK_GBS, "kernel": kernel}


def mfma_roofline(flops_per_launch, us_per_launch, kernel, peak=BF16_PEAK_TFLOPS):
    tf = flops_per_launch / (us_per_launch * 1e-6) / 1e12
    return {"bound": "mfma", "achieved": tf, "peak": peak, "unit": "TFLOP/s",
            "frac": tf / peak, "kernel": kernel}


def llama_sweep(dev, launcher, warmup):
    """32 layers x 7 matrices, 8 tenants, 64 rows: one pass over ~19.7 GB."""
    import torch
    import workloads as wl
    import numpy as np
    g = torch.Generator(device=dev)
    g.manual_seed(1234)
    M, T = wl.LLAMA_ROWS, wl.LLAMA_TENANTS
    x4096 = torch.randn((M, 4096), generator=g, device=dev).to(torch.bfloat16)
    x11008 = torch.randn((M, 11008), generator=g, device=dev).to(torch.bfloat16)
    tid = torch.randint(0, T, (M,), generator=g, device=dev, dtype=torch.int32)
    used = len(np.unique(tid.cpu().numpy()))
    calls, per_matrix = [], {}
    keep = []
    total_bytes = 0
    for layer in range(wl.LLAMA_LAYERS):
        for idx, (name, N, K) in enumerate(wl.LLAMA_MATRICES):
            w = (torch.randn((N, K), generator=g, device=dev) * 0.02).to(torch.bfloat16)
            pk = torch.randint(0, 256, (T, N, K // 32, 4), generator=g, device=dev,
                               dtype=torch.uint8).view(torch.int32).reshape(T, N, K // 32)
            a = torch.rand((T,), generator=g, device=dev) * 9e-4 + 1e-4
            y = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
            x = x4096 if K == 4096 else x11008
            keep.append((w, pk, a, y))
            calls.append(launcher.matmul(x, w, pk, a, tid, y))
            b = algorithmic_bytes(M, N, K, used)
            per_matrix.setdefault(name, {"N": N, "K": K, "bytes": b})
            total_bytes += b
    replay, graphed, graph = capture(calls, calls)
    upload(replay)
    passes = [timed(replay, 1) for _ in range(REPEATS)]
    secs = sorted(passes)[len(passes) // 2]
    # per-matrix-type time: time each type's 32 launches on its own
    for name in per_matrix:
        idxs = [i for i, c in enumerate(calls) if wl.LLAMA_MATRICES[i % 7][0] == name]
        sub = [calls[i] for i in idxs]
        r, _, g2 = capture(sub, sub)
        t = timed(r, 3) / 3 / len(sub)
        del g2
        per_matrix[name]["us"] = t * 1e6
        per_matrix[name]["TBps"] = per_matrix[name]["bytes"] / t / 1e12
        per_matrix[name]["roofline"] = hbm_roofline(per_matrix[name]["bytes"], t * 1e6,
                                                    "batched decode (64 rows, 8 tenants)")
    del keep, calls, graph
    torch.cuda.empty_cache()
    return {"workload": "LLaMA-7B-shaped sweep: 32 layers x {q,k,v,o,gate,up,down}, 8 tenants, "
                        "64 rows", "graphed": graphed, "tenants_used": used,
            "ms_per_pass": secs * 1e3, "bytes_per_pass": total_bytes,
            "TBps": total_bytes / secs / 1e12,
            "repeats": spread([p * 1e3 for p in passes], "ms_per_pass"),
            "roofline": hbm_roofline(total_bytes, secs * 1e6, "batched decode (64 rows, 8 tenants), "
                                     "224 launches"),
            "per_matrix": per_matrix}


def decode_size_sweep(dev, launcher, warmup):
    """The streaming decode kernel (M = 1, K = 4096) at four launch sizes,
    N = 4096 .. 32768 (36 .. 290 MB of W and signs per launch), each on buffer
    sets rotating over more than twice the Infinity Cache.  A least-squares line
    time = fixed + bytes / rate separates the per-launch ramp and drain from the
    streaming rate, which is what bounds one 36 MB launch."""
    pts = []
    for N in (4096, 8192, 16384, 32768):
        r = bench_workload(f"decode M=1, N={N}", [(1, N, 4096)], 1, False,
                           lambda M, N_, K: 2 * M * N_ * K, 40, warmup, dev, launcher, seed=700 + N)
        pts.append({"N": N, "bytes": r["bytes_per_step"], "us": r["avg_launch_us"], "TBps": r["TBps"]})
    xs = [p["bytes"] for p in pts]
    ys = [p["us"] for p in pts]
    mx, my = sum(xs) / len(xs), sum(ys) / len(ys)
    slope = sum((a - mx) * (b - my) for a, b in zip(xs, ys)) / sum((a - mx) ** 2 for a in xs)
    fixed = my - slope * mx
    return {"workload": "decode launch-size sweep: x 1x4096, W_base N x 4096, N = 4096 .. 32768",
            "points": pts, "fit": {"fixed_us": fixed, "asymptotic_GBps": 1e-3 / slope}}


def bench_compress(dev, lib, steps, warmup):
    """Delta compression of LLaMA-7B-gate-shaped weights (11008x4096 bf16 fine and
    base -> packed signs, per-row |delta| sums, scale), buffer sets rotating over
    more than twice the Infinity Cache.  HBM-bound: 4 bytes read per weight."""
    import ctypes
    import torch
    import paper_2609_36800_amd as bd
    rows, K = 11008, 4096
    per = rows * K * 4 + rows * K // 8 + rows * 4 + 4
    nsets = max(2, -(-2 * MALL_BYTES // per))
    g = torch.Generator(device=dev)
    g.manual_seed(77)
    sets = []
    for _ in range(nsets):
        base = (torch.randn((rows, K), generator=g, device=dev) * 0.02).to(torch.bfloat16)
        fine = (base.float() + torch.randn((rows, K), generator=g, device=dev) * 1e-3).to(torch.bfloat16)
        packed = torch.empty((rows, K // 32), dtype=torch.int32, device=dev)
        row_abs = torch.empty((rows,), dtype=torch.float32, device=dev)
        alpha = torch.empty((1,), dtype=torch.float32, device=dev)
        sets.append((fine, base, packed, row_abs, alpha))
    f = lib.bitdelta_compress

    def call_for(st):
        fine, base, packed, row_abs, alpha = st
        args = (fine.data_ptr(), base.data_ptr(), rows, K, bd.BF16, packed.data_ptr(),
                row_abs.data_ptr(), alpha.data_ptr())

        def c():
            rc = f(*args, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
            if rc != 0:
                raise RuntimeError(f"bitdelta_compress failed: {rc}")
        return c
    calls = [call_for(sets[i % nsets]) for i in range(steps)]
    warm = [call_for(sets[i % nsets]) for i in range(max(1, warmup))]
    replay, graphed, graph = capture(calls, warm)
    upload(replay)
    secs = timed(replay, 1)
    reps = [secs] + [timed(replay, 1) for _ in range(REPEATS - 1)]
    del graph, sets
    torch.cuda.empty_cache()
    return {"workload": "delta compression: W_fine, W_base 11008x4096 bf16 -> packed signs, "
                        "per-row |delta| sums and the least-squares scale",
            "steps": steps, "graphed": graphed, "buffer_sets": nsets,
            "us_per_call": secs / steps * 1e6, "bytes_per_call": per,
            "TBps": per * steps / secs / 1e12,
            "repeats": spread([r / steps * 1e6 for r in reps], "us_per_call"),
            "roofline": hbm_roofline(per, secs / steps * 1e6, "compress_kernel + mean_kernel")}


def context_ceilings(dev, warmup):
    """Reference points measured in the same run with library kernels (not this
    library's): torch's elementwise negation kernel (one buffer read, another
    written), as a bandwidth ceiling for a large transfer and for one transfer of
    the decode launch's size (36 MB read + 36 MB written, buffers rotating over
    more than twice the Infinity Cache), torch's sum reading 36 MB per launch
    (a read-only ceiling at the decode launch's size), and torch.matmul's
    plain bf16 GEMM at 4096^3 (no decode), the matrix-core reference for the fused
    prefill.  Context only: none of them is a figure of this library."""
    import torch

    def time_calls(calls, reps):
        replay, graphed, graph = capture(calls, calls[:max(1, warmup)])
        upload(replay)
        secs = timed(replay, reps) / (reps * len(calls))
        del graph
        return secs, graphed

    out = {}
    big = 256 << 20                                   # bf16 elements: 512 MiB
    a = torch.empty(big, dtype=torch.bfloat16, device=dev).fill_(1.0)
    b = torch.empty_like(a)
    secs, graphed = time_calls([lambda: torch.neg(a, out=b)] * 8, 2)
    out["elementwise_copy_512MiB"] = {"us": secs * 1e6, "GBps": 2 * a.numel() * 2 / secs / 1e9,
                          "bytes": 2 * a.numel() * 2, "graphed": graphed}
    del a, b
    n36 = 4096 * 4096 + 4096 * 128 * 2              # the decode launch's W + signs, in bf16 elements
    sets = [(torch.empty(n36, dtype=torch.bfloat16, device=dev).fill_(1.0),
             torch.empty(n36, dtype=torch.bfloat16, device=dev)) for _ in range(16)]
    calls = [(lambda s=s: torch.neg(s[0], out=s[1])) for s in sets] * 4
    secs, graphed = time_calls(calls, 1)
    out["elementwise_copy_36MB"] = {"us": secs * 1e6, "GBps": 2 * n36 * 2 / secs / 1e9, "bytes": 2 * n36 * 2,
                        "graphed": graphed, "buffer_sets": len(sets)}
    del sets, calls
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    x = torch.randn((4096, 4096), generator=g, device=dev).to(torch.bfloat16)
    wt = (torch.randn((4096, 4096), generator=g, device=dev) * 0.02).to(torch.bfloat16).t().contiguous()
    y = torch.empty((4096, 4096), dtype=torch.bfloat16, device=dev)
    secs, graphed = time_calls([lambda: torch.matmul(x, wt, out=y)] * 10, 2)
    fl = 2.0 * 4096 ** 3
    out["torch_matmul_bf16_4096"] = {"us": secs * 1e6, "TFLOPs": fl / secs / 1e12,
                                     "frac_of_bf16_peak": fl / secs / 1e12 / BF16_PEAK_TFLOPS,
                                     "graphed": graphed}
    del x, wt, y
    torch.cuda.empty_cache()
    return out


def cpu_model() -> str:
    """The host CPU's model name as the kernel reports it (empty if unknown)."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return ""


def cpu_baseline(budget_s: float):
    """fp64 oracle timed on the headline workload (the M = 1 and M = 16 pair
    against one 4096x4096 matrix), repeated until about budget_s seconds."""
    import oracle
    import workloads as wl
    p1 = wl.decode(1, seed=0)
    p16 = wl.make_problem(16, 4096, 4096, 1, seed=0)
    p16.w, p16.packed, p16.alpha = p1.w, p1.packed, p1.alpha
    b = algorithmic_bytes(1, 4096, 4096, 1) + algorithmic_bytes(16, 4096, 4096, 1)
    reps, secs = 0, 0.0
    while secs < budget_s and reps < 1000:
        t0 = time.perf_counter()
        oracle.matmul(p1.x, p1.w, p1.packed, p1.alpha)
        oracle.matmul(p16.x, p16.w, p16.packed, p16.alpha)
        secs += time.perf_counter() - t0
        reps += 1
    return {"value": reps * b / secs / 1e12, "unit": "TB/s", "cores": oracle.num_threads(),
            "kind": "oracle", "host_cpus": len(os.sched_getaffinity(0)), "cpu_model": cpu_model(),
            "sample": f"full decode pair (M=1 and M=16, N=K=4096, {b} algorithmic bytes per "
                      f"pass), {reps} passes in {secs:.2f} s, fp64 with OpenMP over features",
            "seconds": secs}


def cpu_baselines():
    """The fp64 oracle on each workload, timed once on this host (wall time,
    fp64 GFLOP/s counting 4*M*N*K for the base and delta sums).  Configs whose
    oracle run takes seconds are timed in full; the 32-layer sweep by one
    matrix of each type (k, v, o run like q; up like gate)."""
    import oracle
    import workloads as wl
    out = []

    def run(name, p, sample):
        t0 = time.perf_counter()
        oracle.matmul(p.x, p.w, p.packed, p.alpha, p.tenant_ids)
        secs = time.perf_counter() - t0
        flops = 4.0 * p.M * p.N * p.K
        out.append({"workload": name, "sample": sample, "seconds": secs,
                    "GFLOPs_fp64": flops / secs / 1e9, "cores": oracle.num_threads(),
                    "cpu_model": cpu_model(), "kind": "oracle"})

    t = wl.tiny(seed=0)
    t.packed = oracle.pack(t.signs[0])[None]
    run("tiny 4x256 . 512x256 (fp32 out)", t, "full")
    run("decode M=1, 4096x4096", wl.decode(1, seed=0), "full")
    run("decode M=16, 4096x4096", wl.decode(16, seed=0), "full")
    run("multi-tenant decode 32 rows x 11008x4096, 16 tenants", wl.mt_decode(seed=0), "full")
    run("prefill 4096x4096x4096", wl.prefill(seed=0), "full")
    run("multi-tenant prefill 4096 rows (16 prompts, 8 tenants) x 4096x4096", wl.mt_prefill(seed=0), "full")
    shared = wl.llama_shared_inputs(seed=0)
    for idx, (name, N, K) in enumerate(wl.LLAMA_MATRICES):
        if name in ("q", "gate", "down"):
            run(f"LLaMA-7B-shaped sweep, {name} ({N}x{K}, 64 rows, 8 tenants)",
                wl.llama_matrix(0, idx, shared=shared),
                "one matrix of the 224 (layer 0); the others of its type have its shape")
    return out


PAPER_CONTEXT = {
    "note": "context only, not a target: speedups the paper reports for its generated "
            "BitDelta kernels over autotuned Triton, measured on an NVIDIA GPU; this run "
            "reports absolute throughput against MI355X peaks",
    "bitdelta_standard_speedup_vs_triton": 3.34,
    "bitdelta_batched_speedup_vs_triton": 2.51,
    "baseline": "autotuned Triton 3.6.0",
    "hardware": "NVIDIA B200 (Blackwell, sm_100a)",
    "precision": "FP16",
    "source": "Section 4.4 (recently published kernels) and Appendix A.2 (BitDelta)",
}


def code_text(src: str) -> str:
    """C/C++ source without comments and with whitespace runs collapsed, so
    that editing a comment does not change the hash of the code."""
    import re
    src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
    src = re.sub(r"//[^\n]*", " ", src)
    return " ".join(src.split())


def kernel_source_hash(read=None):
    """Hash of the dominant kernel's code (comments excluded): a recorded
    traffic figure is only valid for the kernel it was measured on.  `read`
    maps a file name to its text (default: the files in this tree)."""
    import hashlib
    h = hashlib.sha256()
    for f in ("decode.hip", "device.h", "ldscopy.h"):
        if read is None:
            with open(os.path.join(ROOT, "paper_2609_36800_amd", "csrc", f)) as fh:
                text = fh.read()
        else:
            text = read(f)
        h.update(code_text(text).encode())
    return h.hexdigest()[:16]


def recorded_traffic():
    """HBM bytes per launch from the committed counter summary, if it was taken
    on the current kernel source (else None)."""
    path = os.path.join(ROOT, "profiles", "decode_gemv_4096x4096_traffic.json")
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def pmc_pass(steps, workload="decode"):
    """Launches for counter collection.  decode: the headline pair on rotating
    buffer sets, then a plain device copy of 512 MiB whose FETCH_SIZE /
    WRITE_SIZE readings calibrate the counters (known bytes read and written).
    prefill: `steps` launches each of the bf16 and fp16 4096^3 fused GEMM.
    multi: `steps` launches of the batched kernel at 64 rows, 8 tenants,
    4096x4096, on 12 rotating buffer sets.  mtdecode: `steps` launches of the
    multi-tenant decode workload (32 rows, 16 tenants, 11008x4096) on 4
    rotating buffer sets, with the distinct tenants of each set printed.  gate:
    the same at the LLaMA-shaped sweep's gate / up shape (64 rows, 8 tenants,
    11008x4096)."""
    import torch
    import paper_2609_36800_amd as bd
    dev = torch.device("cuda:0")
    launcher = Launcher(bd.load_library())
    if workload in ("mtdecode", "gate"):
        M, T = (32, 16) if workload == "mtdecode" else (64, 8)
        calls, keep, distinct = [], [], []
        for r in range(4):
            d = make_sets(1, M, 11008, 4096, T, True, 21 + r, dev)[0]
            y = torch.empty((M, 11008), dtype=torch.bfloat16, device=dev)
            keep.append((d, y))
            distinct.append(int(torch.unique(d["tenant_ids"]).numel()))
            calls.append(launcher.matmul(d["x"], d["w"], d["packed"], d["alpha"],
                                         d["tenant_ids"], y))
        for i in range(steps):
            calls[i % len(calls)]()
        torch.cuda.synchronize()
        print(json.dumps({"pmc_pass": workload, "launches": steps, "distinct_tenants": distinct}),
              flush=True)
        return
    if workload in ("prefill", "multi"):
        calls, keep = [], []
        if workload == "prefill":
            for dt in ("bf16", "f16"):
                d = make_sets(1, 4096, 4096, 4096, 1, False, 3, dev, dtype=dt)[0]
                y = torch.empty((4096, 4096), dtype=d["x"].dtype, device=dev)
                keep.append((d, y))
                calls += [launcher.matmul(d["x"], d["w"], d["packed"], d["alpha"], None, y)] * steps
        else:
            for r in range(12):
                d = make_sets(1, 64, 4096, 4096, 8, True, 5 + r, dev)[0]
                y = torch.empty((64, 4096), dtype=torch.bfloat16, device=dev)
                keep.append((d, y))
                calls.append(launcher.matmul(d["x"], d["w"], d["packed"], d["alpha"],
                                             d["tenant_ids"], y))
            calls = [calls[i % len(calls)] for i in range(steps)]
        for c in calls:
            c()
        torch.cuda.synchronize()
        print(json.dumps({"pmc_pass": workload, "launches": len(calls)}), flush=True)
        return
    calls = []
    keep = []
    for r in range(8):
        for j, M in enumerate((1, 16)):
            d = make_sets(1, M, 4096, 4096, 1, False, 1 + 1000 * j + r, dev)[0]
            y = torch.empty((M, 4096), dtype=torch.bfloat16, device=dev)
            keep.append((d, y))
            calls.append(launcher.matmul(d["x"], d["w"], d["packed"], d["alpha"], None, y))
    for i in range(steps):
        calls[i % len(calls)]()
    torch.cuda.synchronize()
    src = torch.empty(512 << 20, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"pmc_pass": True, "launches": steps, "copy_bytes": src.numel(),
                      "kernel_source_hash": kernel_source_hash()}), flush=True)


def traffic_from(fetch_dir, write_dir, out_path):
    """Turn the two rocprofv3 --pmc runs of `--pmc-pass` (FETCH_SIZE, then
    WRITE_SIZE, in KiB per dispatch) into HBM bytes per headline launch.  Each
    counter is scaled by what it reads for the 512 MiB calibration copy that
    the same run performs (known bytes read and written)."""
    import csv
    import glob
    import statistics

    def per_dispatch(d, counter):
        vals, names = {}, {}
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                if r["Counter_Name"] != counter:
                    continue
                key = r["Dispatch_Id"]
                vals[key] = vals.get(key, 0.0) + float(r["Counter_Value"])
                names[key] = r["Kernel_Name"]
        return vals, names

    copy_bytes = 512 << 20
    out = {}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        vals, names = per_dispatch(d, counter)
        lib = [v for k, v in vals.items() if "bitdelta" in names[k] and "decode" in names[k]]
        copies = [v for k, v in vals.items() if "bitdelta" not in names[k] and v * 1024 > copy_bytes / 4]
        if not lib or not copies:
            raise SystemExit(f"{counter}: no library or calibration-copy dispatches found in {d}")
        raw = statistics.mean(lib)
        scale = copy_bytes / (statistics.median(copies[-3:]) * 1024)
        out[counter] = (raw, scale)
    hbm = out["FETCH_SIZE"][0] * 1024 * out["FETCH_SIZE"][1] + out["WRITE_SIZE"][0] * 1024 * out["WRITE_SIZE"][1]
    alg = (algorithmic_bytes(1, 4096, 4096, 1) + algorithmic_bytes(16, 4096, 4096, 1)) / 2
    rec = {
        "kernel": "stream_decode_kernel (M=1 and M=16 launches alternating, N=K=4096)",
        "kernel_source_hash": kernel_source_hash(),
        "fetch_kib_per_launch_raw": round(out["FETCH_SIZE"][0], 1),
        "write_kib_per_launch_raw": round(out["WRITE_SIZE"][0], 1),
        "fetch_scale_from_copy": round(out["FETCH_SIZE"][1], 4),
        "write_scale_from_copy": round(out["WRITE_SIZE"][1], 4),
        "hbm_bytes_per_launch": int(round(hbm)),
        "algorithmic_bytes_per_launch": alg,
        "commands": [
            "rocprofv3 --pmc FETCH_SIZE --output-format csv -d <fetch_dir> -o run -- python3 bench.py --pmc-pass --steps 64",
            "rocprofv3 --pmc WRITE_SIZE --output-format csv -d <write_dir> -o run -- python3 bench.py --pmc-pass --steps 64",
            "python3 bench.py --traffic-from <fetch_dir> <write_dir>",
        ],
    }
    with open(out_path, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--only-headline", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-budget", type=float, default=10.0)
    ap.add_argument("--pmc-pass", action="store_true",
                    help="only launch the headline kernels and a calibration copy (for rocprofv3 --pmc)")
    ap.add_argument("--pmc-workload", choices=("decode", "prefill", "multi", "mtdecode", "gate"), default="decode",
                    help="what --pmc-pass launches")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="write the HBM traffic record from two --pmc runs of --pmc-pass (no GPU needed)")
    args = ap.parse_args()

    if args.traffic_from:
        traffic_from(args.traffic_from[0], args.traffic_from[1],
                     os.path.join(ROOT, "profiles", "decode_gemv_4096x4096_traffic.json"))
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(the operator would shard along output features with no exchange).",
              file=sys.stderr)
        sys.exit(2)

    if args.pmc_pass:
        pmc_pass(args.steps, args.pmc_workload)
        return

    import torch
    import paper_2609_36800_amd as bd

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    launcher = Launcher(bd.load_library())

    head = bench_workload(
        "single-tenant decode GEMV pair: x 1x4096 and 16x4096, W_base 4096x4096, "
        "one packed 4096x4096 sign matrix, bf16 out",
        [(1, 4096, 4096), (16, 4096, 4096)], 1, False, lambda M, N, K: 2 * M * N * K,
        args.steps, args.warmup, dev, launcher, seed=1)

    avg_launch_s = head["avg_launch_us"] / 1e6
    per_launch_bytes = head["bytes_per_step"] / head["launches_per_step"]
    achieved = per_launch_bytes / avg_launch_s / 1e9
    roofline = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS, "traffic": recorded_traffic(),
                "kernel": "stream_decode_kernel (single tenant, M <= 16)",
                "per_launch_bytes": per_launch_bytes,
                "avg_launch_us": head["avg_launch_us"]}

    head["roofline"] = hbm_roofline(per_launch_bytes, head["avg_launch_us"], roofline["kernel"])
    workloads = [head]
    if not args.only_headline:
        mt = bench_workload(
            "multi-tenant decode: x 32x4096 (tenant id per row, 16 tenants), W_base 11008x4096",
            [(32, 11008, 4096)], 16, True, lambda M, N, K: 2 * M * N * K,
            100, args.warmup, dev, launcher, seed=50)
        mt["roofline"] = hbm_roofline(mt["bytes_per_step"], mt["avg_launch_us"],
                                      "batched decode (32 rows, 16 tenants)")
        workloads.append(mt)
        pf = bench_workload(
            "prefill: x 4096x4096, W_base 4096x4096, one tenant, fused bf16 GEMM",
            [(4096, 4096, 4096)], 1, False, lambda M, N, K: 2 * M * N * K,
            20, args.warmup, dev, launcher, seed=90, rotate=False)
        pf["mfma_frac"] = pf["TFLOPs"] / BF16_PEAK_TFLOPS
        pf["roofline"] = mfma_roofline(2.0 * 4096 ** 3, pf["avg_launch_us"], "prefill_stream_kernel (bf16)")
        workloads.append(pf)
        import workloads as wl
        c = wl.MT_PREFILL
        mpf = bench_workload(
            "multi-tenant prefill: x 4096x4096 as 16 prompts of random length, one tenant per "
            "prompt drawn from 8, W_base 4096x4096, grouped fused bf16 GEMM",
            [(c["M"], c["N"], c["K"])], c["T"], True, lambda M, N, K: 2 * M * N * K,
            20, args.warmup, dev, launcher, seed=130, rotate=False, prompts=c["prompts"])
        mpf["mfma_frac"] = mpf["TFLOPs"] / BF16_PEAK_TFLOPS
        mpf["roofline"] = mfma_roofline(2.0 * c["M"] * c["N"] * c["K"], mpf["avg_launch_us"],
                                        "prefill_stream_kernel, grouped form (bf16)")
        workloads.append(mpf)
        # the paper's own precision: the same decode pair and prefill with fp16 x and W
        d16 = bench_workload(
            "fp16 decode GEMV pair: x 1x4096 and 16x4096, W_base 4096x4096 (fp16), fp16 out",
            [(1, 4096, 4096), (16, 4096, 4096)], 1, False, lambda M, N, K: 2 * M * N * K,
            args.steps, args.warmup, dev, launcher, seed=301, dtype="f16")
        d16["roofline"] = hbm_roofline(d16["bytes_per_step"] / 2, d16["avg_launch_us"],
                                       "stream_decode_kernel (fp16)")
        workloads.append(d16)
        pf16 = bench_workload(
            "fp16 prefill: x 4096x4096, W_base 4096x4096 (fp16), one tenant, fused fp16 GEMM",
            [(4096, 4096, 4096)], 1, False, lambda M, N, K: 2 * M * N * K,
            20, args.warmup, dev, launcher, seed=390, rotate=False, dtype="f16")
        pf16["mfma_frac"] = pf16["TFLOPs"] / F16_PEAK_TFLOPS
        pf16["roofline"] = mfma_roofline(2.0 * 4096 ** 3, pf16["avg_launch_us"],
                                         "prefill_stream_kernel (fp16)", F16_PEAK_TFLOPS)
        workloads.append(pf16)
        workloads.append(llama_sweep(dev, launcher, args.warmup))
        workloads.append(bench_compress(dev, launcher.lib, 50, args.warmup))
        sweep = decode_size_sweep(dev, launcher, args.warmup)
        workloads.append(sweep)
        context = context_ceilings(dev, args.warmup)
        # the same-run read ceiling for one launch of the headline's size: a
        # library copy moving the decode launch's W + signs in and the same out
        cop = context["elementwise_copy_36MB"]["GBps"]
        roofline["same_run_copy_ceiling"] = {
            "GBps": cop, "what": "torch elementwise copy, 36 MB read + 36 MB written per launch, "
                                 "16 rotating buffer pairs", "frac_of_ceiling": achieved / cop}
        fit = sweep["fit"]
        roofline["launch_size_fit"] = {
            "what": "the same decode kernel (M=1, K=4096) timed at N = 4096 .. 32768 (36 .. 290 MB per "
                    "launch); least-squares time = fixed_us + bytes / asymptotic rate",
            "fixed_us": fit["fixed_us"], "asymptotic_GBps": fit["asymptotic_GBps"],
            "frac_of_asymptote_at_headline_size": achieved / fit["asymptotic_GBps"]}
    else:
        context = {}
    context["paper"] = PAPER_CONTEXT

    cpu = None if args.no_cpu else cpu_baseline(args.cpu_budget)
    cpu_per_config = None if (args.no_cpu or args.only_headline) else cpu_baselines()

    out = {
        "metric": METRIC, "value": head["TBps"], "unit": "TB/s", "n_gpus": 1,
        "steps": head["steps"], "warmup": args.warmup, "ms_per_step": head["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": head["workload"], "global_batch": 17, "K": 4096, "N": 4096,
                   "parallelism": "none (1 GPU)"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "cpu_baseline_per_config": cpu_per_config,
        "workloads": workloads,
        "context": context,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
