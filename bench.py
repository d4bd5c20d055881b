#!/usr/bin/env python3
"""Benchmark of the fused causal attention hot path on one MI355X.

A step is one forward (O, LSE) plus one backward (dQ + D, then dK, dV) over the
GPT-2-small attention workload, bf16, B=8 H=12 S=1024 D=64, causal, scale 1/8,
with every input already resident in HBM.  Throughput is the counted causal
FLOPs of the step (forward 2*B*H*S^2*D, backward 5*B*H*S^2*D) over the wall
time of exactly --steps steps, bracketed by device synchronisations.

The same timed region also records HIP events around each kernel, on the
stream the kernels run on, on every 8th step (--event-every; at least 8 steps
are sampled); the slowest kernel's mean duration over those launches gives the
roofline entry, beside the same kernel's mean duration in the committed
rocprofv3 kernel trace.  After the timed region the step is timed again
--repeats times (median reported) and with the last-level cache evicted before
each step (--cold), and every workload (the tiny float32 one, GPT-2 small/medium, XL
width, long context, and GPT-2 small stored [B, S, H, D]) is timed too --
forward, backward and whole step -- under "configs", and shapes across the
paper's attention sweep under "sweep", the fused loss head under "lmhead" and
the memory-bound operators (LayerNorm, GELU, softmax cross entropy, forward
and backward, with their HBM bandwidth) under "memops" (--configs 0 skips
all of these).  On
rank 0 the float64 CPU oracle is then timed on a bounded sample of the same
workload (whole (batch, head) slices) as a reported baseline.  Prints ONE JSON
line.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "causal attention fwd+bwd TFLOP/s (bf16, 1 MI355X) at B8 H12 S1024 D64; % MFMA peak"
DEFAULT_WORKLOAD = "gpt2_small_B8_H12_S1024_D64"
# MI355X dense matrix-core peaks (TFLOP/s): 256 CUs x 2.4 GHz x FLOP/clock/CU
PEAK_TFLOPS = {"bf16": 2516.6, "f32": 157.3}
HBM_PEAK_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2608_00029_amd", "csrc")


# Sources the attention kernels are compiled from (the loss head and the
# memory-bound operators live in other files and do not change them).
ATTN_SOURCES = ("attn_bf16.hip", "attn_fwd.hip", "attn_bwd.hip", "attn_device.h", "attn_sched.h", "attn_launch.h",
                "bf16_stream.h")


def kernel_source_digest(names=ATTN_SOURCES) -> str:
    """sha256 over the attention kernels' sources (names and bytes), so that a
    stored counter measurement can be tied to the kernels it was taken on."""
    h = hashlib.sha256()
    for p in sorted(os.path.join(CSRC, n) for n in names):
        h.update(os.path.basename(p).encode())
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    rocprofv3 counter summary (FETCH_SIZE and WRITE_SIZE, each scaled by the
    factor a plain copy of known size gives), or None when there is no such
    summary or the kernel sources changed since the counters were taken."""
    path = os.path.join(PROFILES, f"hbm_traffic_{workload}.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.lstrip().startswith("#"):
                key, val = line.split(":", 1)
                fields[key.strip()] = val.strip()
    if fields.get("kernel_sources_sha256") != kernel_source_digest():
        return None
    val = fields.get(f"{kernel}.traffic_bytes_per_launch")
    return int(float(val)) if val else None


def kernel_flops(w):
    """Algorithmic FLOPs per launch of each kernel: 2*D per contraction per
    visible (query, key) pair, B*H*S^2/2 pairs when causal (B*H*S^2 if not).
    forward: 2 contractions (Q K^T, P V); dq kernel: 3 (Q K^T, dO V^T, dS K);
    dk/dv kernel: 4 (Q K^T, dO V^T, P^T dO, dS^T Q)."""
    pairs = w.B * w.H * w.S * w.S * (0.5 if w.causal else 1.0)
    per = 2.0 * w.D * pairs
    return {"attn_fwd": 2 * per, "attn_bwd_dq": 3 * per, "attn_bwd_dkdv": 4 * per}


def cpu_baseline(w, inputs, budget_s: float):
    """Time the float64 oracle (as it stands) on whole (batch, head) slices of
    the workload until about `budget_s` seconds have been spent."""
    import oracle.attn_oracle as orc
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = len(os.sched_getaffinity(0))
    q, k, v, do = inputs
    heads = [(b, h) for b in range(w.B) for h in range(w.H)]
    done = 0
    t0 = time.perf_counter()
    for b, h in heads:
        sl = lambda t: t[b:b + 1, h:h + 1]  # noqa: E731
        orc.attn_fwd(sl(q), sl(k), sl(v), w.scale, w.causal)
        orc.attn_bwd(sl(q), sl(k), sl(v), sl(do), w.scale, w.causal)
        done += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    fwd_f, bwd_f = w.counted_flops()
    per_head = (fwd_f + bwd_f) / (w.B * w.H)
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), cpu_model)
    except OSError:
        pass
    return {"value": round(per_head * done / dt / 1e12, 6), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle", "cpu_model": cpu_model,
            "sample": f"{done} of {w.B * w.H} (batch, head) slices of {w.name}, fwd+bwd in float64, "
                      f"{dt:.1f} s wall"}


def time_workload(w, bd, steps: int, warmup: int, layout: str = "bhsd"):
    """Forward, backward (dQ then dK/dV) and whole-step times of one workload,
    inputs resident in HBM: mean ms over `steps` launches of each, timed with
    HIP events on the stream the kernels run on.  layout "bshd" stores the
    tensors [B, S, H, D] (read and written in place by the kernels)."""
    import ctypes
    import torch
    from paper_2608_00029_amd.workloads import workload_inputs
    dev = torch.device("cuda:0")
    q, k, v, do = (t.to(dev) for t in workload_inputs(w))
    if layout == "bshd":
        q, k, v, do = (t.transpose(1, 2).contiguous() for t in (q, k, v, do))
    o = torch.empty_like(q)
    lse = torch.empty((w.B, w.H, w.S), dtype=torch.float32, device=dev)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
    ws = torch.empty((bd.workspace_bytes(w.B, w.H, w.S, w.D) // 4,), dtype=torch.float32, device=dev)
    L = bd.lib()
    stream = torch.cuda.current_stream(dev)
    lay = bd.CATTN_BSHD if layout == "bshd" else bd.CATTN_BHSD
    shape = (w.B, w.H, w.S, w.D, float(w.scale), int(w.causal), bd.CATTN_BF16 if w.dtype == "bf16" else bd.CATTN_F32,
             lay, ctypes.c_void_p(stream.cuda_stream))
    P = lambda t: t.data_ptr()  # noqa: E731

    def fwd():
        return L.cattn_attn_fwd_ex(P(q), P(k), P(v), P(o), P(lse), *shape)

    def bwd():
        return L.cattn_attn_bwd_ex(P(q), P(k), P(v), P(o), P(do), P(lse), P(dq), P(dk), P(dv), P(ws), *shape)

    for _ in range(warmup):
        if fwd() != 0 or bwd() != 0:
            raise RuntimeError(f"{w.name}: {bd.last_error_string()}")
    out = {}
    for name, fs in (("fwd", (fwd,)), ("bwd", (bwd,)), ("step", (fwd, bwd))):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            for f in fs:
                f()
        e1.record(stream)
        torch.cuda.synchronize()
        out[name] = e0.elapsed_time(e1) / steps
    fwd_f, bwd_f = w.counted_flops()
    return {"fwd_ms": round(out["fwd"], 5), "bwd_ms": round(out["bwd"], 5), "step_ms": round(out["step"], 5),
            "fwd_tflops": round(fwd_f / (out["fwd"] * 1e-3) / 1e12, 2),
            "bwd_tflops": round(bwd_f / (out["bwd"] * 1e-3) / 1e12, 2),
            "step_tflops": round((fwd_f + bwd_f) / (out["step"] * 1e-3) / 1e12, 2),
            "pct_peak": round(100.0 * (fwd_f + bwd_f) / (out["step"] * 1e-3) / 1e12 / PEAK_TFLOPS[w.dtype], 2)}


def time_lmhead(wl, bd, steps: int, warmup: int):
    """The fused loss head (projection with per-tile softmax statistics, merge,
    mean) at one shape, inputs resident in HBM: mean ms per call over `steps`
    calls, timed with HIP events on the stream the kernels run on.  Algorithmic
    work: 2*M*N*K FLOPs; bytes: X and W read once, float32 logits written once,
    the partials written and read once, LSE and the row losses written."""
    import ctypes
    import torch
    from paper_2608_00029_amd.workloads import make_lmhead_inputs
    dev = torch.device("cuda:0")
    x, w, y = (t.to(dev) for t in make_lmhead_inputs(wl.M, wl.N, wl.K, wl.w_sigma, wl.seed))
    z = torch.empty((wl.M, wl.N), dtype=torch.float32, device=dev)
    lse, rl = (torch.empty((wl.M,), dtype=torch.float32, device=dev) for _ in range(2))
    loss = torch.empty((1,), dtype=torch.float32, device=dev)
    ws = torch.empty((bd.lmhead_workspace_bytes(wl.M, wl.N, wl.K) // 4,), dtype=torch.float32, device=dev)
    L = bd.lib()
    stream = torch.cuda.current_stream(dev)
    sp = ctypes.c_void_p(stream.cuda_stream)
    args = [t.data_ptr() for t in (x, w, y, z, lse, rl, loss, ws)]

    def call():
        st = L.cattn_lmhead_fwd(*args, wl.M, wl.N, wl.K, sp)
        if st != 0:
            raise RuntimeError(f"{wl.name}: {bd.last_error_string()}")

    for _ in range(warmup):
        call()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(steps):
        call()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    flops = 2.0 * wl.M * wl.N * wl.K
    nbytes = 2 * (wl.M + wl.N) * wl.K + 4 * wl.M * wl.N + 2 * 8 * wl.M * (wl.N // 64) + 4 * 3 * wl.M
    return {"M": wl.M, "N": wl.N, "K": wl.K, "ms": round(ms, 5), "tflops": round(flops / (ms * 1e-3) / 1e12, 2),
            "pct_mfma_peak": round(100.0 * flops / (ms * 1e-3) / 1e12 / PEAK_TFLOPS["bf16"], 2),
            "hbm_gbs_algorithmic": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "floor_us": {"mfma": round(flops / (PEAK_TFLOPS["bf16"] * 1e12) * 1e6, 1),
                         "hbm": round(nbytes / (HBM_PEAK_GBS * 1e9) * 1e6, 1)}}


def time_memops(wl, bd, steps: int, warmup: int):
    """One memory-bound operator (LayerNorm, GELU or softmax cross entropy) at
    the paper's shape, forward and backward, inputs resident in HBM: mean ms per
    call over `steps` calls each, timed with HIP events on the stream the
    kernels run on.  Bandwidth is reported twice: over the algorithmic bytes
    (every input read once, every output written once, workspace partials
    written and read once) against the 8 TB/s HBM peak, and over the paper's
    own byte counts (one read and one write of the activation for LayerNorm and
    GELU, one read of the logits for the cross-entropy forward, a read and a
    write of the vocabulary-sized gradient for its backward)."""
    import ctypes
    import torch
    from paper_2608_00029_amd import workloads as W
    dev = torch.device("cuda:0")
    L = bd.lib()
    sp = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    R, C = wl.rows, wl.C
    f32 = dict(dtype=torch.float32, device=dev)

    def checked(name, st):
        if st != 0:
            raise RuntimeError(f"{wl.name} {name}: {bd.last_error_string()}")

    # raw C-ABI calls on preallocated buffers, so that the host enqueues faster than the GPU drains
    if wl.op == "layernorm":
        x, g, be, dy = (t.to(dev) for t in W.make_layernorm_inputs(R, C, wl.seed))
        y, dx = torch.empty_like(x), torch.empty_like(x)
        mean, rstd, dg, db = torch.empty(R, **f32), torch.empty(R, **f32), torch.empty(C, **f32), torch.empty(C, **f32)
        ws = torch.empty((bd.layernorm_bwd_workspace_bytes(R, C) // 4,), **f32)
        p_fwd = [t.data_ptr() for t in (x, g, be, y, mean, rstd)]
        p_bwd = [t.data_ptr() for t in (x, g, mean, rstd, dy, dx, dg, db, ws)]
        fwd = lambda: checked("fwd", L.cattn_layernorm_fwd(*p_fwd, R, C, ctypes.c_float(1e-5), sp))
        bwd = lambda: checked("bwd", L.cattn_layernorm_bwd(*p_bwd, R, C, sp))
        n_ws = ws.numel() * 4
        alg = (8 * R * C + 8 * C + 8 * R, 12 * R * C + 8 * R + 12 * C + 2 * n_ws)
        paper = (8 * R * C, 8 * R * C)
    elif wl.op == "gelu":
        n = R * C
        x, dy = (t.to(dev) for t in W.make_gelu_inputs(n, wl.seed))
        y = torch.empty_like(x)
        fwd = lambda: checked("fwd", L.cattn_gelu_fwd(x.data_ptr(), y.data_ptr(), n, sp))
        bwd = lambda: checked("bwd", L.cattn_gelu_bwd(x.data_ptr(), dy.data_ptr(), y.data_ptr(), n, sp))
        alg = (8 * n, 12 * n)
        paper = (8 * n, 8 * n)
    else:
        z, t = (a.to(dev) for a in W.make_sce_inputs(R, C, wl.seed, n_real=W.GPT2_VOCAB))
        lse, rl, loss = torch.empty(R, **f32), torch.empty(R, **f32), torch.empty(1, **f32)
        dz = torch.empty_like(z)
        p_fwd = [a.data_ptr() for a in (z, t, lse, rl, loss)]
        fwd = lambda: checked("fwd", L.cattn_sce_fwd(*p_fwd, R, C, sp))
        bwd = lambda: checked("bwd", L.cattn_sce_bwd(z.data_ptr(), t.data_ptr(), lse.data_ptr(),
                                                     ctypes.c_float(1.0 / R), dz.data_ptr(), R, C, sp))
        alg = (4 * R * C + 16 * R + 4, 8 * R * C + 8 * R)
        paper = (4 * R * C, 8 * R * C)
    fwd()  # the backward reads what the forward writes (mean / rstd, lse)
    out = {"rows": R, "C": C}
    stream = torch.cuda.current_stream(dev)
    torch.cuda.synchronize()
    for name, f, ab, nb in (("fwd", fwd, alg[0], paper[0]), ("bwd", bwd, alg[1], paper[1])):
        for _ in range(warmup):
            f()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            f()
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / steps
        gbs = ab / (ms * 1e-3) / 1e9
        cgbs = copy_gbs(ab)
        out[name] = {"ms": round(ms, 5), "gbs_algorithmic": round(gbs, 1), "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 3),
                     "gbs_paper_bytes": round(nb / (ms * 1e-3) / 1e9, 1), "bytes_algorithmic": ab,
                     "copy_gbs_same_bytes": round(cgbs, 1), "frac_of_copy": round(gbs / cgbs, 3)}
    return out


def copy_gbs(nbytes: int, reps: int = 10) -> float:
    """Read + write bandwidth of torch's device-to-device copy moving the same
    number of bytes (nbytes / 2 read, nbytes / 2 written).  A reference point
    for a kernel that streams its bytes once, not a roof: kernels whose
    streams are read-only, or written with non-temporal stores, exceed it."""
    import torch
    n = max(1, nbytes // 8)
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    return 8 * n / (ms * 1e-3) / 1e9


def measured_trace_us(kernel: str, workload: str):
    """Mean duration (us) of `kernel` on `workload` in the committed rocprofv3
    kernel-trace summary, or None when there is none or the kernel sources
    changed since it was taken."""
    path = os.path.join(PROFILES, f"kernel_trace_{workload}.txt")
    if not os.path.exists(path):
        return None
    digest, us = None, None
    names = {"attn_fwd": "attn_fwd_bf16_kernel", "attn_bwd_dq": "attn_bwd_dq_bf16_kernel",
             "attn_bwd_dkdv": "attn_bwd_dkdv_bf16_kernel"}
    with open(path) as f:
        for line in f:
            if line.startswith("# kernel_sources_sha256:"):
                digest = line.split(":", 1)[1].strip()
            elif not line.startswith("#") and line.strip().startswith(names.get(kernel, "?")):
                us = float(line.split()[-4])  # columns after the name: calls, avg_us, min_us, max_us, pct
    return us if digest == kernel_source_digest() else None


def time_repeats(kernels, stream, repeats: int, steps: int, flops: float):
    """The step timed `repeats` more times, `steps` steps each, between device
    synchronisations (no events): median and spread of ms per step."""
    import statistics
    import torch
    ms = []
    for _ in range(repeats):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            for _, f in kernels:
                f()
        torch.cuda.synchronize()
        ms.append((time.perf_counter() - t0) * 1e3 / steps)
    med = statistics.median(ms)
    return {"repeats": repeats, "steps_each": steps, "ms_per_step": [round(x, 5) for x in ms],
            "median_ms_per_step": round(med, 5), "median_tflops": round(flops / (med * 1e-3) / 1e12, 2)}


def time_cold(kernels, stream, steps: int, flops: float, peak: float):
    """The step with the 256 MB last-level cache (MALL) evicted before every
    step: 512 MB are written between steps.  Each step is bracketed by HIP
    events on the kernels' stream, so the eviction writes are not timed."""
    import torch
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda:0")
    times = []
    for i in range(steps + 1):
        flush.fill_(i & 0xFF)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _, f in kernels:
            f()
        e1.record(stream)
        torch.cuda.synchronize()
        if i > 0:
            times.append(e0.elapsed_time(e1))
    times.sort()
    med = times[len(times) // 2]
    del flush
    return {"steps": steps, "evicted_bytes_between_steps": 512 << 20, "median_ms_per_step": round(med, 5),
            "median_tflops": round(flops / (med * 1e-3) / 1e12, 2),
            "pct_mfma_peak": round(100.0 * flops / (med * 1e-3) / 1e12 / peak, 2),
            "note": "each step bracketed by HIP events (dispatch latency of the first kernel included)"}


def copy_probe(mib: int) -> int:
    """A plain copy of known size: it reads and writes exactly mib MiB per launch."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_per_launch": n * 4, "launches": 5}), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--warmup", type=int, default=300)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--event-every", type=int, default=8,
                    help="bracket each kernel with HIP events on every Nth timed step (1: every step)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="budget of the CPU-oracle baseline (0 disables it)")
    ap.add_argument("--configs", type=int, default=1,
                    help="also time every workload (forward, backward, step) after the timed region (0 disables)")
    ap.add_argument("--repeats", type=int, default=5,
                    help="after the timed region, time the step this many more times (median reported; 0 disables)")
    ap.add_argument("--repeat-steps", type=int, default=100, help="steps per repeat")
    ap.add_argument("--cold", type=int, default=1,
                    help="also time the step with the 256 MB MALL evicted (512 MB written) before each step")
    ap.add_argument("--cold-steps", type=int, default=20, help="steps of the cold variant")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="instead of the benchmark, run 5 plain device-to-device copies of this many MiB "
                         "(reference kernel for calibrating rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    ap.add_argument("--only", choices=("memops", "lmhead"), default=None,
                    help="instead of the benchmark, time only the memory-bound operators (forward and "
                         "backward) or only the fused loss head, --steps calls each after --warmup, and "
                         "print their JSON (for counter collection)")
    args = ap.parse_args()
    if args.copy_probe_mib > 0:
        return copy_probe(args.copy_probe_mib)

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this build measures the attention kernels on ONE GPU only; "
              "multi-GPU runs (--gpus N > 1) are not part of it.", file=sys.stderr)
        return 2

    import torch
    from paper_2608_00029_amd import binding as bd
    from paper_2608_00029_amd.workloads import BY_NAME, workload_inputs

    if not torch.cuda.is_available():
        print("bench.py: no HIP device visible", file=sys.stderr)
        return 1
    if args.only == "memops":
        from paper_2608_00029_amd.workloads import MEMOPS_WORKLOADS
        print(json.dumps({c.name: time_memops(c, bd, steps=args.steps, warmup=args.warmup)
                          for c in MEMOPS_WORKLOADS}), flush=True)
        return 0
    if args.only == "lmhead":
        from paper_2608_00029_amd.workloads import LMHEAD_WORKLOADS
        print(json.dumps({c.name: time_lmhead(c, bd, steps=args.steps, warmup=args.warmup)
                          for c in LMHEAD_WORKLOADS}), flush=True)
        return 0
    w = BY_NAME[args.workload]
    dev = torch.device("cuda:0")
    cpu_inputs = workload_inputs(w)
    q, k, v, do = (t.to(dev) for t in cpu_inputs)
    o = torch.empty_like(q)
    lse = torch.empty((w.B, w.H, w.S), dtype=torch.float32, device=dev)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
    ws = torch.empty((bd.workspace_bytes(w.B, w.H, w.S, w.D) // 4,), dtype=torch.float32, device=dev)
    dcode = bd.CATTN_BF16 if w.dtype == "bf16" else bd.CATTN_F32
    L = bd.lib()
    stream = torch.cuda.current_stream(dev)
    sp = __import__("ctypes").c_void_p(stream.cuda_stream)
    P = lambda t: t.data_ptr()  # noqa: E731
    shape = (w.B, w.H, w.S, w.D, float(w.scale), int(w.causal), dcode, sp)

    def fwd():
        return L.cattn_attn_fwd(P(q), P(k), P(v), P(o), P(lse), *shape)

    def bwd_dq():
        return L.cattn_attn_bwd_dq(P(q), P(k), P(v), P(o), P(do), P(lse), P(dq), P(ws), *shape)

    def bwd_dkdv():
        return L.cattn_attn_bwd_dkdv(P(q), P(k), P(v), P(do), P(lse), P(ws), P(dk), P(dv), *shape)

    kernels = [("attn_fwd", fwd), ("attn_bwd_dq", bwd_dq), ("attn_bwd_dkdv", bwd_dkdv)]
    for _ in range(args.warmup):
        for name, f in kernels:
            st = f()
            if st != 0:
                raise RuntimeError(f"{name}: {bd.status_string(st)}: {bd.last_error_string()}")
    torch.cuda.synchronize()

    # Every --event-every-th timed step brackets each kernel with HIP events on the
    # kernels' stream; the other steps run bare.  An event between two kernels
    # costs the GPU a few microseconds, so recording them on every step would
    # inflate the step time the throughput is computed from by about a tenth.
    # at least 8 sampled steps whenever the run has that many
    every = max(1, min(args.event_every, args.steps // 8))
    sampled = [i for i in range(args.steps) if i % every == 0]
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(kernels) + 1)] for _ in sampled]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        if i % every == 0:
            e = ev[i // every]
            e[0].record(stream)
            for j, (_, f) in enumerate(kernels):
                f()
                e[j + 1].record(stream)
        else:
            for _, f in kernels:
                f()
    torch.cuda.synchronize()
    t1 = time.perf_counter()

    per_kernel_ms = {name: sum(e[j].elapsed_time(e[j + 1]) for e in ev) / len(ev)
                     for j, (name, _) in enumerate(kernels)}
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    fwd_f, bwd_f = w.counted_flops()
    tflops = (fwd_f + bwd_f) / (ms_per_step * 1e-3) / 1e12
    peak = PEAK_TFLOPS[w.dtype]

    kf = kernel_flops(w)
    dom = max(per_kernel_ms, key=per_kernel_ms.get)
    achieved = kf[dom] / (per_kernel_ms[dom] * 1e-3) / 1e12
    trace_us = measured_trace_us(dom, w.name)
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": measured_traffic(dom, w.name), "kernel": dom,
                "flops_per_launch": kf[dom], "mean_launch_us": round(per_kernel_ms[dom] * 1e3, 2),
                "timed_launches": len(ev),
                # the same kernel's mean duration in the committed rocprofv3 kernel trace (no event marker
                # before the launch, so no dispatch latency in it), while the kernel sources are unchanged
                "trace_mean_launch_us": trace_us,
                "frac_from_trace": round(kf[dom] / (trace_us * 1e-6) / 1e12 / peak, 4) if trace_us else None}

    line = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic: seeded N(0,1) Q, K, V, dO rounded to bf16, inputs resident in HBM",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "S": w.S, "D": w.D, "causal": w.causal,
                   "scale": w.scale, "parallelism": "single-gpu"},
        "pct_mfma_peak": round(100.0 * tflops / peak, 2),
        "kernels_us": {n: round(t * 1e3, 2) for n, t in per_kernel_ms.items()},
        "roofline": roofline,
    }
    if args.repeats > 0:
        line["repeats"] = time_repeats(kernels, stream, args.repeats, args.repeat_steps, fwd_f + bwd_f)
    if args.cold:
        line["cold"] = time_cold(kernels, stream, args.cold_steps, fwd_f + bwd_f, peak)
    if args.configs:
        from paper_2608_00029_amd.workloads import SWEEP, WORKLOADS
        line["configs"] = {c.name: time_workload(c, bd, steps=20, warmup=5) for c in WORKLOADS}
        line["configs"][w.name + "_bshd"] = time_workload(w, bd, steps=20, warmup=5, layout="bshd")
        line["sweep"] = {c.name: time_workload(c, bd, steps=20, warmup=5) for c in SWEEP}
        from paper_2608_00029_amd.workloads import LMHEAD_WORKLOADS
        line["lmhead"] = {c.name: time_lmhead(c, bd, steps=20, warmup=3) for c in LMHEAD_WORKLOADS}
        from paper_2608_00029_amd.workloads import MEMOPS_WORKLOADS
        line["memops"] = {c.name: time_memops(c, bd, steps=20, warmup=3) for c in MEMOPS_WORKLOADS}
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(w, cpu_inputs, args.cpu_seconds)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
