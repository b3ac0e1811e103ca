#!/usr/bin/env python3
"""Benchmark of the DLA layer forward on one MI355X.

One step = one prefill of the 16k-token workload from an empty cache (B=4,
H=16, T=16384, d_k=d_v=128, C=128, tau=0.5, bf16 inputs, float32 states,
long stable spans alternating with short i.i.d. bursts): token frames, the
boundary scan with the capacity schedule, the state update and the readout --
every step of the hot path.  `value` is prefill tokens/s (B*T tokens per step)
with all inputs resident in HBM.

Also reported on the same line:
  * roofline of the dominant kernel (the readout), from HIP events that the
    library records around each of its launches in the timed steps, and of
    the whole call (the method's FLOPs over the step time); fractions against
    the data-sheet peaks and against the peaks measured on this device by the
    library's measurement kernels (dla_peak.h);
  * the other prefill workloads (4k tokens at C = 64, 64k tokens at C = 256);
  * the decode step at C = 128 on full caches built from a 32k-token prefix
    (B=64, H=32), with float32 and with bfloat16 storage of the closed
    states, and on few heads (B=1, H=32: several workgroups per head);
  * cache and workspace bytes;
  * a sweep of a Mamba-2-shaped layer under DLA and under fixed merging
    policies (single state, every-K blocking, log-linear buckets) on the same
    kernels: prefill tokens/s and memory over batch size and context length;
  * cpu_baseline: the float64 oracle on bounded samples (a prefill of one
    sequence, and decode steps on a few heads of the GPU-built cache).

    python bench.py [--steps K] [--warmup W] [--gpus 1]
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

METRIC = "DLA layer fwd tokens/sec (prefill) + decode-step µs; % of HBM/MFMA roofline"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA (data sheet)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E (data sheet)
PROFILES = os.path.join(ROOT, "profiles")
# sources whose kernels the counter summaries describe
KERNEL_SOURCES = {
    "prefill_readout_kernel": ["prefill_readout.hip", "prefill_chunk.h", "prefill.h", "mfma.h",
                               "dla_common.h"],
    "decode_kernel": ["decode.hip", "decode.h", "dla_common.h"],
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_digest(kernel: str) -> str:
    """sha256 over the sources of a kernel with comments and whitespace removed,
    to tell whether a counter summary still describes the code being timed (a
    change to a comment leaves it valid)."""
    import hashlib
    import re
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2606_10650_amd", "csrc", f)) as fh:
            src = fh.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()


def counter_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    rocprofv3 counter summary (FETCH_SIZE + WRITE_SIZE, scaled by the copy-kernel
    calibration), or None when there is none for the current sources."""
    path = os.path.join(PROFILES, f"{kernel}_{workload}_counters.md")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if line.startswith("- ") and ": " in line:
            k, v = line[2:].split(": ", 1)
            kv[k.strip()] = v.strip().strip("`")
    if kv.get("source_sha256") != source_digest(kernel):
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_probe(args, torch):
    """A plain device copy of known size, to calibrate the FETCH_SIZE and
    WRITE_SIZE counters against bytes moved."""
    n = args.copy_probe_mib << 20
    src = torch.empty(n, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": n, "launches": 5}), flush=True)


def measured_peaks(torch, dla):
    """Dense bfloat16 MFMA rate and HBM read bandwidth of this device, from the
    library's measurement kernels: the best of three runs each."""
    blocks, iters = 2048, 4096
    sink = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    dla.peak_mfma_bf16(blocks, 64, sink)   # warm-up
    best = 1e30
    for _ in range(3):
        ev[0].record()
        dla.peak_mfma_bf16(blocks, iters, sink)
        ev[1].record()
        torch.cuda.synchronize()
        best = min(best, ev[0].elapsed_time(ev[1]))
    tflops = blocks * 16.0 * iters * 32768 / (best * 1e-3) / 1e12
    buf = torch.empty(4 << 30, dtype=torch.uint8, device="cuda")
    buf.fill_(1)
    rb = 8192
    rsink = torch.empty(rb * 256, dtype=torch.float32, device="cuda")
    dla.peak_hbm_read(buf, rb, rsink)
    best = 1e30
    for _ in range(3):
        ev[0].record()
        dla.peak_hbm_read(buf, rb, rsink)
        ev[1].record()
        torch.cuda.synchronize()
        best = min(best, ev[0].elapsed_time(ev[1]))
    gbs = buf.numel() / (best * 1e-3) / 1e9
    del buf
    torch.cuda.empty_cache()
    return {"mfma_bf16_tflops": round(tflops, 1), "hbm_read_gbs": round(gbs, 1),
            "how": ("dla_peak_mfma_bf16: 2048 workgroups x 4 waves x 4 independent chains of "
                    "v_mfma_f32_32x32x16_bf16; dla_peak_hbm_read: one read of 4 GiB with 16-byte "
                    "non-temporal loads; best of 3")}


def frac(achieved, peak):
    return round(achieved / peak, 4)


def prefill_bench(args, torch, dla, W, steps, warmup, with_events=True, serial_steps=3,
                  pool_budget_log2=0):
    from paper_2606_10650_amd.workloads import make_inputs
    t0 = time.time()
    x = make_inputs(W)
    log(f"[bench] generated {W.label} in {time.time() - t0:.1f}s")

    def dev(a, shape):
        if W.dtype == "bf16":
            t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
        else:
            t = torch.from_numpy(a)
        return t.reshape(shape).cuda()

    B, H, T = W.B, W.H, W.T
    q = dev(x["q"], (B, H, T, W.dk))
    k = dev(x["k"], (B, H, T, W.dk))
    v = dev(x["v"], (B, H, T, W.dv))
    lam = dev(x["lam"], (B, H, T, W.C))
    g = torch.from_numpy(x["g"]).reshape(B, H, T).cuda()
    del x
    cache = dla.cache_alloc(B, H, W.C, W.dk, W.dv)
    ws_pipe = dla.workspace_bytes(cache, T, k.dtype, pool_budget_log2=pool_budget_log2)
    ws_serial = dla.workspace_bytes(cache, T, k.dtype, serial=True,
                                    pool_budget_log2=pool_budget_log2)
    ws = torch.empty(max(ws_pipe, ws_serial), dtype=torch.uint8, device="cuda")
    out = torch.empty((B, H, T, W.dv), dtype=k.dtype, device="cuda")
    bnd = torch.empty((B, H, T), dtype=torch.int8, device="cuda")
    mrg = torch.empty((B, H, T), dtype=torch.int32, device="cuda")
    scr = torch.empty((B, H, T), dtype=torch.float32, device="cuda")
    desc = cache.desc
    nbytes = cache.buf.numel()

    def step(events=None, rev=None, serial=False):
        import ctypes
        n = ctypes.c_size_t(nbytes)
        dla._check(dla.lib().dla_state_cache_alloc(ctypes.byref(desc), dla._ptr(cache.buf),
                                                   ctypes.byref(n), dla._stream(cache.device)),
                   "cache init")
        dla.prefill(cache, q, k, v, g, lam, tau=W.tau, out=out, boundary=bnd, merge_idx=mrg,
                    score=scr, workspace=ws, stage_events=events, readout_events=rev,
                    serial=serial, pool_budget_log2=pool_budget_log2)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    # the timed steps: the pipelined prefill, with every readout launch
    # bracketed by a pair of events on the stream it runs on
    nseg = dla.prefill_segments(cache, T, k.dtype, pool_budget_log2=pool_budget_log2)
    revs = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * nseg)]
            for _ in range(steps)] if with_events else [None] * steps
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    for e in [start, stop] + [e for r in revs if r for e in r]:
        e.record()   # created here, outside the timed region
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record()
    for i in range(steps):
        step(rev=revs[i])
    stop.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / steps
    log(f"[bench] {W.name} prefill wall clock {ms:.3f} ms/step, "
        f"events {start.elapsed_time(stop) / steps:.3f} ms/step")
    res = {"ms_per_step": ms, "value": B * T / (ms * 1e-3), "workspace_bytes": ws_pipe,
           "cache_bytes": nbytes, "segments": nseg}
    # algorithmic work from this run's exports: per token and head 2 m_t d_k d_v
    # (the readout over the m_t live states) + 4 d_k d_v (accumulate and score)
    b = bnd.cpu().numpy().reshape(B * H, T).astype(np.int64)
    mm = (mrg.cpu().numpy().reshape(B * H, T) >= 0).astype(np.int64)
    m_t = np.cumsum(b, axis=1) - np.cumsum(mm, axis=1)
    d2 = float(W.dk * W.dv)
    flops_ro = 2.0 * d2 * m_t.sum()
    flops_call = flops_ro + 4.0 * d2 * m_t.size
    flops_call_cap = (2.0 * W.C + 4.0) * d2 * m_t.size
    res["decisions"] = {"boundaries": int(b.sum()), "merges": int(mm.sum()),
                        "mean_live_states": round(float(m_t.mean()), 2)}
    call = flops_call / (ms * 1e-3) / 1e12
    res["roofline_call"] = {
        "bound": "mfma", "achieved": round(call, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
        "frac": frac(call, PEAK_BF16_TFLOPS),
        "frac_at_m_eq_C": frac(flops_call_cap / (ms * 1e-3) / 1e12, PEAK_BF16_TFLOPS),
        "flops_per_step": flops_call, "flops_per_step_at_m_eq_C": flops_call_cap}
    if with_events:
        ro_launch = np.array([[r[2 * j].elapsed_time(r[2 * j + 1]) for j in range(nseg)]
                              for r in revs])
        ro_ms = float(ro_launch.sum(axis=1).mean())   # readout time per step, all launches
        achieved = flops_ro / (ro_ms * 1e-3) / 1e12
        res["roofline"] = {"kernel": "prefill_readout_kernel", "bound": "mfma",
                           "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                           "unit": "TFLOP/s", "frac": frac(achieved, PEAK_BF16_TFLOPS),
                           "traffic": counter_traffic("prefill_readout_kernel", W.name),
                           "launches_per_step": nseg,
                           "launch_ms_mean": round(float(ro_launch.mean()), 4),
                           "readout_ms_per_step": round(ro_ms, 4),
                           "flops_per_launch": flops_ro / nseg,
                           "flops_per_launch_at_m_eq_C": 2.0 * d2 * W.C * m_t.size / nseg}
    if serial_steps:
        # stage breakdown: the same step with the stages one after another
        ns = len(dla.PREFILL_STAGES)
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(ns + 1)]
               for _ in range(serial_steps)]
        for e in evs:
            step(events=e, serial=True)
        torch.cuda.synchronize()
        stages = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(ns)] for e in evs])
        res["stages_ms_serial"] = dict(zip(dla.PREFILL_STAGES,
                                           [round(float(s), 4) for s in stages.mean(axis=0)]))
        if "roofline" in res:
            # the same launches alone on the chip: in the timed (pipelined) steps
            # the scan and the next segment's update share the CUs with them
            ser = res["stages_ms_serial"]["readout"]
            res["roofline"]["readout_ms_per_step_serial"] = ser
            res["roofline"]["frac_serial"] = frac(flops_ro / (ser * 1e-3) / 1e12, PEAK_BF16_TFLOPS)
    del q, k, v, lam, g, out, ws, cache
    torch.cuda.empty_cache()
    return res


def delta_prefill_bench(args, torch, dla, W, steps):
    """The Gated DeltaNet form of the prefill (dla_prefill_delta) on workload W,
    step sizes beta ~ U(0.05, 1): ms per call and tokens/s, with the
    sequential scan's share measured in a skip-readout call."""
    from paper_2606_10650_amd.workloads import make_prefix_torch
    t0 = time.time()
    q, k, v, g, lam = make_prefix_torch(W, "cuda", with_lambda=True)
    gen = torch.Generator(device="cuda").manual_seed(W.seed + 29)
    beta = 0.05 + 0.95 * torch.rand((W.B, W.H, W.T), device="cuda", generator=gen)
    torch.cuda.synchronize()
    log(f"[bench] delta prefill: {W.label} drawn in {time.time() - t0:.1f}s")
    cache = dla.cache_alloc(W.B, W.H, W.C, W.dk, W.dv)
    ws = torch.empty(dla.delta_workspace_bytes(cache, W.T, k.dtype), dtype=torch.uint8,
                     device="cuda")
    out = torch.empty((W.B, W.H, W.T, W.dv), dtype=k.dtype, device="cuda")

    def run(skip=False):
        dla.cache_reset(cache)
        dla.prefill_delta(cache, None if skip else q, k, v, g, beta, None if skip else lam,
                          tau=W.tau, out=None if skip else out, skip_readout=skip, workspace=ws,
                          want_exports=False)

    run()
    torch.cuda.synchronize()
    e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    e[0].record()
    for _ in range(steps):
        run()
    e[1].record()
    e[2].record()
    run(skip=True)
    e[3].record()
    torch.cuda.synchronize()
    ms = e[0].elapsed_time(e[1]) / steps
    res = {"workload": f"prefill, Gated DeltaNet form, {W.label}, beta ~ U(0.05, 1)",
           "ms_per_call": round(ms, 3), "tokens_per_s": round(W.B * W.T / (ms * 1e-3), 1),
           "ms_without_readout": round(e[2].elapsed_time(e[3]), 3),
           "workspace_bytes": ws.numel(), "calls": steps}
    del q, k, v, g, lam, beta, ws, out, cache
    torch.cuda.empty_cache()
    return res


def decode_bytes(W, m_live, state_dtype_bf16):
    """HBM bytes of one decode step per head on a full cache with a boundary
    and a merge: every live state read once; the merged pair written, with
    bfloat16 storage also the state that closes, and the new newest state;
    the token vectors, lambda row and output."""
    D = W.dk * W.dv
    if state_dtype_bf16:
        rd = (m_live - 1) * D * 2 + D * 4
        wr = 2 * D * 2 + D * 4
    else:
        rd = m_live * D * 4
        wr = 2 * D * 4
    return rd + wr + (2 * W.dk + W.dv + W.C + W.dv) * 2


def decode_bench(args, torch, dla, W, steps, state_dtype, label, delta=False):
    from paper_2606_10650_amd.workloads import make_decode_tokens_torch, make_prefix_torch
    t0 = time.time()
    _, k, v, g = make_prefix_torch(W, "cuda")
    torch.cuda.synchronize()
    cache = dla.cache_alloc(W.B, W.H, W.C, W.dk, W.dv, state_dtype=state_dtype)
    dla.prefill(cache, None, k, v, g, None, tau=W.tau, skip_readout=True, want_exports=False)
    torch.cuda.synchronize()
    log(f"[bench] {label}: prefix drawn and absorbed in {time.time() - t0:.1f}s")
    del k, v, g
    torch.cuda.empty_cache()
    q, kk, vv, gg, lam = make_decode_tokens_torch(W, steps + 2, "cuda")
    beta = None
    if delta:
        # step sizes of the delta rule, U(0.05, 1) per head and token
        gen = torch.Generator(device="cuda").manual_seed(W.seed + 17)
        beta = 0.05 + 0.95 * torch.rand((steps + 2, W.B, W.H), device="cuda", generator=gen)

    def one(c, i, **kw):
        if delta:
            return dla.decode_step_delta(c, q[i], kk[i], vv[i], gg[i], beta[i], lam[i],
                                         tau=W.tau, out=out, **kw)
        return dla.decode_step(c, q[i], kk[i], vv[i], gg[i], lam[i], tau=W.tau, out=out, **kw)

    out = torch.empty((W.B, W.H, W.dv), dtype=torch.bfloat16, device="cuda")
    bnd = torch.empty((steps, W.B, W.H), dtype=torch.int8, device="cuda")
    mrg = torch.empty((steps, W.B, W.H), dtype=torch.int32, device="cuda")
    m_before = int(dla.cache_export(cache, heads=[0])["m"][0])
    # warm-up on a copy of the cache, then the timed steps on the prefix cache
    warm = dla.StateCache(W.B, W.H, W.C, W.dk, W.dv, cache.buf.clone(), state_dtype)
    for i in range(2):
        one(warm, i, want_exports=False)
    torch.cuda.synchronize()
    del warm
    torch.cuda.empty_cache()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    for e in evs:
        e.record()   # created here, outside the timed region
    torch.cuda.synchronize()
    # The stream is held by a short device-side sleep while the steps are
    # enqueued, so that the events time the kernels and not the host's
    # enqueueing (a step on few heads takes less time on the device than the
    # Python call that enqueues it); the wall clock is reported beside.
    torch.cuda._sleep(int(2e6) * (1 + steps // 8))
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(steps):
        one(cache, i + 2, boundary=bnd[i], merge_idx=mrg[i], score=None)
        evs[i + 1].record()
    t_enq = time.perf_counter() - t0
    torch.cuda.synchronize()
    us = np.array([evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(steps)])
    nb = int(bnd.sum().item())
    nm = int((mrg >= 0).sum().item())
    nh = W.B * W.H
    sb = state_dtype == dla.DLA_BF16
    bytes_step = decode_bytes(W, W.C, sb) * nh
    ach = bytes_step / (np.mean(us) * 1e-6) / 1e9
    res = {
        "config": {"workload": (f"decode {W.B}x{W.H} heads, C={W.C}, d={W.dk}, prefix {W.T} "
                                f"tokens, {'bf16' if sb else 'f32'} state storage"
                                + (", delta rule on the newest state" if delta else "")),
                   "B": W.B, "H": W.H, "C": W.C, "prefix_tokens": W.T, "steps": steps,
                   "state_dtype": "bf16" if sb else "f32"},
        "us_per_step_mean": round(float(np.mean(us)), 2),
        "us_per_step_p50": round(float(np.median(us)), 2),
        "us_per_step_host_enqueue": round(t_enq / steps * 1e6, 2),
        "live_states_before": m_before,
        "boundaries": nb, "merges": nm,
        "cache_bytes": cache.buf.numel(),
        "roofline": {"kernel": "decode_kernel", "bound": "hbm", "achieved": round(ach, 1),
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": frac(ach, PEAK_HBM_GBS),
                     "traffic": (None if delta else
                                 counter_traffic("decode_kernel", W.name) if not sb else
                                 counter_traffic("decode_kernel", W.name + "_bf16")),
                     "bytes_per_launch": bytes_step},
    }
    if args.decode_cpu_heads and W.B * W.H > 1000 and not sb:
        res["_cache"] = cache   # for the CPU baseline of the decode step
    else:
        del cache
    torch.cuda.empty_cache()
    return res


def policy_sweep(args, torch, dla):
    """Prefill throughput and memory of one Mamba-2-shaped layer (48 heads, state
    size d_k = 128, head dimension d_v = 64, bf16 inputs, float32 states) under
    DLA (C = 30, tau = 0.6) and under fixed policies on the same kernels, driven
    through the override path: a single state (the base model), every-64-token
    blocking with C = 30, and log-linear buckets (C = ceil(log2 T) + 1).  The
    two sweeps of the paper's efficiency study (Sec. 4.3): batch size at 128
    tokens, and context length at batch 1.  Inputs: segments of geometric length
    (mean 64 tokens).  Memory is what the layer holds besides its inputs and
    outputs: the state cache and the prefill workspace."""
    from paper_2606_10650_amd import policies as P
    from paper_2606_10650_amd.workloads import Workload, make_prefix_torch
    base = Workload("mamba2_layer", 1, 48, 128, 128, 64, 30, 0.6, "bf16", -0.05, 7, "geom",
                    mean_len=64)
    points = [("batch", B, 128) for B in (1, 16, 64, 256)] + \
             [("context", 1, T) for T in (1024, 4096, 16384, 65536)]
    rows = []
    # bring the device out of its idle clocks before the first (smallest) point
    a = torch.randn(4096, 4096, device="cuda", dtype=torch.bfloat16)
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 0.3:
        for _ in range(20):
            a = (a @ a).clamp_(-1, 1)
        torch.cuda.synchronize()
    del a
    for sweep, B, T in points:
        W = base.replace(B=B, T=T)
        q, k, v, g, lam = make_prefix_torch(W, "cuda", with_lambda=True)
        for pol in ("single_state", "every_k", "log_linear", "dla"):
            C, b, m = P.schedule(pol, T, C_dla=W.C, K=64)
            shp = (B, W.H, T)
            bo = None if b is None else torch.from_numpy(b).cuda().expand(shp).contiguous()
            mo = None if m is None else torch.from_numpy(m).cuda().expand(shp).contiguous()
            lamC = lam[..., :C].contiguous()
            cache = dla.cache_alloc(B, W.H, C, W.dk, W.dv)
            wsb = dla.workspace_bytes(cache, T, k.dtype)
            ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
            out = torch.empty((B, W.H, T, W.dv), dtype=k.dtype, device="cuda")
            bnd = torch.empty(shp, dtype=torch.int8, device="cuda")
            mrg = torch.empty(shp, dtype=torch.int32, device="cuda")

            def step(e0=None, e1=None):
                dla.cache_reset(cache)
                if e0 is not None:
                    e0.record()
                dla.prefill(cache, q, k, v, g, lamC, tau=W.tau, out=out, boundary=bnd,
                            merge_idx=mrg, boundary_override=bo, merge_override=mo, workspace=ws)
                if e1 is not None:
                    e1.record()

            for _ in range(3):
                step()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            step()
            torch.cuda.synchronize()
            n = int(min(200, max(args.sweep_steps, 0.05 / max(time.perf_counter() - t0, 1e-6))))
            evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                   for _ in range(n)]
            for e in evs:
                step(*e)
            torch.cuda.synchronize()
            ms = float(np.mean([a.elapsed_time(z) for a, z in evs]))
            bb = bnd.cpu().numpy().reshape(-1, T).astype(np.int64)
            mm = (mrg.cpu().numpy().reshape(-1, T) >= 0).astype(np.int64)
            live = np.cumsum(bb, axis=1) - np.cumsum(mm, axis=1)
            io = sum(t.numel() * t.element_size() for t in (q, k, v, g, lamC, out))
            rows.append({"sweep": sweep, "B": B, "T": T, "policy": pol, "C": C,
                         "ms": round(ms, 4), "tokens_per_s": round(B * T / (ms * 1e-3), 1),
                         "cache_MB": round(cache.buf.numel() / 2**20, 3),
                         "workspace_MB": round(wsb / 2**20, 3),
                         "io_MB": round(io / 2**20, 3),
                         "boundaries": int(bb.sum()), "merges": int(mm.sum()),
                         "mean_live_states": round(float(live.mean()), 2), "steps_timed": n})
            log(f"[sweep] {sweep} B={B} T={T} {pol} C={C}: {ms:.4f} ms, "
                f"{rows[-1]['tokens_per_s']:.0f} tok/s, cache {rows[-1]['cache_MB']} MB, "
                f"workspace {rows[-1]['workspace_MB']} MB, live {rows[-1]['mean_live_states']}")
            del cache, ws, out, bnd, mrg, bo, mo, lamC
        del q, k, v, g, lam
        torch.cuda.empty_cache()
    return {"layer": ("Mamba-2-780M-shaped layer: H=48, d_k=128, d_v=64, bf16 inputs, f32 "
                      "states, geometric segments (mean 64); DLA C=30 tau=0.6; every_k K=64 "
                      "C=30; log_linear C=ceil(log2 T)+1; single_state C=1"),
            "timing": "HIP events around each prefill call (cache reset outside), mean",
            "rows": rows}


def cpu_baseline(args, W):
    from oracle import oracle_forward, oracle_threads
    from paper_2606_10650_amd.workloads import make_inputs, to_f64
    heads = [(0, h) for h in range(W.H)]
    Ts = args.cpu_tokens
    w = W.replace(T=Ts)
    x = make_inputs(w, heads=heads)
    f = lambda a: to_f64(a, w.dtype)
    t0 = time.perf_counter()
    oracle_forward(f(x["k"]), f(x["v"]), x["g"].astype(np.float64), w.C, w.tau, q=f(x["q"]),
                   lam=f(x["lam"]))
    dt = time.perf_counter() - t0
    return {"value": round(Ts / dt, 2), "unit": "tokens/s", "cores": oracle_threads(),
            "kind": "oracle",
            "sample": (f"float64 oracle, sequence 0 of the prefill workload ({W.H} heads, first "
                       f"{Ts} of {W.T} tokens, {dt:.1f} s); tokens/s counts sequence tokens "
                       f"(all heads of a token together), comparable with value / B")}


def cpu_decode_baseline(args, torch, dla, W, cache):
    """The float64 oracle's decode step from the GPU-built cache of a few heads
    (copied to the host), timed on the host cores: microseconds per step for
    all B*H heads, scaled from the sample (heads are independent)."""
    from oracle import OracleCache, oracle_forward, oracle_threads
    from paper_2606_10650_amd.workloads import make_decode_tokens_torch
    nh = W.B * W.H
    heads = list(range(args.decode_cpu_heads))
    steps = args.decode_cpu_steps
    exp = dla.cache_export(cache, heads=heads)
    # the oracle's cache: true states exp(G - F_j) times the stored values
    oc = OracleCache.empty(len(heads), W.C, W.dk, W.dv)
    for i in range(len(heads)):
        m = int(exp["m"][i])
        oc.m[i], oc.n[i], oc.ibar[i] = m, exp["n"][i], exp["ibar"][i]
        oc.S[i, :m] = np.exp(exp["G"][i] - exp["F"][i, :m])[:, None, None] * exp["stored"][i, :m]
    q, k, v, g, lam = make_decode_tokens_torch(W, steps, "cpu")

    def host(t):
        t = t.reshape(steps, nh, -1)[:, heads].float().numpy().astype(np.float64)
        return np.ascontiguousarray(np.transpose(t, (1, 0, 2)))
    xq, xk, xv, xl, xg = host(q), host(k), host(v), host(lam), host(g)[..., 0]
    t0 = time.perf_counter()
    oracle_forward(xk, xv, xg, W.C, W.tau, q=xq, lam=xl, cache=oc)
    dt = time.perf_counter() - t0
    us_all = dt / steps * 1e6 * nh / len(heads)
    return {"us_per_step": round(us_all, 1), "unit": "us/step (all heads)",
            "cores": oracle_threads(), "kind": "oracle",
            "sample": (f"float64 oracle, {steps} decode steps of {len(heads)} of the {nh} heads "
                       f"from the GPU-built cache ({dt:.1f} s), scaled to all heads")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="cfg3")
    ap.add_argument("--decode-steps", type=int, default=256)
    ap.add_argument("--other-steps", type=int, default=5)
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-others", action="store_true")
    ap.add_argument("--no-peaks", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--sweep-steps", type=int, default=3)
    ap.add_argument("--cpu-tokens", type=int, default=16384)
    ap.add_argument("--decode-cpu-heads", type=int, default=128)
    ap.add_argument("--decode-cpu-steps", type=int, default=64)
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures a single GPU (--gpus 1): the DLA layer shards over (batch, head) "
              "with no exchange between GPUs, so N GPUs run N independent shares of the heads.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    if args.copy_probe_mib:
        copy_probe(args, torch)
        return
    from paper_2606_10650_amd import dla
    from paper_2606_10650_amd.workloads import WORKLOADS
    W = WORKLOADS[args.workload]
    pre = prefill_bench(args, torch, dla, W, args.steps, args.warmup)
    log(f"[bench] prefill {pre['ms_per_step']:.3f} ms/step, serial stages {pre['stages_ms_serial']}")
    res = {
        "metric": METRIC,
        "value": round(pre["value"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(pre["ms_per_step"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": (f"prefill {W.name}: B={W.B} H={W.H} T={W.T} d_k={W.dk} "
                                f"d_v={W.dv} C={W.C} tau={W.tau} bf16 inputs, f32 states, "
                                f"{W.structure}"),
                   "B": W.B, "H": W.H, "T": W.T, "C": W.C, "d_k": W.dk, "d_v": W.dv,
                   "tau": W.tau},
        "stages_ms_serial": pre["stages_ms_serial"],
        "decisions": pre["decisions"],
        "roofline": pre["roofline"],
        "roofline_call": pre["roofline_call"],
        "memory": {"cache_bytes": pre["cache_bytes"], "workspace_bytes": pre["workspace_bytes"]},
    }
    if not args.no_peaks:
        pk = measured_peaks(torch, dla)
        res["peaks_measured"] = pk
        for key in ("roofline", "roofline_call"):
            res[key]["frac_measured_peak"] = frac(res[key]["achieved"], pk["mfma_bf16_tflops"])
        log(f"[bench] measured peaks {pk}")
    if not args.no_others:
        others = {}
        for name in ("cfg2", "cfg4"):
            Wo = WORKLOADS[name]
            r = prefill_bench(args, torch, dla, Wo, args.other_steps, 1, serial_steps=0)
            others[name] = {
                "workload": (f"prefill {name}: B={Wo.B} H={Wo.H} T={Wo.T} d={Wo.dk} C={Wo.C} "
                             f"bf16, {Wo.structure}"),
                "ms_per_step": round(r["ms_per_step"], 4), "tokens_per_s": round(r["value"], 1),
                "roofline_readout_frac": r["roofline"]["frac"],
                "roofline_call_frac": r["roofline_call"]["frac"],
                "roofline_call_frac_at_m_eq_C": r["roofline_call"]["frac_at_m_eq_C"],
                "workspace_bytes": r["workspace_bytes"], "decisions": r["decisions"]}
        res["prefill_workloads"] = others
    if not args.no_others:
        # the prefill's state copies under smaller budgets (flags bits 8..15):
        # less workspace, more segments, identical results
        pb = {}
        for kb in (31, 30):
            r = prefill_bench(args, torch, dla, W, args.other_steps, 1, with_events=False,
                              serial_steps=0, pool_budget_log2=kb)
            pb[f"2^{kb}"] = {"workspace_bytes": r["workspace_bytes"], "segments": r["segments"],
                             "ms_per_step": round(r["ms_per_step"], 4)}
            log(f"[bench] pool budget 2^{kb}: {pb[f'2^{kb}']}")
        res["memory"]["pool_budget"] = pb
    cache5 = None
    if not args.no_decode:
        W5 = WORKLOADS["cfg5"]
        dec = {}
        for sd, tag in ((dla.DLA_F32, "f32"), (dla.DLA_BF16, "bf16")):
            d = decode_bench(args, torch, dla, W5, args.decode_steps, sd, f"decode {tag}")
            cache5 = d.pop("_cache", cache5)
            dec[tag] = d
            log(f"[bench] decode ({tag} states) {d['us_per_step_mean']} us/step")
        res["decode"] = dec["f32"]
        res["decode_bf16_states"] = dec["bf16"]
        few = W5.replace(B=1, T=8192)
        d = decode_bench(args, torch, dla, few, 64, dla.DLA_F32, "decode few heads")
        res["decode_few_heads"] = d
        log(f"[bench] decode (1x32 heads) {d['us_per_step_mean']} us/step")
        # Gated DeltaNet form of the step (the prefix is absorbed by the gated
        # prefill; only the timed steps take the delta rule)
        d = decode_bench(args, torch, dla, W5, args.decode_steps, dla.DLA_BF16,
                         "decode delta bf16", delta=True)
        d.pop("_cache", None)
        res["decode_delta_bf16_states"] = d
        log(f"[bench] decode delta (bf16 states) {d['us_per_step_mean']} us/step")
        if pk := res.get("peaks_measured"):
            for key in ("decode", "decode_bf16_states", "decode_few_heads",
                        "decode_delta_bf16_states"):
                res[key]["roofline"]["frac_measured_peak"] = frac(res[key]["roofline"]["achieved"],
                                                                  pk["hbm_read_gbs"])
    if not args.no_others:
        # the Gated DeltaNet form's prefill on the 4k-token and the 16k-token workloads
        dp = {}
        for name in ("cfg2", "cfg3"):
            dp[name] = delta_prefill_bench(args, torch, dla, WORKLOADS[name], 2)
            log(f"[bench] delta prefill {name}: {dp[name]}")
        res["prefill_delta"] = dp
    if not args.no_sweep:
        res["policy_sweep"] = policy_sweep(args, torch, dla)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(args, W)
        if cache5 is not None:
            res["cpu_baseline"]["decode"] = cpu_decode_baseline(args, torch, dla,
                                                                WORKLOADS["cfg5"], cache5)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
