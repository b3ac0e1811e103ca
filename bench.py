#!/usr/bin/env python3
"""Benchmark of the DLA layer forward on one MI355X.

One step = one prefill of the 16k-token workload from an empty cache (B=4,
H=16, T=16384, d_k=d_v=128, C=128, tau=0.5, bf16 inputs, float32 states,
long stable spans alternating with short i.i.d. bursts): token frames, the
boundary scan with the capacity schedule, and the readout + state update --
every step of the hot path.  `value` is prefill tokens/s (B*T tokens per step)
with all inputs resident in HBM.

Also reported on the same line:
  * roofline of the dominant kernel (the readout) from HIP events that the
    library records around each of its launches in the timed steps (the
    prefill is pipelined: the scan runs on a second stream, segment by
    segment, beside the update and readout of the segments already scanned);
    the stage breakdown comes from three more steps run with serial stages;
  * the decode step at C = 128 on full caches built from a 32k-token prefix
    (B=64, H=32): mean and median microseconds per step over 256 steps, with
    its HBM roofline;
  * cpu_baseline: the float64 oracle on a bounded sample of the prefill
    workload, timed on the host cores.

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
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
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


def prefill_bench(args, torch, dla, W):
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
    ws = torch.empty(max(dla.workspace_bytes(cache, T, k.dtype),
                         dla.workspace_bytes(cache, T, k.dtype, serial=True)),
                     dtype=torch.uint8, device="cuda")
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
                    serial=serial)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # the timed steps: the pipelined prefill, with every readout launch
    # bracketed by a pair of events on the stream it runs on
    nseg = dla.prefill_segments(cache, T, k.dtype)
    revs = [[torch.cuda.Event(enable_timing=True) for _ in range(2 * nseg)]
            for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    for e in [start, stop] + [e for r in revs for e in r]:
        e.record()   # created here, outside the timed region
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record()
    for i in range(args.steps):
        step(rev=revs[i])
    stop.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / args.steps
    log(f"[bench] prefill wall clock {ms:.3f} ms/step, "
        f"events {start.elapsed_time(stop) / args.steps:.3f} ms/step")
    ro_launch = np.array([[r[2 * j].elapsed_time(r[2 * j + 1]) for j in range(nseg)] for r in revs])
    ro_ms = float(ro_launch.sum(axis=1).mean())   # readout time per step, all launches
    # stage breakdown: the same step with the stages one after another
    ns = len(dla.PREFILL_STAGES)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(ns + 1)] for _ in range(3)]
    for e in evs:
        step(events=e, serial=True)
    torch.cuda.synchronize()
    stages = np.array([[e[i].elapsed_time(e[i + 1]) for i in range(ns)] for e in evs])
    st_ms = stages.mean(axis=0)

    # algorithmic work of the readout kernel, from this run's exports: the sum
    # over tokens of 2 m_t d_k d_v (the readout over the m_t live states)
    b = bnd.cpu().numpy().reshape(B * H, T).astype(np.int64)
    mm = (mrg.cpu().numpy().reshape(B * H, T) >= 0).astype(np.int64)
    m_t = np.cumsum(b, axis=1) - np.cumsum(mm, axis=1)
    flops = 2.0 * W.dk * W.dv * m_t.sum()
    flops_cap = 2.0 * W.dk * W.dv * W.C * m_t.size
    achieved = flops / (ro_ms * 1e-3) / 1e12
    return {
        "ms_per_step": ms,
        "value": B * T / (ms * 1e-3),
        "stages_ms_serial": dict(zip(dla.PREFILL_STAGES, [round(float(s), 4) for s in st_ms])),
        "roofline": {"kernel": "prefill_readout_kernel", "bound": "mfma",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": counter_traffic("prefill_readout_kernel", W.name),
                     "launches_per_step": nseg,
                     "launch_ms_mean": round(float(ro_launch.mean()), 4),
                     "flops_per_launch": flops / nseg,
                     "flops_per_launch_at_m_eq_C": flops_cap / nseg},
        "decisions": {"boundaries": int(b.sum()), "merges": int(mm.sum()),
                      "mean_live_states": round(float(m_t.mean()), 2)},
    }


def decode_bench(args, torch, dla, W):
    from paper_2606_10650_amd.workloads import make_decode_tokens, make_prefix_torch
    t0 = time.time()
    _, k, v, g = make_prefix_torch(W, "cuda")
    torch.cuda.synchronize()
    log(f"[bench] decode prefix {W.label} drawn on device in {time.time() - t0:.1f}s")
    cache = dla.cache_alloc(W.B, W.H, W.C, W.dk, W.dv)
    t0 = time.time()
    dla.prefill(cache, None, k, v, g, None, tau=W.tau, skip_readout=True, want_exports=False)
    torch.cuda.synchronize()
    log(f"[bench] decode prefix absorbed in {time.time() - t0:.1f}s")
    del k, v, g
    torch.cuda.empty_cache()
    steps = args.decode_steps
    x = make_decode_tokens(W, steps=steps + 2)

    def dev(a, shape):
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).reshape(shape).cuda()

    nh = W.B * W.H
    q = dev(x["q"], (W.B, W.H, steps + 2, W.dk)).permute(2, 0, 1, 3).contiguous()
    kk = dev(x["k"], (W.B, W.H, steps + 2, W.dk)).permute(2, 0, 1, 3).contiguous()
    vv = dev(x["v"], (W.B, W.H, steps + 2, W.dv)).permute(2, 0, 1, 3).contiguous()
    lam = dev(x["lam"], (W.B, W.H, steps + 2, W.C)).permute(2, 0, 1, 3).contiguous()
    gg = torch.from_numpy(x["g"]).reshape(W.B, W.H, steps + 2).permute(2, 0, 1).contiguous().cuda()
    out = torch.empty((W.B, W.H, W.dv), dtype=torch.bfloat16, device="cuda")
    bnd = torch.empty((steps, W.B, W.H), dtype=torch.int8, device="cuda")
    mrg = torch.empty((steps, W.B, W.H), dtype=torch.int32, device="cuda")
    m_before = dla.cache_export(cache, heads=[0])["m"][0]
    # warm-up on a copy of the cache, then 256 timed steps on the prefix cache
    warm = dla.StateCache(W.B, W.H, W.C, W.dk, W.dv, cache.buf.clone())
    for i in range(2):
        dla.decode_step(warm, q[i], kk[i], vv[i], gg[i], lam[i], tau=W.tau, out=out,
                        want_exports=False)
    torch.cuda.synchronize()
    del warm
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    evs[0].record()
    for i in range(steps):
        dla.decode_step(cache, q[i + 2], kk[i + 2], vv[i + 2], gg[i + 2], lam[i + 2], tau=W.tau,
                        out=out, boundary=bnd[i], merge_idx=mrg[i], score=None)
        evs[i + 1].record()
    torch.cuda.synchronize()
    us = np.array([evs[i].elapsed_time(evs[i + 1]) * 1e3 for i in range(steps)])
    nb = int(bnd.sum().item())
    nm = int((mrg >= 0).sum().item())
    # HBM bytes per step: every live state read once (float32), plus the written
    # states (merged pair and new state, or the accumulated newest state), plus
    # the token vectors, lambda row and output
    m_live = W.C  # full caches
    per_head = m_live * W.dk * W.dv * 4 + 2 * W.dk * W.dv * 4 + (2 * W.dk + W.dv + W.C + W.dv) * 2
    bytes_step = per_head * nh
    ach = bytes_step / (np.mean(us) * 1e-6) / 1e9
    return {
        "config": {"workload": f"decode {W.B}x{W.H} heads, C={W.C}, d={W.dk}, prefix {W.T} tokens",
                   "B": W.B, "H": W.H, "C": W.C, "prefix_tokens": W.T, "steps": steps},
        "us_per_step_mean": round(float(np.mean(us)), 2),
        "us_per_step_p50": round(float(np.median(us)), 2),
        "live_states_before": int(m_before),
        "boundaries": nb, "merges": nm,
        "roofline": {"kernel": "decode_kernel", "bound": "hbm", "achieved": round(ach, 1),
                     "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
                     "traffic": counter_traffic("decode_kernel", W.name),
                     "bytes_per_launch": bytes_step},
    }


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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="cfg3")
    ap.add_argument("--decode-steps", type=int, default=256)
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=16384)
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the DLA layer shards over (batch, head) with no "
              "exchange between GPUs, and this build runs on a single MI355X (--gpus 1).",
              file=sys.stderr)
        sys.exit(2)
    import torch
    if args.copy_probe_mib:
        copy_probe(args, torch)
        return
    from paper_2606_10650_amd import dla
    from paper_2606_10650_amd.workloads import WORKLOADS
    W = WORKLOADS[args.workload]
    pre = prefill_bench(args, torch, dla, W)
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
    }
    if not args.no_decode:
        res["decode"] = decode_bench(args, torch, dla, WORKLOADS["cfg5"])
        log(f"[bench] decode {res['decode']['us_per_step_mean']} us/step")
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(args, W)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
