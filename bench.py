"""Benchmark of the fused linear + cross-entropy forward + backward step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload llama3_8b] [--gpus 1]

One step = one lce_forward_backward call (loss, dH, dW) over the whole synthetic batch, inputs
already resident in HBM. Prints ONE JSON line with tokens/s, the fraction of the bf16 dense MFMA
peak (credited work 6*N*H*V), the live roofline of the dominant kernel (HIP events recorded by the
library on its launch stream), the forward-only rate (loss without gradients, 2*N*H*V), the step
with the final RMSNorm fused in front (lce_rmsnorm_forward_backward), a training step of the output
layer with host-resident weights and its hiding factor (lce_head_train_step), peak
device memory against a materialised-logits PyTorch baseline, the median and fastest single step,
the rate of the W streams (W's bytes per logits / dH launch over its duration), the three
contraction shapes of one chunk as plain hipBLASLt GEMMs (context), the steps of the other
workloads (Qwen2.5-7B, Mistral-Large, the small one; extra keys, not the headline), and the float64
CPU oracle timed on one whole forward + backward of the same workload, with the host's CPU model,
sockets, cores and BLAS library.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 4096 flop/clk x 2.4 GHz, dense
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
METRIC = "fused LCE fwd+bwd tokens/s and % bf16 MFMA peak (H=4096,V=128256,N=8192)"
KERNEL_SOURCES = ("paper_2603_16428_amd/csrc/lce_gemm.hpp", "paper_2603_16428_amd/csrc/lce_aux.hpp",
                  "paper_2603_16428_amd/csrc/lce_api.hip")


def kernel_source_hash() -> str:
    """Identifies the kernels a stored counter measurement belongs to."""
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, kind: str):
    """HBM bytes per launch of `kind` from the stored FETCH_SIZE / WRITE_SIZE summary.

    The summary (profiles/lce_hbm_traffic_<workload>.md) holds a JSON block written from two
    rocprofv3 --pmc runs of this script, both counters already scaled by what they read for a
    plain device copy of known size. Returns None when there is no summary or when the kernel
    sources have changed since the counters were taken.
    """
    path = os.path.join(ROOT, "profiles", f"lce_hbm_traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        m = re.search(r"```json\n(.*?)\n```", f.read(), re.S)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("source_hash") != kernel_source_hash() or rec.get("workload") != workload:
        return None
    k = rec.get("per_launch", {}).get(kind)
    return None if k is None else int(k["fetch_bytes"] + k["write_bytes"])


def copy_calibration(mib: int):
    """Plain device-to-device copies of known size: the yardstick for the HBM byte counters."""
    import torch
    n = mib << 20
    src = torch.ones(n, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    log(f"copy calibration: 3 copies of {n} bytes")
    del src, dst
    torch.cuda.empty_cache()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def host_info():
    """The host the CPU baseline runs on: CPU model, sockets, usable cores, BLAS library and threads."""
    model, sockets = None, set()
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                k, _, v = line.partition(":")
                k, v = k.strip(), v.strip()
                if k == "model name" and model is None:
                    model = v
                elif k == "physical id":
                    sockets.add(v)
    except OSError:
        pass
    blas = {}
    try:
        from threadpoolctl import threadpool_info
        for i in threadpool_info():
            if i.get("user_api") == "blas":
                blas = {"library": i.get("internal_api"), "version": i.get("version"),
                        "threads": int(i.get("num_threads", 1))}
                break
    except Exception:  # threadpoolctl missing
        pass
    return {"cpu_model": model, "sockets": len(sockets) or None, "affinity_cores": len(os.sched_getaffinity(0)),
            "blas": blas}


def cpu_baseline(d, tokens: int):
    """The float64 oracle, as it stands, on the first `tokens` tokens (all of V and H): by default
    the whole workload, one complete forward + backward."""
    import oracle
    info = host_info()
    threads = info["blas"].get("threads") or info["affinity_cores"]
    n = min(tokens, d["N"])
    X, y = d["hidden"][:n], d["labels"][:n]
    t = time.perf_counter()
    oracle.forward_backward(X, d["weight"], y, d["ignore_index"], d["reduction"], rows_per_block=256)
    dt = time.perf_counter() - t
    what = "all" if n == d["N"] else f"first {n} of"
    return {"value": n / dt, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{what} {d['N']} tokens of {d['name']} (V={d['V']}, H={d['H']}): one float64 "
                      f"forward+backward (loss, dH, dW) incl. the upcast, {dt:.1f} s",
            "seconds": round(dt, 2), "host": info}


def materialised_baseline(X, W, y, ignore_index, reduction, reps=3):
    """Peak memory and time of the plain PyTorch step that builds the N x V logits."""
    import torch
    import torch.nn.functional as F
    Xg = X.detach().clone().requires_grad_(True)
    Wg = W.detach().clone().requires_grad_(True)
    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    times = []
    for _ in range(reps):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        logits = Xg @ Wg.T
        loss = F.cross_entropy(logits.float(), y, ignore_index=ignore_index, reduction=reduction)
        gx, gw = torch.autograd.grad(loss, [Xg, Wg])
        e.record()
        torch.cuda.synchronize()
        times.append(s.elapsed_time(e))
        del logits, loss, gx, gw
    peak = torch.cuda.max_memory_allocated() - base
    del Xg, Wg
    torch.cuda.empty_cache()
    return peak, min(times)


def other_workload(lce, name, dtype_override, steps=10, warmup=3):
    """One more workload's step, timed like the main one (fewer steps): ms, tokens/s, fraction of
    the dense peak, and each contraction's share."""
    import torch
    import workloads
    t0 = time.time()
    d = workloads.make_inputs(name, seed=0, dtype=dtype_override)
    N, H, V = d["N"], d["H"], d["V"]
    dev = torch.device("cuda:0")
    X, W, y = d["hidden"].to(dev), d["weight"].to(dev), d["labels"].to(dev)
    plan = lce.plan_info(N, H, V, X.dtype, True, 0)
    ws = torch.empty(plan["workspace_bytes"], dtype=torch.uint8, device=dev)
    out = (torch.empty(1, dtype=torch.float32, device=dev), torch.empty_like(X), torch.empty_like(W))
    for _ in range(warmup):
        lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], 0, ws, out)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # The step time without per-kernel events (a short step's host work would show in it), then
    # the same steps again with them, for each kernel kind's share.
    a.record(stream)
    for _ in range(steps):
        lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], 0, ws, out)
    b.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / steps
    lce.timing_enable(True)
    for _ in range(steps):
        lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], 0, ws, out)
    torch.cuda.synchronize()
    kern = lce.timing_read()
    lce.timing_enable(False)
    peak = PEAK_FP32_TFLOPS if X.dtype == torch.float32 else PEAK_BF16_TFLOPS
    frac = 6.0 * N * H * V / (ms * 1e-3) / 1e12 / peak
    # The same step replayed from a HIP graph.
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    with torch.cuda.stream(side):
        lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], 0, ws, out)
    stream.wait_stream(side)
    torch.cuda.synchronize()
    cg = torch.cuda.CUDAGraph()
    with torch.cuda.graph(cg):
        lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], 0, ws, out)
    for _ in range(warmup):
        cg.replay()
    torch.cuda.synchronize()
    a.record(stream)
    for _ in range(steps):
        cg.replay()
    b.record(stream)
    torch.cuda.synchronize()
    gms = a.elapsed_time(b) / steps
    del cg
    rec = {"N": N, "H": H, "V": V, "dtype": d["dtype"], "reduction": d["reduction"], "steps": steps,
           "chunk_tokens": plan["chunk_tokens"], "chunks": plan["chunks"], "dh_splits": plan["dh_splits"],
           "ms_per_step": round(ms, 4), "tokens_per_s": round(N / (ms * 1e-3), 1), "mfma_peak_frac": round(frac, 4),
           "graph_replay_ms_per_step": round(gms, 4),
           "kernels_ms_per_step": {k: round(v[0] / steps, 4) for k, v in kern.items() if v[1]}}
    log(f"{name}: {ms:.3f} ms/step ({100 * frac:.1f}% of peak), graph replay {gms:.3f} ms/step; "
        f"inputs {time.time() - t0:.0f} s")
    del X, W, y, ws, out
    torch.cuda.empty_cache()
    return rec


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama3_8b")
    ap.add_argument("--dtype", choices=["bf16", "fp16", "fp32"], default=None,
                    help="override the workload's element type (same draws, rounded to this type)")
    ap.add_argument("--chunk", type=int, default=0, help="tokens per chunk (0 = automatic)")
    ap.add_argument("--cpu-sample-tokens", type=int, default=0, help="oracle tokens (0 = the whole workload)")
    ap.add_argument("--other-workloads", default="qwen25_7b,mistral_large,small_bf16",
                    help="comma-separated workloads whose step is also timed (extra keys); empty for none")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-memory", action="store_true", help="skip the materialised-logits comparison")
    ap.add_argument("--no-rmsnorm", action="store_true", help="skip timing the variant with the final RMSNorm")
    ap.add_argument("--no-blas", action="store_true", help="skip the hipBLASLt GEMMs timed as context")
    ap.add_argument("--no-graph", action="store_true", help="skip timing the step replayed from a HIP graph")
    ap.add_argument("--no-head-train", action="store_true",
                    help="skip the output-layer training step with host-resident weights")
    ap.add_argument("--vocab-blocks", type=int, default=8, help="pipeline blocks of the head training step")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="also run plain copies of this many MiB (yardstick for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2603_16428_amd as lce
    import workloads

    lce.load_library()
    log(f"kernel sources {kernel_source_hash()}")
    t0 = time.time()
    d = workloads.make_inputs(args.workload, seed=0, dtype=args.dtype)
    # The workload as reported (and as its stored counter summaries are named): the dtype is part
    # of it when it is not the workload's own.
    wl_name = args.workload if args.dtype is None else f"{args.workload}_{args.dtype}"
    N, H, V = d["N"], d["H"], d["V"]
    log(f"inputs {args.workload} N={N} H={H} V={V} ready in {time.time() - t0:.1f}s")
    dev = torch.device("cuda:0")
    X, W, y = d["hidden"].to(dev), d["weight"].to(dev), d["labels"].to(dev)
    dtype = X.dtype
    chunk = args.chunk or lce.auto_chunk_tokens(N, H, V, dtype)
    chunks = -(-N // chunk)

    torch.cuda.synchronize()
    base = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    ws = torch.empty(lce.workspace_size(N, H, V, dtype, True, args.chunk), dtype=torch.uint8, device=dev)
    out = (torch.empty(1, dtype=torch.float32, device=dev), torch.empty_like(X), torch.empty_like(W))
    lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], args.chunk, ws, out)
    torch.cuda.synchronize()
    # The library allocates nothing: its footprint is the workspace and outputs the caller passes.
    # (The allocator's own figure rounds the workspace's segment up to 2 MiB.)
    lce_alloc = torch.cuda.max_memory_allocated() - base
    lce_peak = sum(t.numel() * t.element_size() for t in (ws,) + out)
    ws_keep = ws

    for _ in range(args.warmup):
        lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], args.chunk, ws, out)
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps), loss {out[0].item():.6f}")

    stream = torch.cuda.current_stream()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    lce.timing_enable(True)
    torch.cuda.synchronize()
    start.record(stream)
    for k in range(args.steps):
        lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], args.chunk, ws, out)
        if k < args.steps - 1:
            marks[k].record(stream)
    stop.record(stream)
    torch.cuda.synchronize()
    total_ms = start.elapsed_time(stop)
    bounds = [start] + marks[:args.steps - 1] + [stop]
    per_step = sorted(bounds[k].elapsed_time(bounds[k + 1]) for k in range(args.steps))
    kern = lce.timing_read()
    lce.timing_enable(False)
    ms = total_ms / args.steps
    log(f"timed {args.steps} steps: {ms:.3f} ms/step; per kind: "
        + ", ".join(f"{k} {v[0] / args.steps:.3f} ms ({v[1]} launches)" for k, v in kern.items()))

    flops = 6.0 * N * H * V
    peak = PEAK_FP32_TFLOPS if dtype == torch.float32 else PEAK_BF16_TFLOPS  # fp16 dense = bf16 dense
    tflops = flops / (ms * 1e-3) / 1e12
    # Dominant kernel: the GEMM kind with the largest share of the step. Each of the three
    # contractions performs 2*N*H*V flops per step, spread over its launches.
    gemm_kinds = ("logits_lse_gemm", "dh_gemm", "dw_gemm")
    dom = max(gemm_kinds, key=lambda k: kern[k][0])
    dom_ms, dom_launches = kern[dom]
    per_launch_flops = 2.0 * N * H * V * args.steps / dom_launches
    achieved = per_launch_flops / (dom_ms / dom_launches * 1e-3) / 1e12
    roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": measured_traffic(wl_name, dom), "kernel": dom,
                "per_launch_flops": per_launch_flops, "avg_launch_ms": dom_ms / dom_launches,
                "all_kernels_ms_per_step": {k: round(v[0] / args.steps, 4) for k, v in kern.items()},
                "gemm_frac": {k: round(2.0 * N * H * V * args.steps / (kern[k][0] * 1e-3) / 1e12 / peak, 4)
                              for k in gemm_kinds}}
    # The W streams: both the logits and the dH contraction read all of W once per launch (V x H of
    # the dtype); their rate is W's bytes over the launch's duration.
    w_bytes = V * H * X.element_size()
    w_stream = {k: round(w_bytes / (kern[k][0] / kern[k][1] * 1e-3) / 1e9, 1)
                for k in ("logits_lse_gemm", "dh_gemm")}
    w_stream.update({"unit": "GB/s", "w_bytes_per_launch": w_bytes, "launches_per_step": chunks,
                     "hbm_peak_gbs": PEAK_HBM_GBS})
    log("W streams: " + ", ".join(f"{k} {v}" for k, v in w_stream.items()))

    # The same step captured once in a HIP graph and replayed (the library allocates nothing and
    # never synchronizes, so a caller can capture it): no host launch work per kernel.
    graph = None
    if not args.no_graph:
        side = torch.cuda.Stream()
        side.wait_stream(stream)
        with torch.cuda.stream(side):
            lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], args.chunk, ws, out)
        stream.wait_stream(side)
        torch.cuda.synchronize()
        cg = torch.cuda.CUDAGraph()
        with torch.cuda.graph(cg):
            lce.forward_backward(X, W, y, d["ignore_index"], d["reduction"], args.chunk, ws, out)
        for _ in range(args.warmup):
            cg.replay()
        torch.cuda.synchronize()
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for _ in range(args.steps):
            cg.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        gms = g0.elapsed_time(g1) / args.steps
        graph = {"ms_per_step": round(gms, 4), "tokens_per_s": round(N / (gms * 1e-3), 1),
                 "mfma_peak_frac": round(flops / (gms * 1e-3) / 1e12 / peak, 4)}
        del cg
        log(f"graph replay: {gms:.3f} ms/step")

    # Context: the three contraction shapes of one chunk as plain hipBLASLt GEMMs (torch.mm, 2-D
    # operands; no epilogue work, no log-sum-exp, no dlogits).
    blas = None
    if not args.no_blas and dtype != torch.float32:
        nc = chunk
        Xc = X[:nc]
        dZ = (torch.randn(nc, V, device=dev) * 1e-4).to(dtype)
        shapes = {"logits": (Xc, W.t()), "dh": (dZ, W), "dw": (dZ.t(), Xc)}
        blas = {}
        for name, (a, b) in shapes.items():
            for _ in range(3):
                c = a @ b
            torch.cuda.synchronize()
            b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            b0.record(stream)
            for _ in range(10):
                c = a @ b
            b1.record(stream)
            torch.cuda.synchronize()
            bms = b0.elapsed_time(b1) / 10
            blas[f"{name}_ms"] = round(bms, 4)
            blas[f"{name}_tflops"] = round(2.0 * nc * H * V / (bms * 1e-3) / 1e12, 1)
            del c
        del dZ, shapes
        torch.cuda.empty_cache()
        log("hipBLASLt context (one chunk's shapes): " + ", ".join(f"{k} {v}" for k, v in blas.items()))

    # Forward only (loss, no gradients): 2 N H V credited flops per call, reported beside the step.
    fws = torch.empty(lce.workspace_size(N, H, V, dtype, False), dtype=torch.uint8, device=dev)
    for _ in range(2):
        lce.forward(X, W, y, d["ignore_index"], d["reduction"], workspace=fws)
    torch.cuda.synchronize()
    f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    f0.record(stream)
    for _ in range(args.steps):
        lce.forward(X, W, y, d["ignore_index"], d["reduction"], workspace=fws)
    f1.record(stream)
    torch.cuda.synchronize()
    fms = f0.elapsed_time(f1) / args.steps
    del fws
    forward_only = {"ms_per_call": round(fms, 4), "tokens_per_s": round(N / (fms * 1e-3), 1),
                    "tflops": round(2.0 * N * H * V / (fms * 1e-3) / 1e12, 1),
                    "mfma_peak_frac": round(2.0 * N * H * V / (fms * 1e-3) / 1e12 / peak, 4)}
    log(f"forward only: {fms:.3f} ms/call")

    # The same step with the final RMSNorm in front (pre-norm rows and a gain drawn by the generator).
    rmsnorm = None
    if not args.no_rmsnorm:
        r = workloads.make_rmsnorm_inputs(args.workload, seed=0, dtype=args.dtype, base=d)
        h, gam = r["hidden"].to(dev), r["gamma"].to(dev)
        rws = torch.empty(lce.rmsnorm_workspace_size(N, H, V, dtype, True, args.chunk), dtype=torch.uint8, device=dev)
        for _ in range(2):
            lce.rmsnorm_forward_backward(h, gam, W, y, r["eps"], d["ignore_index"], d["reduction"], args.chunk, rws)
        torch.cuda.synchronize()
        r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        r0.record(stream)
        for _ in range(args.steps):
            lce.rmsnorm_forward_backward(h, gam, W, y, r["eps"], d["ignore_index"], d["reduction"], args.chunk, rws)
        r1.record(stream)
        torch.cuda.synchronize()
        rms = r0.elapsed_time(r1) / args.steps
        rmsnorm = {"ms_per_step": round(rms, 4), "tokens_per_s": round(N / (rms * 1e-3), 1),
                   "extra_ms_vs_lce": round(rms - ms, 4)}
        del h, gam, rws
        log(f"with the final RMSNorm fused: {rms:.3f} ms/step")

    # A training step of the output layer with its weights in host memory (FP32 master, AdamW on
    # the CPU, 16-bit pinned gradient and parameter buffers), pipelined over vocabulary blocks, and
    # the same work run phase after phase. Hiding factor eta = T_bwd / (T_d2h + T_update).
    head = None
    if not args.no_head_train and dtype != torch.float32:
        threads = min(16, len(os.sched_getaffinity(0)))
        st = lce.HeadState(W.clone())
        kw = dict(lr=1e-4, betas=(0.9, 0.95), weight_decay=0.01, ignore_index=d["ignore_index"],
                  reduction=d["reduction"], chunk_tokens=args.chunk, vocab_blocks=args.vocab_blocks,
                  threads=threads, workspace=ws_keep)
        rec = {}
        for name, overlap in (("pipelined", True), ("sequential", False)):
            lce.head_train_step(st, X, y, overlap=overlap, **kw)
            runs = [lce.head_train_step(st, X, y, overlap=overlap, **kw)[2] for _ in range(3)]
            rec[name] = {k: round(float(np.median([r[k] for r in runs])), 3) for k in runs[0]}
        p_ = rec["pipelined"]
        bwd = p_["gpu_ms"] - fms
        head = {"vocab_blocks": args.vocab_blocks, "threads": threads, "pipelined_ms": p_["step_ms"],
                "sequential_ms": rec["sequential"]["step_ms"], "gpu_ms": p_["gpu_ms"], "bwd_ms": round(bwd, 3),
                "d2h_ms": p_["d2h_ms"], "update_ms": p_["update_ms"], "h2d_ms": p_["h2d_ms"],
                "tail_ms": p_["tail_ms"], "eta": round(bwd / (p_["d2h_ms"] + p_["update_ms"]), 4),
                "phases_sequential": rec["sequential"]}
        del st
        log(f"head train step: pipelined {p_['step_ms']:.1f} ms, sequential {rec['sequential']['step_ms']:.1f} ms, "
            f"d2h {p_['d2h_ms']:.1f} ms, update {p_['update_ms']:.1f} ms, eta {head['eta']:.3f}")

    if args.copy_calibration:
        copy_calibration(args.copy_calibration)

    memory = {"lce_peak_bytes": int(lce_peak), "lce_allocator_peak_bytes": int(lce_alloc)}
    if not args.no_memory:
        del ws, ws_keep
        torch.cuda.empty_cache()
        mpeak, mtime = materialised_baseline(X, W, y, d["ignore_index"], d["reduction"])
        memory.update({"materialised_peak_bytes": int(mpeak), "reduction_vs_materialised": round(1 - lce_peak / mpeak, 4),
                       "materialised_ms_per_step": round(mtime, 3)})
        log(f"materialised baseline: peak {mpeak / 1e9:.2f} GB, {mtime:.2f} ms; LCE peak {lce_peak / 1e9:.2f} GB")

    result = {
        "metric": METRIC, "value": round(N / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "ms_per_step_median": round(per_step[len(per_step) // 2], 4), "ms_per_step_min": round(per_step[0], 4),
        "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None,
        "dtype": {torch.bfloat16: "bf16", torch.float16: "f16", torch.float32: "f32"}[dtype],
        "data": "synthetic", "tflops": round(tflops, 1), "mfma_peak_frac": round(tflops / peak, 4),
        "config": {"workload": wl_name,
                   "N": N, "H": H, "V": V, "reduction": d["reduction"],
                   "chunk_tokens": chunk, "chunks": chunks, "seed": 0},
        "roofline": roofline, "w_stream": w_stream, "graph_replay": graph, "forward_only": forward_only,
        "rmsnorm_fused": rmsnorm,
        "head_train_step": head, "memory": memory, "hipblaslt_context": blas,
    }
    others = [w for w in args.other_workloads.split(",") if w]
    if others:
        del X, W, out
        torch.cuda.empty_cache()
        result["other_workloads"] = {w: other_workload(lce, w, args.dtype) for w in others}
    if not args.no_cpu_baseline:
        log("timing the float64 oracle on the host cores ...")
        result["cpu_baseline"] = cpu_baseline(d, args.cpu_sample_tokens or d["N"])
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
