#!/usr/bin/env python3
"""Throughput of biased graph attention (forward + backward) on one MI355X.

One step = gt_attn_fwd followed by the backward (gt_attn_bwd's three
stages, launched one by one through gt_attn_bwd_phase so that each kernel is
bracketed by HIP events on the stream it runs on) over the clustered-graph
workload: N = 131072 nodes, H = 8 heads, head dim 64, bf16, spd from BFS on
a 64-community planted-partition graph (17.2 GB of uint8 in HBM), bias
table [8, 64].

FLOP convention (non-causal attention): forward 4 N^2 d H, backward
10 N^2 d H (the recomputed S plus the dP, dV, dK and dQ products), so one
step is 14 N^2 d H = 1.2315e14 FLOP; softmax, bias and table-gradient work
are not counted.

Prints ONE JSON line. Inputs are synthetic and seeded; they are generated
and copied to the GPU before the timed region.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import platform
import statistics
import sys
import time
from pathlib import Path

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

PEAK_BF16 = 2516.6e12        # MI355X dense bf16 matrix-core FLOP/s
PEAK_HBM = 8.0e12            # MI355X HBM3E bytes/s


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="sbm128k", choices=("sbm128k", "ba16k"),
                   help="single-layer bf16 workload (the headline is sbm128k)")
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--cpu-rows", type=int, default=512,
                   help="query rows of the oracle CPU baseline sample")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--hbm-probe", action="store_true",
                   help="also time one read-only pass over the resident spd matrix (a torch "
                        "reduction over it as int64 words: the achievable rate for the spd "
                        "stream) and add it to the line")
    p.add_argument("--batch", default=None, metavar="B,N,d",
                   help="instead of the headline, time a batch of B graphs of N nodes (H = 8, "
                        "head dim d, bf16, 64 spd buckets, i.i.d. uniform spd per graph) through "
                        "the batched entry points and print one JSON line for it")
    p.add_argument("--copy-calibration", action="store_true",
                   help="run one plain 1 GiB device copy before the timed region (its "
                        "FETCH_SIZE / WRITE_SIZE counters calibrate the kernels')")
    return p.parse_args()


def make_device_inputs(w, seed, dev):
    import numpy as np
    import torch

    t0 = time.time()
    N = w.N
    spd = torch.empty((N, N), dtype=torch.uint8, device=dev)
    chunk = min(N, 8192)
    host = torch.empty((chunk, N), dtype=torch.uint8, pin_memory=True)
    hv = host.numpy()
    for r0 in range(0, N, chunk):
        n = min(chunk, N - r0)
        w.spd_block(r0, n, seed=seed, out=hv[:n])
        spd[r0:r0 + n].copy_(host[:n])
    torch.cuda.synchronize()
    log(f"spd {N}x{N} generated and uploaded in {time.time() - t0:.1f}s")
    td = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    q, k, v = w.qkv(seed)
    do = w.d_out(seed)

    def up(x):
        return torch.from_numpy(x).to(td).to(dev)

    Q, K, V, dO = up(q), up(k), up(v), up(do)
    T = torch.from_numpy(w.table(seed)).to(dev)
    del q, k, v, do
    log(f"inputs ready in {time.time() - t0:.1f}s")
    return dict(q=Q, k=K, v=V, do=dO, table=T, spd=spd)


def run_gpu(w, args, dev):
    import torch

    import paper_2609_34420_amd as gt

    x = make_device_inputs(w, args.seed, dev)
    H, N, d = w.H, w.N, w.d
    scale = w.scale()
    O = torch.empty_like(x["q"])
    L = torch.empty((H, N), dtype=torch.float32, device=dev)
    grads = (torch.empty_like(x["q"]), torch.empty_like(x["k"]), torch.empty_like(x["v"]),
             torch.empty_like(x["table"]))
    ws = torch.empty(gt.gt_attn_bwd_workspace_size(H, N, d, x["q"].dtype), dtype=torch.uint8,
                     device=dev)
    stream = torch.cuda.current_stream()
    # BFS distances on an undirected graph are symmetric: spd is its own
    # transpose, which lets the key-stationary stage read rows.
    spd_t = x["spd"] if w.spd_symmetric else None

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        gt.gt_attn_fwd(x["q"], x["k"], x["v"], x["spd"], x["table"], scale=scale, out=O, lse=L)
        if ev is not None:
            ev[1].record(stream)
        for ph in range(3):
            gt.gt_attn_bwd_phase(ph, x["q"], x["k"], x["v"], x["spd"], x["table"], O, L, x["do"],
                                 scale=scale, workspace=ws, grads=grads, spd_t=spd_t)
            if ev is not None:
                ev[2 + ph].record(stream)

    probe = None
    if args.hbm_probe:
        spd = x["spd"]
        words = spd.view(-1).view(torch.int64)     # the same bytes, 8 to a word
        torch.sum(words)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(5):
            torch.sum(words)
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / 5
        probe = {"what": "torch.sum over the spd matrix read as int64 words (read-only pass)",
                 "bytes": spd.numel(), "ms": ms, "GB_per_s": spd.numel() / (ms * 1e-3) / 1e9}
        log(f"HBM probe: {spd.numel() / 1e9:.2f} GB read in {ms:.3f} ms = {probe['GB_per_s']:.0f} GB/s")

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("copy calibration: 1 GiB device-to-device copy done")

    for i in range(args.warmup):
        step()
        torch.cuda.synchronize()
        log(f"warmup step {i + 1}/{args.warmup} done")

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for s in range(args.steps):
        step(evs[s])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = {"fwd": [], "bwd_prep": [], "bwd_dkdv": [], "bwd_dq": [], "step": []}
    for e in evs:
        per["fwd"].append(e[0].elapsed_time(e[1]))
        per["bwd_prep"].append(e[1].elapsed_time(e[2]))
        per["bwd_dkdv"].append(e[2].elapsed_time(e[3]))
        per["bwd_dq"].append(e[3].elapsed_time(e[4]))
        per["step"].append(e[0].elapsed_time(e[4]))
    total_ms = evs[0][0].elapsed_time(evs[-1][4])
    log(f"timed {args.steps} steps: {total_ms:.1f} ms (events), {wall * 1e3:.1f} ms (wall)")
    for kname, v in per.items():
        log(f"  {kname:9s} mean {sum(v) / len(v):9.3f} ms  min {min(v):9.3f} ms")
    return total_ms, wall, per, probe


_KERNEL_FILES = {"fwd": "fwd_bf16_kernel", "bwd_dkdv": "bwd_dkdv_bf16_kernel",
                 "bwd_dq": "bwd_dq_bf16_kernel"}


# Device sources of the timed kernels (the host-side C ABI and the merge
# kernel do not change what the counters measured).
_HOST_OR_UNTIMED = {"api.hip", "merge.hip"}


def kernel_sources_sha256() -> str:
    h = hashlib.sha256()
    for p in sorted((ROOT / "paper_2609_34420_amd" / "csrc").glob("*.[hc]*")):
        if p.name in _HOST_OR_UNTIMED:
            continue
        h.update(p.name.encode())
        h.update(p.read_bytes())
    return h.hexdigest()


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch (calibrated FETCH_SIZE + WRITE_SIZE) recorded under
    profiles/, or None when the kernels changed since the counters were taken."""
    f = ROOT / "profiles" / f"traffic_{workload}.json"
    if not f.exists():
        return None
    rec = json.loads(f.read_text())
    if rec.get("kernel_source_sha256") != kernel_sources_sha256():
        return None
    k = rec["kernels"].get(_KERNEL_FILES[kernel])
    return None if k is None else k["fetch_bytes"] + k["write_bytes"]


def cpu_baseline(w, args):
    """The oracle (fp64 NumPy) on a bounded row sample of the same workload:
    forward for R query rows against all N keys, and the backward of those
    rows; credited 14 R N d H FLOP."""
    import numpy as np

    import oracle

    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()
                            if i.get("user_api") == "blas"] or [1])
    except Exception:
        blas_threads = 1
    R = args.cpu_rows
    rows = w.sample_rows(R - 2, seed=args.seed)
    q, k, v = w.qkv(args.seed)
    do = w.d_out(args.seed)
    table = w.table(args.seed)
    spd_rows = w.spd_rows(rows, seed=args.seed)
    qr, dor = q[:, rows], do[:, rows]
    t0 = time.perf_counter()
    oracle.block_attention(qr, k, v, spd_rows, table, w.scale())
    oracle.block_backward(qr, k, v, spd_rows, table, w.scale(), dor)
    dt = time.perf_counter() - t0
    flop = 14.0 * len(rows) * w.N * w.d * w.H
    log(f"oracle sample: {len(rows)} rows fwd+bwd in {dt:.1f}s on {blas_threads} BLAS threads")
    return {"value": flop / dt / 1e12, "unit": "TFLOP/s", "cores": int(blas_threads),
            "kind": "oracle",
            "sample": (f"{len(rows)} seeded query rows of N={w.N} against all keys, forward and "
                       f"backward in fp64 NumPy ({dt:.1f} s); credited 14*R*N*d*H FLOP; elementwise "
                       f"NumPy is single-threaded, matrix products use {blas_threads} BLAS threads; "
                       f"host {platform.processor() or platform.machine()}, os.cpu_count()={os.cpu_count()}")}


def run_batch(args):
    """Batches of short graphs (the paper's training batches of sampled
    sequences) through gt_attn_fwd_batch / gt_attn_bwd_batch."""
    import torch

    import paper_2609_34420_amd as gt

    B, N, d = (int(x) for x in args.batch.split(","))
    H, nb = 8, 64
    dev = "cuda:0"
    torch.cuda.set_device(0)
    g = torch.Generator(device=dev)
    g.manual_seed(args.seed)
    shape = (B, H, N, d)
    q, k, v = ((torch.randn(shape, device=dev, generator=g) / math.sqrt(d)).bfloat16() for _ in range(3))
    do = torch.randn(shape, device=dev, generator=g).bfloat16()
    spd = torch.randint(0, nb, (B, N, N), dtype=torch.uint8, device=dev, generator=g)
    table = torch.randn(H, nb, device=dev, generator=g) * 0.02
    scale = 1.0 / math.sqrt(d)
    O = torch.empty_like(q)
    L = torch.empty((B, H, N), dtype=torch.float32, device=dev)
    grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v), torch.empty_like(table))
    ws = torch.empty(gt.gt_attn_bwd_workspace_size(B * H, N, d, torch.bfloat16), dtype=torch.uint8,
                     device=dev)
    stream = torch.cuda.current_stream()

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        gt.gt_attn_fwd_batch(q, k, v, spd, table, scale=scale, out=O, lse=L)
        if ev is not None:
            ev[1].record(stream)
        gt.gt_attn_bwd_batch(q, k, v, spd, table, O, L, do, scale=scale, workspace=ws, grads=grads)
        if ev is not None:
            ev[2].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    for e in evs:
        step(e)
    torch.cuda.synchronize()
    fwd = [e[0].elapsed_time(e[1]) for e in evs]
    bwd = [e[1].elapsed_time(e[2]) for e in evs]
    ms = sum(f + b for f, b in zip(fwd, bwd)) / args.steps
    elems = float(B) * H * N * N
    flop = 14.0 * elems * d
    print(json.dumps({
        "metric": f"batched biased-attention fwd+bwd at B={B}, N={N}, H={H}, d={d}",
        "value": flop / (ms * 1e-3) / 1e12, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "dtype": "bf16",
        "data": "synthetic", "score_elements_per_ns": elems / (ms * 1e6),
        "kernel_ms": {"fwd": sum(fwd) / len(fwd), "bwd": sum(bwd) / len(bwd)},
        "config": {"workload": f"batch of {B} graphs of {N} nodes, i.i.d. uniform spd over {nb} "
                               f"buckets, H={H}, d={d}, bf16", "parallelism": "single GPU"},
    }), flush=True)


def graph_label(w) -> str:
    kind = w.graph[0]
    if kind == "sbm":
        return f"clustered planted-partition graph, {w.graph[1]} communities"
    if kind == "ba":
        return f"Barabasi-Albert graph, m={w.graph[1]}"
    return f"Erdos-Renyi graph, average degree {w.graph[1]}"


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; the context-parallel "
                          "ring across GPUs is not built (see the single-GPU ring step), "
                          f"asked for --gpus {args.gpus} / WORLD_SIZE {world}"}))
        sys.exit(2)
    if args.batch:
        run_batch(args)
        return
    import torch

    import synth

    w = synth.workload(args.workload)
    dev = "cuda:0"
    torch.cuda.set_device(0)
    total_ms, wall, per, probe = run_gpu(w, args, dev)
    K = args.steps
    ms = total_ms / K
    flop = w.flops_fwd_bwd
    tflops = flop / (ms * 1e-3) / 1e12

    N2dH = float(w.N) * w.N * w.d * w.H
    kernels = {
        "bwd_dkdv": (8.0 * N2dH, "dK/dV/dtable kernel: S recompute, dP, dV, dK products (8 N^2 d H)"),
        "fwd": (4.0 * N2dH, "forward kernel: Q K^T and P V products (4 N^2 d H)"),
        "bwd_dq": (2.0 * N2dH, "dQ kernel: the dQ product (2 N^2 d H credited; its S and dP "
                               "recomputation is not)"),
    }
    mean = {k: sum(v) / len(v) for k, v in per.items()}
    dom = max(("fwd", "bwd_dkdv", "bwd_dq"), key=lambda k: mean[k])
    achieved = kernels[dom][0] / (mean[dom] * 1e-3)
    traffic = measured_traffic(w.name, dom)
    roofline = {"bound": "mfma", "achieved": achieved / 1e12, "peak": PEAK_BF16 / 1e12,
                "unit": "TFLOP/s", "frac": achieved / PEAK_BF16, "traffic": traffic,
                "kernel": dom, "kernel_ms": mean[dom], "flop_per_launch": kernels[dom][0],
                "flop_rule": kernels[dom][1]}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args)

    out = {
        "metric": f"biased-attention fwd+bwd TFLOP/s and % bf16 MFMA peak at N={w.N}, H={w.H}, d={w.d}",
        "value": tflops,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "strong",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "pct_of_bf16_peak": 100.0 * tflops * 1e12 / PEAK_BF16,
        "config": {"workload": f"{w.name}: {graph_label(w)}, N={w.N}, H={w.H}, d={w.d}, "
                               f"{w.n_buckets} spd buckets, bf16",
                   "N": w.N, "H": w.H, "d": w.d, "n_buckets": w.n_buckets,
                   "flop_per_step": flop, "parallelism": "single GPU"},
        "kernel_ms": mean,
        "step_ms_stats": {"mean": ms, "median": statistics.median(per["step"]),
                          "min": min(per["step"]), "max": max(per["step"])},
        "wall_ms_per_step": wall * 1e3 / K,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if probe is not None:
        out["hbm_probe"] = probe
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
