#!/usr/bin/env python3
"""Throughput of biased graph attention (forward + backward) on one MI355X.

Default workload (the headline): one step = gt_attn_fwd followed by the
backward (gt_attn_bwd's three stages, launched one by one through
gt_attn_bwd_phase so that each kernel is bracketed by HIP events on the
stream it runs on) at N = 131072 nodes, H = 8 heads, head dim 64, bf16, spd
from BFS on a 64-community planted-partition graph (17.2 GB of uint8 in
HBM), bias table [8, 64].

Other workloads (--workload):
  ba16k    N = 16384, H = 8, d = 64, bf16, Barabasi-Albert spd, 32 buckets
  tiny     N = 512, H = 4, d = 32, fp32 (vector-ALU kernels), 22 buckets
  cp256k   one device's share of the context-parallel ring at N = 262144:
           query shard 3 of 8 (32768 rows, with only its spd rows) against
           the 8 KV blocks in ring order, merged in place; the step is the
           forward ring, and the backward ring over the same blocks is
           timed beside it
  deep32k  a 12-layer stack at N = 32768, H = 16, d = 64, bf16, 256 Zipf
           buckets: the forward of layers 1..12, then the backward of
           layers 12..1

FLOP convention (non-causal attention): forward 4 N^2 d H, backward
10 N^2 d H (the recomputed S plus the dP, dV, dK and dQ products), so one
step of one layer is 14 N^2 d H (1.2315e14 at the headline); softmax, bias
and table-gradient work are not counted.

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
import subprocess
import sys
import time
from pathlib import Path

ROOT = Path(__file__).resolve().parent
sys.path.insert(0, str(ROOT))

PEAK_BF16 = 2516.6e12        # MI355X dense bf16 matrix-core FLOP/s
PEAK_F32_VALU = 157.3e12     # MI355X fp32 vector FLOP/s
PEAK_HBM = 8.0e12            # MI355X HBM3E bytes/s
WORKLOADS = ("sbm128k", "ba16k", "tiny", "cp256k", "deep32k")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="sbm128k", choices=WORKLOADS,
                   help="the headline is sbm128k")
    p.add_argument("--seed", type=int, default=0)
    p.add_argument("--cpu-rows", type=int, default=512,
                   help="query rows of the oracle CPU baseline sample (row-sampled workloads)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--hbm-probe", action="store_true",
                   help="also time one read-only pass over the resident spd matrix (a torch "
                        "reduction over it as int64 words: the achievable rate for the spd "
                        "stream) and add it to the line")
    p.add_argument("--batch", default=None, metavar="B,N,d",
                   help="instead of a workload, time a batch of B graphs of N nodes (H = 8, "
                        "head dim d, bf16, 64 spd buckets, i.i.d. uniform spd per graph) through "
                        "the batched entry points and print one JSON line for it")
    p.add_argument("--copy-calibration", action="store_true",
                   help="run one plain 1 GiB device copy before the timed region (its "
                        "FETCH_SIZE / WRITE_SIZE counters calibrate the kernels')")
    return p.parse_args()


# ---------------------------------------------------------------------------
# host and timing helpers
# ---------------------------------------------------------------------------
def host_record() -> dict:
    """The host the CPU baseline ran on: CPU model, sockets, physical cores,
    logical CPUs visible to this process and the BLAS thread setting."""
    rec = {"os_cpu_count": os.cpu_count(), "machine": platform.machine()}
    try:
        rec["sched_affinity"] = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        pass
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        kv = {}
        for line in out.splitlines():
            if ":" in line:
                a, b = line.split(":", 1)
                kv[a.strip()] = b.strip()
        rec["model_name"] = kv.get("Model name")
        sockets = int(kv.get("Socket(s)", "0") or 0)
        per = int(kv.get("Core(s) per socket", "0") or 0)
        rec["sockets"] = sockets
        rec["physical_cores"] = sockets * per if sockets and per else None
        rec["threads_per_core"] = kv.get("Thread(s) per core")
    except (OSError, ValueError, subprocess.SubprocessError):
        rec["model_name"] = platform.processor() or None
    try:
        from threadpoolctl import threadpool_info
        rec["blas_threads"] = max([i.get("num_threads", 1) for i in threadpool_info()
                                   if i.get("user_api") == "blas"] or [1])
    except Exception:
        rec["blas_threads"] = 1
    return rec


class Timer:
    """HIP events recorded on the launch stream around named launches."""

    def __init__(self, stream):
        import torch
        self.torch = torch
        self.stream = stream
        self.marks = []

    def mark(self, name):
        e = self.torch.cuda.Event(enable_timing=True)
        e.record(self.stream)
        self.marks.append((name, e))

    def per_name(self):
        """Milliseconds between each mark and the next, summed by the name of
        the interval's opening mark; also the number of intervals."""
        tot, cnt = {}, {}
        for (n, a), (_, b) in zip(self.marks, self.marks[1:]):
            if n is None:
                continue
            tot[n] = tot.get(n, 0.0) + a.elapsed_time(b)
            cnt[n] = cnt.get(n, 0) + 1
        return tot, cnt


def timed_steps(step, args, stream):
    """W untimed warmup steps, then K timed steps each bracketed by events;
    returns (per-step ms list, per-kernel mean ms per launch, launches per
    step, wall ms per step)."""
    import torch
    for i in range(args.warmup):
        step(None)
        torch.cuda.synchronize()
        log(f"warmup step {i + 1}/{args.warmup} done")
    timers = [Timer(stream) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in timers:
        t.mark("step")
        step(t)
        t.mark(None)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / args.steps
    steps = [t.marks[0][1].elapsed_time(t.marks[-1][1]) for t in timers]
    tot, cnt = {}, {}
    for t in timers:
        a, c = t.per_name()
        for n in a:
            if n == "step":
                continue
            tot[n] = tot.get(n, 0.0) + a[n]
            cnt[n] = cnt.get(n, 0) + c[n]
    per_launch = {n: tot[n] / cnt[n] for n in tot}
    launches = {n: cnt[n] // args.steps for n in cnt}
    log(f"timed {args.steps} steps: mean {sum(steps) / len(steps):.3f} ms (events), {wall:.3f} ms (wall)")
    for n in per_launch:
        log(f"  {n:12s} {per_launch[n]:9.3f} ms per launch x {launches[n]}")
    return steps, per_launch, launches, wall


def upload_spd(w, seed, dev, rows=None):
    import torch
    r0, r1 = (0, w.N) if rows is None else rows
    n = r1 - r0
    spd = torch.empty((n, w.N), dtype=torch.uint8, device=dev)
    chunk = min(n, 8192)
    host = torch.empty((chunk, w.N), dtype=torch.uint8, pin_memory=True)
    hv = host.numpy()
    for a in range(0, n, chunk):
        m = min(chunk, n - a)
        w.spd_block(r0 + a, m, seed=seed, out=hv[:m])
        spd[a:a + m].copy_(host[:m])
    torch.cuda.synchronize()
    return spd


def device_tensors(w, seed, dev, layer=0):
    import torch
    td = torch.bfloat16 if w.dtype == "bf16" else torch.float32

    def up(x):
        return torch.from_numpy(x).to(td).to(dev)

    q, k, v = w.qkv(seed, layer=layer)
    x = dict(q=up(q), k=up(k), v=up(v), do=up(w.d_out(seed, layer=layer)),
             table=torch.from_numpy(w.table(seed, layer=layer)).to(dev))
    return x


def dtable_spread(runs):
    """Run-to-run spread of dtable over repeated backward runs on identical
    inputs (its reduction order varies): largest |difference| to the first
    run, absolute and relative to the largest |dtable|."""
    base = runs[0]
    diff = max(float((r - base).abs().max()) for r in runs[1:])
    scale = float(base.abs().max())
    return {"runs": len(runs), "max_abs_diff": diff,
            "max_rel_diff": diff / scale if scale > 0 else 0.0}


# The kernel symbol behind each timed launch name.
KERNEL_SYMBOLS = {"fwd": "fwd_bf16_kernel", "fwd_ring_step": "fwd_bf16_kernel",
                  "bwd_prep": "bwd_prep_kernel", "bwd_dkdv": "bwd_dkdv_bf16_kernel",
                  "bwd_dq": "bwd_dq_bf16_kernel", "fwd_valu": "fwd_valu_kernel",
                  "bwd_dkdv_valu": "bwd_dkdv_valu_kernel", "bwd_dq_valu": "bwd_dq_valu_kernel"}


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch (calibrated FETCH_SIZE + WRITE_SIZE) recorded under
    profiles/, or None when the kernels changed since the counters were taken."""
    f = ROOT / "profiles" / f"traffic_{workload}.json"
    if not f.exists():
        return None
    rec = json.loads(f.read_text())
    if rec.get("kernel_source_sha256") != kernel_sources_sha256():
        return None
    k = rec["kernels"].get(KERNEL_SYMBOLS.get(kernel, kernel))
    return None if k is None else k["fetch_bytes"] + k["write_bytes"]


# Device sources of the kernels the traffic record measured: every source
# except the host-side C ABI and the kernels that the full-width workloads
# never launch (the merge, and the short-sequence forward and backward).
_HOST_OR_UNTIMED = {"api.hip", "merge.hip", "fwd_short.hip", "bwd_short.hip"}


def kernel_sources_sha256() -> str:
    h = hashlib.sha256()
    for p in sorted((ROOT / "paper_2609_34420_amd" / "csrc").glob("*.[hc]*")):
        if p.name in _HOST_OR_UNTIMED:
            continue
        h.update(p.name.encode())
        h.update(p.read_bytes())
    return h.hexdigest()


# ---------------------------------------------------------------------------
# workloads
# ---------------------------------------------------------------------------
def run_layer(w, args, dev):
    """One layer over all N nodes: forward, then the three backward stages."""
    import torch

    import paper_2609_34420_amd as gt

    t0 = time.time()
    spd = upload_spd(w, args.seed, dev)
    log(f"spd {w.N}x{w.N} generated and uploaded in {time.time() - t0:.1f}s")
    x = device_tensors(w, args.seed, dev)
    log(f"inputs ready in {time.time() - t0:.1f}s")
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
    spd_t = spd if w.spd_symmetric else None
    names = ("bwd_prep", "bwd_dkdv", "bwd_dq") if w.dtype == "bf16" else ("bwd_prep", "bwd_dkdv_valu",
                                                                         "bwd_dq_valu")
    fname = "fwd" if w.dtype == "bf16" else "fwd_valu"

    def step(t):
        if t: t.mark(fname)
        gt.gt_attn_fwd(x["q"], x["k"], x["v"], spd, x["table"], scale=scale, out=O, lse=L)
        for ph in range(3):
            if t: t.mark(names[ph])
            gt.gt_attn_bwd_phase(ph, x["q"], x["k"], x["v"], spd, x["table"], O, L, x["do"],
                                 scale=scale, workspace=ws, grads=grads, spd_t=spd_t)

    extra = {}
    if args.hbm_probe:
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
        extra["hbm_probe"] = {"what": "torch.sum over the spd matrix read as int64 words (read-only pass)",
                              "bytes": spd.numel(), "ms": ms, "GB_per_s": spd.numel() / (ms * 1e-3) / 1e9}
        log(f"HBM probe: {spd.numel() / 1e9:.2f} GB read in {ms:.3f} ms")
    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("copy calibration: 1 GiB device-to-device copy done")

    steps, per_launch, launches, wall = timed_steps(step, args, stream)
    runs = []
    for _ in range(3):
        gt.gt_attn_bwd(x["q"], x["k"], x["v"], spd, x["table"], O, L, x["do"], scale=scale,
                       workspace=ws, grads=grads, spd_t=spd_t)
        runs.append(grads[3].clone())
    torch.cuda.synchronize()
    extra["dtable_spread"] = dtable_spread(runs)
    N2dH = float(N) * N * d * H
    flops = {fname: 4.0 * N2dH, names[1]: 8.0 * N2dH, names[2]: 2.0 * N2dH}
    rules = {fname: "forward kernel: Q K^T and P V products (4 N^2 d H)",
             names[1]: "dK/dV/dtable kernel: S recompute, dP, dV, dK products (8 N^2 d H)",
             names[2]: "dQ kernel: the dQ product (2 N^2 d H credited; its S and dP recomputation "
                       "is not)"}
    return dict(steps=steps, per_launch=per_launch, launches=launches, wall=wall, flops=flops,
                rules=rules, flop_per_step=w.flops_fwd_bwd, extra=extra)


def run_cp(w, args, dev):
    """One device's share of the context-parallel ring (Section III-A-1):
    query shard `w.shard` of `w.shards` with only its spd rows; the 8 KV
    blocks are resident as separate buffers (as they arrive in the ring).
    The step is the forward ring (the first block with gt_attn_ring_step,
    the others merged in place with gt_attn_ring_step_acc); the backward
    ring (gt_attn_bwd_ring_step over the same blocks with the merged O, LSE)
    is timed after it."""
    import torch

    import paper_2609_34420_amd as gt
    from paper_2609_34420_amd import ring

    P, S, rank = w.shards, w.S, w.shard
    r0 = rank * S
    t0 = time.time()
    spd = upload_spd(w, args.seed, dev, rows=(r0, r0 + S))
    log(f"spd shard [{S}, {w.N}] generated and uploaded in {time.time() - t0:.1f}s")
    x = device_tensors(w, args.seed, dev)
    Qs = x["q"][:, r0:r0 + S].contiguous()
    dOs = x["do"][:, r0:r0 + S].contiguous()
    T = x["table"]
    bounds = [b * S for b in range(P + 1)]
    steps_kv = ring.ring_steps(bounds, rank)
    blocks = [(c0, x["k"][:, c0:c1].contiguous(), x["v"][:, c0:c1].contiguous())
              for c0, c1 in steps_kv]
    del x
    torch.cuda.empty_cache()
    H, d = w.H, w.d
    scale = w.scale()
    o_acc = torch.empty((H, S, d), dtype=torch.float32, device=dev)
    l_acc = torch.empty((H, S), dtype=torch.float32, device=dev)
    stream = torch.cuda.current_stream()
    log(f"inputs ready in {time.time() - t0:.1f}s")

    def fwd_ring(t):
        for i, (c0, Kb, Vb) in enumerate(blocks):
            if t: t.mark("fwd_ring_step")
            if i == 0:
                gt.gt_attn_ring_step(Qs, Kb, Vb, spd, 0, c0, T, scale=scale, out=o_acc, lse=l_acc)
            else:
                gt.gt_attn_ring_step_acc(Qs, Kb, Vb, spd, 0, c0, T, (o_acc, l_acc), scale=scale)

    steps, per_launch, launches, wall = timed_steps(fwd_ring, args, stream)
    # backward ring over the same blocks, with the merged output
    O, L = gt.gt_attn_merge(o_acc[None], l_acc[None], dtype=torch.bfloat16)
    dq = torch.zeros((H, S, d), dtype=torch.float32, device=dev)
    dtab = torch.zeros_like(T)
    dkv = [(torch.zeros((H, S, d), dtype=torch.float32, device=dev),
            torch.zeros((H, S, d), dtype=torch.float32, device=dev)) for _ in blocks]
    ws = torch.empty(gt.gt_attn_bwd_ring_workspace_size(H, S, S, d, torch.bfloat16),
                     dtype=torch.uint8, device=dev)

    def bwd_ring(t):
        for (c0, Kb, Vb), (dk_b, dv_b) in zip(blocks, dkv):
            if t: t.mark("bwd_ring_step")
            gt.gt_attn_bwd_ring_step(Qs, O, L, dOs, Kb, Vb, spd, 0, c0, T, scale=scale,
                                     acc=(dq, dk_b, dv_b, dtab), workspace=ws)

    class _A:
        pass
    a2 = _A()
    a2.warmup, a2.steps = 1, max(2, args.steps // 2)
    bsteps, bper, blaunch, _ = timed_steps(bwd_ring, a2, stream)
    runs = []
    for _ in range(3):
        dtab.zero_()
        bwd_ring(None)
        runs.append(dtab.clone())
    torch.cuda.synchronize()
    SkN = float(S) * w.N * d * H
    bwd_ms = sum(bsteps) / len(bsteps)
    extra = {"bwd_ring": {"ms_per_ring": bwd_ms, "steps": a2.steps,
                          "value": 10.0 * SkN / (bwd_ms * 1e-3) / 1e12, "unit": "TFLOP/s",
                          "flop_rule": "10 Sq N d H (S recompute, dP, dV, dK, dQ) over the 8 steps",
                          "per_launch_ms": bper.get("bwd_ring_step")},
             "dtable_spread": dtable_spread(runs)}
    flops = {"fwd_ring_step": 4.0 * float(S) * S * d * H}
    rules = {"fwd_ring_step": "one ring step: Q_shard K_blk^T and P V_blk (4 Sq Sk d H)"}
    return dict(steps=steps, per_launch=per_launch, launches=launches, wall=wall, flops=flops,
                rules=rules, flop_per_step=4.0 * SkN, extra=extra)


def run_deep(w, args, dev):
    """12 layers sharing one spd, each with its own Q, K, V, dO and table:
    the forward of layers 1..12 (outputs kept), then the backward of layers
    12..1."""
    import torch

    import paper_2609_34420_amd as gt

    t0 = time.time()
    spd = upload_spd(w, args.seed, dev)
    log(f"spd {w.N}x{w.N} generated and uploaded in {time.time() - t0:.1f}s")
    layers = [device_tensors(w, args.seed, dev, layer=l) for l in range(w.layers)]
    log(f"{w.layers} layers of inputs ready in {time.time() - t0:.1f}s")
    H, N, d = w.H, w.N, w.d
    scale = w.scale()
    for x in layers:
        x["O"] = torch.empty_like(x["q"])
        x["L"] = torch.empty((H, N), dtype=torch.float32, device=dev)
        x["grads"] = (torch.empty_like(x["q"]), torch.empty_like(x["k"]), torch.empty_like(x["v"]),
                      torch.empty_like(x["table"]))
    ws = torch.empty(gt.gt_attn_bwd_workspace_size(H, N, d, torch.bfloat16), dtype=torch.uint8,
                     device=dev)
    stream = torch.cuda.current_stream()
    names = ("bwd_prep", "bwd_dkdv", "bwd_dq")

    def step(t):
        for x in layers:
            if t: t.mark("fwd")
            gt.gt_attn_fwd(x["q"], x["k"], x["v"], spd, x["table"], scale=scale, out=x["O"],
                           lse=x["L"])
        for x in reversed(layers):
            for ph in range(3):
                if t: t.mark(names[ph])
                gt.gt_attn_bwd_phase(ph, x["q"], x["k"], x["v"], spd, x["table"], x["O"], x["L"],
                                     x["do"], scale=scale, workspace=ws, grads=x["grads"])

    steps, per_launch, launches, wall = timed_steps(step, args, stream)
    x = layers[0]
    runs = []
    for _ in range(3):
        gt.gt_attn_bwd(x["q"], x["k"], x["v"], spd, x["table"], x["O"], x["L"], x["do"],
                       scale=scale, workspace=ws, grads=x["grads"])
        runs.append(x["grads"][3].clone())
    torch.cuda.synchronize()
    N2dH = float(N) * N * d * H
    flops = {"fwd": 4.0 * N2dH, "bwd_dkdv": 8.0 * N2dH, "bwd_dq": 2.0 * N2dH}
    rules = {"fwd": "forward kernel of one layer (4 N^2 d H)",
             "bwd_dkdv": "dK/dV/dtable kernel of one layer (8 N^2 d H)",
             "bwd_dq": "dQ kernel of one layer (2 N^2 d H credited)"}
    return dict(steps=steps, per_launch=per_launch, launches=launches, wall=wall, flops=flops,
                rules=rules, flop_per_step=w.flops_fwd_bwd,
                extra={"dtable_spread": dtable_spread(runs)})


# ---------------------------------------------------------------------------
# CPU baseline: the oracle on a bounded sample of the same workload
# ---------------------------------------------------------------------------
def cpu_baseline(w, args):
    import numpy as np

    import oracle

    host = host_record()
    scale = w.scale()
    if w.name == "tiny":
        q, k, v = w.qkv(args.seed)
        do, table = w.d_out(args.seed), w.table(args.seed)
        spd = w.spd_block(0, w.N, seed=args.seed)
        t0 = time.perf_counter()
        oracle.forward(q, k, v, spd, table, scale)
        oracle.backward(q, k, v, spd, table, scale, do)
        dt = time.perf_counter() - t0
        flop = w.flops_fwd_bwd
        what = f"the whole workload (N={w.N}, H={w.H}), forward and backward"
    elif w.name == "cp256k":
        r0 = w.shard * w.S
        R = args.cpu_rows // 2
        rows = w.sample_rows(R - 2, seed=args.seed, lo=r0, hi=r0 + w.S)
        q, k, v = w.qkv(args.seed)
        table = w.table(args.seed)
        spd_rows = w.spd_rows(rows, seed=args.seed)
        t0 = time.perf_counter()
        oracle.block_attention(q[:, rows], k, v, spd_rows, table, scale)
        dt = time.perf_counter() - t0
        flop = 4.0 * len(rows) * w.N * w.d * w.H
        what = (f"{len(rows)} seeded query rows of shard {w.shard} against all {w.N} keys, forward "
                f"(the ring's result over every block); credited 4*R*N*d*H FLOP")
    else:
        rows = w.sample_rows(args.cpu_rows - 2, seed=args.seed)
        q, k, v = w.qkv(args.seed)
        do, table = w.d_out(args.seed), w.table(args.seed)
        spd_rows = w.spd_rows(rows, seed=args.seed)
        qr, dor = q[:, rows], do[:, rows]
        t0 = time.perf_counter()
        oracle.block_attention(qr, k, v, spd_rows, table, scale)
        oracle.block_backward(qr, k, v, spd_rows, table, scale, dor)
        dt = time.perf_counter() - t0
        flop = 14.0 * len(rows) * w.N * w.d * w.H
        what = (f"{len(rows)} seeded query rows of N={w.N} against all keys"
                f"{' (layer 1)' if w.layers > 1 else ''}, forward and backward; credited "
                f"14*R*N*d*H FLOP")
    log(f"oracle sample: {what} in {dt:.1f}s on {host.get('blas_threads')} BLAS threads")
    return {"value": flop / dt / 1e12, "unit": "TFLOP/s", "cores": int(host.get("blas_threads") or 1),
            "kind": "oracle",
            "sample": (f"{what} in fp64 NumPy ({dt:.1f} s); elementwise NumPy is single-threaded, "
                       f"matrix products use {host.get('blas_threads')} BLAS threads"),
            "host": host}


# ---------------------------------------------------------------------------
# batches of short graphs
# ---------------------------------------------------------------------------
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

    def step(t):
        if t: t.mark("fwd")
        gt.gt_attn_fwd_batch(q, k, v, spd, table, scale=scale, out=O, lse=L)
        if t: t.mark("bwd")
        gt.gt_attn_bwd_batch(q, k, v, spd, table, O, L, do, scale=scale, workspace=ws, grads=grads)

    # A step here is well under a millisecond: the warmup runs for at least
    # 100 ms (and W steps), so that the timed steps see the clocks of a
    # sustained load, and every event recorded in the stream leaves a gap of a
    # few microseconds before the next launch, so the K timed steps run back
    # to back between one pair of events; the per-kernel times come from K
    # more steps with an event around each launch.
    t_w, n_w = time.perf_counter(), 0
    while n_w < args.warmup or time.perf_counter() - t_w < 0.1:
        step(None)
        torch.cuda.synchronize()
        n_w += 1
    log(f"warmup: {n_w} steps")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(args.steps):
        step(None)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    log(f"timed {args.steps} steps back to back: {ms:.4f} ms per step (events)")
    steps, per_launch, _, _ = timed_steps(step, argparse.Namespace(steps=args.steps, warmup=0), stream)
    elems = float(B) * H * N * N
    flop = 14.0 * elems * d
    print(json.dumps({
        "metric": f"batched biased-attention fwd+bwd at B={B}, N={N}, H={H}, d={d}",
        "value": flop / (ms * 1e-3) / 1e12, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "dtype": "bf16",
        "data": "synthetic", "score_elements_per_ns": elems / (ms * 1e6),
        "kernel_ms": per_launch, "ms_per_step_with_kernel_events": sum(steps) / len(steps),
        "config": {"workload": f"batch of {B} graphs of {N} nodes, i.i.d. uniform spd over {nb} "
                               f"buckets, H={H}, d={d}, bf16", "parallelism": "single GPU"},
    }), flush=True)


def graph_label(w) -> str:
    if w.spd_law is not None:
        return f"i.i.d. Zipf(s={w.spd_law[1]}) spd over {w.n_buckets} buckets"
    kind = w.graph[0]
    if kind == "sbm":
        return f"clustered planted-partition graph, {w.graph[1]} communities"
    if kind == "ba":
        return f"Barabasi-Albert graph, m={w.graph[1]}"
    return f"Erdos-Renyi graph, average degree {w.graph[1]}"


def metric_of(w) -> str:
    if w.name == "cp256k":
        return (f"context-parallel forward ring TFLOP/s and % bf16 MFMA peak, one device's share: "
                f"query shard {w.shard} of {w.shards} (Sq={w.S}) against N={w.N} keys, H={w.H}, "
                f"d={w.d}")
    if w.layers > 1:
        return (f"{w.layers}-layer biased-attention fwd+bwd TFLOP/s and % bf16 MFMA peak at N={w.N}, "
                f"H={w.H}, d={w.d}")
    prec = "bf16 MFMA" if w.dtype == "bf16" else "fp32 vector"
    return f"biased-attention fwd+bwd TFLOP/s and % {prec} peak at N={w.N}, H={w.H}, d={w.d}"


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
    if w.name == "cp256k":
        r = run_cp(w, args, dev)
    elif w.layers > 1:
        r = run_deep(w, args, dev)
    else:
        r = run_layer(w, args, dev)
    K = args.steps
    ms = sum(r["steps"]) / len(r["steps"])
    tflops = r["flop_per_step"] / (ms * 1e-3) / 1e12
    peak = PEAK_BF16 if w.dtype == "bf16" else PEAK_F32_VALU

    # dominant kernel: the largest share of the step
    share = {n: r["per_launch"][n] * r["launches"][n] for n in r["per_launch"] if n in r["flops"]}
    dom = max(share, key=share.get)
    achieved = r["flops"][dom] / (r["per_launch"][dom] * 1e-3)
    roofline = {"bound": "mfma" if w.dtype == "bf16" else "alu", "achieved": achieved / 1e12,
                "peak": peak / 1e12, "unit": "TFLOP/s", "frac": achieved / peak,
                "traffic": measured_traffic(w.name, dom), "kernel": dom,
                "kernel_ms": r["per_launch"][dom], "launches_per_step": r["launches"][dom],
                "flop_per_launch": r["flops"][dom], "flop_rule": r["rules"][dom]}

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, args)

    out = {
        "metric": metric_of(w),
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
        "pct_of_peak": 100.0 * tflops * 1e12 / peak,
        "config": {"workload": f"{w.name}: {graph_label(w)}, N={w.N}, H={w.H}, d={w.d}, "
                               f"{w.n_buckets} spd buckets, {w.dtype}"
                               + (f", {w.layers} layers" if w.layers > 1 else "")
                               + (f", query shard {w.shard} of {w.shards}" if w.shards > 1 else ""),
                   "N": w.N, "H": w.H, "d": w.d, "n_buckets": w.n_buckets, "layers": w.layers,
                   "flop_per_step": r["flop_per_step"], "parallelism": "single GPU"},
        "kernel_ms": r["per_launch"],
        "launches_per_step": r["launches"],
        "step_ms_stats": {"mean": ms, "median": statistics.median(r["steps"]),
                          "min": min(r["steps"]), "max": max(r["steps"])},
        "wall_ms_per_step": r["wall"],
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if w.dtype == "bf16":
        out["pct_of_bf16_peak"] = out["pct_of_peak"]
    out.update(r["extra"])
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
