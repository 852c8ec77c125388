"""GPU parity over seeded random shapes: dtype, head dim, graph count, node
count, head count, bucket count (bytes past it included), -inf table entries
and the optional spd transpose drawn per case. The forward of every graph is
checked against the fp64 oracle; the backward against the oracle's backward
of the same inputs (the forward output in the input dtype, as the API passes
it), so a degenerate table (one bucket) does not measure the bf16 rounding
of O through Dlt instead of the kernels."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34420_amd as gt
import synth
from gpu_common import TOL, check_fwd, check_grads, rel_l2, say, tdtype, to_dev, to_np

pytestmark = pytest.mark.gpu


def _draw(seed):
    g = np.random.default_rng(1000 + seed)
    return dict(
        dt=str(g.choice(["bf16", "bf16", "f32"])),
        d=int(g.choice([8, 16, 32, 64, 64])),
        B=int(g.integers(1, 4)),
        N=int(g.choice([int(g.integers(1, 80)), int(g.integers(80, 420)), 16 * int(g.integers(1, 30))])),
        H=int(g.integers(1, 4)),
        nb=int(g.choice([1, int(g.integers(2, 40)), int(g.integers(100, 257))])),
        neg_inf=bool(g.random() < 0.3),
        use_t=bool(g.random() < 0.5),
        seed=seed,
    )


@pytest.mark.parametrize("seed", range(24))
def test_random_shape(seed):
    c = _draw(seed)
    dt, d, B, N, H, nb = c["dt"], c["d"], c["B"], c["N"], c["H"], c["nb"]
    g = np.random.default_rng(seed)
    shape = (B, H, N, d)
    q, k, v = (g.standard_normal(shape).astype(np.float32) / np.float32(math.sqrt(d)) for _ in range(3))
    do = g.standard_normal(shape).astype(np.float32)
    if dt == "bf16":
        q, k, v, do = (synth.round_bf16(x) for x in (q, k, v, do))
    table = (g.standard_normal((H, nb)) * 0.5).astype(np.float32)
    if c["neg_inf"] and nb > 2:
        table[:, 0] = -np.inf
    spd = g.integers(0, min(255, nb + 3) + 1, size=(B, N, N)).astype(np.uint8)
    spd_t = np.ascontiguousarray(np.swapaxes(spd, -1, -2)) if c["use_t"] else None
    td = tdtype(dt)
    Q, K, V, dO = (to_dev(x, td) for x in (q, k, v, do))
    T, S = to_dev(table), to_dev(spd, torch.uint8)
    St = None if spd_t is None else to_dev(spd_t, torch.uint8)
    scale = 1.0 / math.sqrt(d)
    say(f"random shape {c}")
    O, L = gt.gt_attn_fwd_batch(Q, K, V, S, T, scale=scale)
    torch.cuda.synchronize()
    # The backward is checked as a function of its inputs: both sides get the
    # oracle's forward output, rounded to the input dtype as the API hands it
    # over (Dlt = rowsum(dO * O) is taken from that O on both sides).
    o_in = np.zeros(shape, np.float32)
    l_in = np.zeros((B, H, N), np.float32)
    refs = []
    for b in range(B):
        o_r, l_r = oracle.forward(q[b], k[b], v[b], spd[b], table, scale)
        check_fwd(f"random {seed} graph {b}", to_np(O[b]), to_np(L[b]), o_r, l_r, dt)
        o_in[b] = synth.round_bf16(o_r.astype(np.float32)) if dt == "bf16" else o_r.astype(np.float32)
        l_in[b] = l_r.astype(np.float32)
        refs.append(oracle.ring_backward_step(q[b], o_in[b], l_in[b], do[b], k[b], v[b], spd[b], 0, 0,
                                              table, scale))
    dq, dk, dv, dtab = gt.gt_attn_bwd_batch(Q, K, V, S, T, to_dev(o_in, td), to_dev(l_in), dO,
                                            scale=scale, spd_t=St)
    torch.cuda.synchronize()
    dt_ref = np.zeros((H, nb))
    for b, (gq, gk, gv, gt_) in enumerate(refs):
        check_grads(f"random {seed} graph {b}",
                    dict(dq=to_np(dq[b]), dk=to_np(dk[b]), dv=to_np(dv[b])),
                    dict(dq=gq, dk=gk, dv=gv), dt)
        dt_ref += gt_
    got = to_np(dtab)
    assert np.isfinite(got).all()
    e = rel_l2(got, dt_ref)
    say(f"random {seed}: dtable rel-L2 {e:.3e}")
    assert e <= TOL[dt]["grad"] or np.abs(got - dt_ref).max() <= 1e-6


def _draw_packed(seed):
    g = np.random.default_rng(5000 + seed)
    return dict(
        d=int(g.choice([8, 16, 32])),
        B=int(g.integers(5, 40)),
        N=int(g.choice([4 * int(g.integers(1, 33)), int(g.integers(1, 129))])),
        hpb=int(g.choice([2, 16, 64, 128])),
        nb=int(g.choice([int(g.integers(2, 40)), int(g.integers(100, 128))])),
        neg_inf=bool(g.random() < 0.3),
        use_t=bool(g.random() < 0.5),
    )


@pytest.mark.parametrize("seed", range(12))
def test_random_packed_batch(seed):
    """Batches of short sequences (N <= 128, bf16, d <= 32) at random graph
    and head counts, so the short-sequence kernels pack 2, 4 or 8 sequences
    of a head to a workgroup, often with a partly filled last group and with
    several groups per workgroup (up to 128 heads per graph). Every graph's
    forward against the fp64 oracle; the backward as a function of its
    inputs, as in test_random_shape."""
    c = _draw_packed(seed)
    d, B, N, hpb, nb = c["d"], c["B"], c["N"], c["hpb"], c["nb"]
    g = np.random.default_rng(seed + 77)
    shape = (B, hpb, N, d)
    q, k, v = (synth.round_bf16(g.standard_normal(shape).astype(np.float32) / np.float32(math.sqrt(d)))
               for _ in range(3))
    do = synth.round_bf16(g.standard_normal(shape).astype(np.float32))
    table = (g.standard_normal((hpb, nb)) * 0.5).astype(np.float32)
    if c["neg_inf"]:
        table[:, 0] = -np.inf
    spd = g.integers(0, nb + 3, size=(B, N, N)).astype(np.uint8)
    St = to_dev(np.ascontiguousarray(np.swapaxes(spd, -1, -2)), torch.uint8) if c["use_t"] else None
    Q, K, V, dO = (to_dev(x, torch.bfloat16) for x in (q, k, v, do))
    T, S = to_dev(table), to_dev(spd, torch.uint8)
    scale = 1.0 / math.sqrt(d)
    say(f"random packed batch {c}")
    O, L = gt.gt_attn_fwd_batch(Q, K, V, S, T, scale=scale)
    torch.cuda.synchronize()
    o_in = np.zeros(shape, np.float32)
    l_in = np.zeros((B, hpb, N), np.float32)
    refs = []
    for b in range(B):
        o_r, l_r = oracle.forward(q[b], k[b], v[b], spd[b], table, scale)
        check_fwd(f"packed {seed} graph {b}", to_np(O[b]), to_np(L[b]), o_r, l_r, "bf16")
        o_in[b] = synth.round_bf16(o_r.astype(np.float32))
        l_in[b] = l_r.astype(np.float32)
        refs.append(oracle.ring_backward_step(q[b], o_in[b], l_in[b], do[b], k[b], v[b], spd[b], 0, 0,
                                              table, scale))
    dq, dk, dv, dtab = gt.gt_attn_bwd_batch(Q, K, V, S, T, to_dev(o_in, torch.bfloat16), to_dev(l_in), dO,
                                            scale=scale, spd_t=St)
    torch.cuda.synchronize()
    dt_ref = np.zeros((hpb, nb))
    for b, (gq, gk, gv, gt_) in enumerate(refs):
        check_grads(f"packed {seed} graph {b}",
                    dict(dq=to_np(dq[b]), dk=to_np(dk[b]), dv=to_np(dv[b])),
                    dict(dq=gq, dk=gk, dv=gv), "bf16")
        dt_ref += gt_
    got = to_np(dtab)
    assert np.isfinite(got).all()
    e = rel_l2(got, dt_ref)
    say(f"packed {seed}: dtable rel-L2 {e:.3e}")
    assert e <= TOL["bf16"]["grad"]
