"""GPU parity at sizes the oracle computes in full: the HIP path (through the
C ABI) against the fp64 oracle, element by element, on the same seeded
inputs. Sizes span several tiles and ragged tails; edge cases cover N = 1,
empty KV blocks, fully masked rows, out-of-range buckets, asymmetric spd,
unaligned spd slices and row/column offsets."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34420_amd as gt
import synth
from gpu_common import (DEV, TOL, check_fwd, check_grads, max_abs, rel_l2, say, tdtype,
                        to_dev, to_np)

pytestmark = pytest.mark.gpu


def _case(H, N, d, nb, seed, dt, hi=None, table_std=0.5, qkv_std=None, neg_inf=False):
    g = np.random.default_rng(seed)
    qkv_std = (1.0 / math.sqrt(d)) if qkv_std is None else qkv_std
    q, k, v = (g.standard_normal((H, N, d)).astype(np.float32) * np.float32(qkv_std) for _ in range(3))
    do = g.standard_normal((H, N, d)).astype(np.float32)
    if dt == "bf16":
        q, k, v, do = (synth.round_bf16(x) for x in (q, k, v, do))
    table = (g.standard_normal((H, nb)) * table_std).astype(np.float32)
    if neg_inf:
        table[:, : max(1, nb // 3)] = -np.inf
    spd = g.integers(0, hi if hi is not None else nb, size=(N, N)).astype(np.uint8)
    return q, k, v, do, table, spd


def _run_full(q, k, v, do, table, spd, dt, scale, spd_t=None):
    td = tdtype(dt)
    Q, K, V, dO = (to_dev(x, td) for x in (q, k, v, do))
    T = to_dev(table)
    S = to_dev(spd, torch.uint8)
    St = None if spd_t is None else (S if spd_t is spd else to_dev(spd_t, torch.uint8))
    O, L = gt.gt_attn_fwd(Q, K, V, S, T, scale=scale)
    dq, dk, dv, dtab = gt.gt_attn_bwd(Q, K, V, S, T, O, L, dO, scale=scale, spd_t=St)
    torch.cuda.synchronize()
    return dict(o=to_np(O), lse=to_np(L), dq=to_np(dq), dk=to_np(dk), dv=to_np(dv),
                dtable=to_np(dtab))


def _oracle_full(q, k, v, do, table, spd, scale):
    O, L = oracle.forward(q, k, v, spd, table, scale)
    dq, dk, dv, dt = oracle.backward(q, k, v, spd, table, scale, do)
    return dict(o=O, lse=L, dq=dq, dk=dk, dv=dv, dtable=dt)


def test_tiny_workload_fp32():
    """N=512, H=4, d=32 fp32, Erdos-Renyi spd clipped at 20: full oracle."""
    w = synth.workload("tiny")
    q, k, v = w.qkv(0)
    do = w.d_out(0)
    table = w.table(0)
    spd = w.spd_block(0, w.N)
    say("tiny fp32 N=512 H=4 d=32")
    got = _run_full(q, k, v, do, table, spd, "f32", w.scale())
    ref = _oracle_full(q, k, v, do, table, spd, w.scale())
    check_fwd("tiny", got["o"], got["lse"], ref["o"], ref["lse"], "f32")
    check_grads("tiny", got, ref, "f32")


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("d", [8, 16, 32, 64])
@pytest.mark.parametrize("N", [1, 7, 33, 100, 1000])
def test_ragged_sizes(N, d, dt):
    """Ragged N (not a tile multiple), asymmetric random spd with buckets past
    the table (bias 0, no gradient)."""
    H, nb = 2, 10
    q, k, v, do, table, spd = _case(H, N, d, nb, seed=N * 7 + d, dt=dt, hi=nb + 4)
    scale = 1.0 / math.sqrt(d)
    say(f"ragged {dt} N={N} d={d}")
    got = _run_full(q, k, v, do, table, spd, dt, scale)
    ref = _oracle_full(q, k, v, do, table, spd, scale)
    check_fwd(f"ragged N={N}", got["o"], got["lse"], ref["o"], ref["lse"], dt)
    if N > 1:
        check_grads(f"ragged N={N}", got, ref, dt)
    else:
        # N = 1: dV = dO and dQ = dK = dtable = 0 (P = 1, so dS = dP - Dlt = 0
        # up to the rounding of O and LSE)
        assert max_abs(got["dv"], do) <= TOL[dt]["o"]
        for name in ("dq", "dk", "dtable"):
            assert np.abs(got[name]).max() <= 1e-6, name


@pytest.mark.parametrize("d,N", [(8, 600), (32, 600), (64, 600), (8, 256), (16, 256), (8, 200), (32, 200)])
def test_large_and_rising_scores(d, N):
    """Score ranges far past the forward's block-sum limit, bf16. Head 0:
    large Q, K and table entries (scores spread over tens of units, so the
    softmax is nearly one-hot). Head 1: every query's scores rise along the
    keys (q_i . k_j grows with j, up to about 170), so each new key block
    moves the row max and the exact rescaling path runs on every block.
    N = 256 and 200 run the short-sequence kernels (whole-sequence forward,
    fused backward), N = 600 the full-width ones.
    (The fp32 bars are absolute and sized for scores of order one.) The
    backward is checked as a function of its inputs, to the relative bar
    except head 1's dQ on the matrix cores (see below)."""
    dt = "bf16"
    H, nb = 2, 12
    q, k, v, do, table, spd = _case(H, N, d, nb, seed=40 + d + (N % 600), dt=dt, table_std=4.0, qkv_std=1.5)
    g = np.random.default_rng(41 + d + (N % 600))
    u = np.abs(g.standard_normal(d)) + 0.1
    u /= np.linalg.norm(u)
    span = 40.0 * math.sqrt(d)                     # scores up to span * scale * max|q|
    q[1] = u[None, :] * (1.0 + np.abs(g.standard_normal((N, 1))))
    k[1] = u[None, :] * (span * np.arange(N) / N)[:, None]
    table[1] *= 0.05
    v *= 0.25                                      # exact in bf16
    q, k = synth.round_bf16(q.astype(np.float32)), synth.round_bf16(k.astype(np.float32))
    scale = 1.0 / math.sqrt(d)
    say(f"large scores {dt} d={d} N={N}")
    td = tdtype(dt)
    Q, K, V, dO = (to_dev(x, td) for x in (q, k, v, do))
    T, S = to_dev(table), to_dev(spd, torch.uint8)
    O, L = gt.gt_attn_fwd(Q, K, V, S, T, scale=scale)
    torch.cuda.synchronize()
    o_r, l_r = oracle.forward(q, k, v, spd, table, scale)
    assert np.isfinite(to_np(O)).all() and np.isfinite(to_np(L)).all()
    check_fwd(f"large d={d}", to_np(O), to_np(L), o_r, l_r, dt)
    # Backward as a function of its inputs: with a nearly one-hot softmax
    # dS = P (dP - Dlt) nearly cancels, so both sides take the oracle's O
    # rounded to bf16 (Dlt comes from it) and its LSE.
    o_in = synth.round_bf16(o_r.astype(np.float32))
    l_in = l_r.astype(np.float32)
    gq, gk, gv, gtab = oracle.ring_backward_step(q, o_in, l_in, do, k, v, spd, 0, 0, table, scale)
    dq, dk, dv, dtab = gt.gt_attn_bwd(Q, K, V, S, T, to_dev(o_in, td), to_dev(l_in), dO, scale=scale)
    torch.cuda.synchronize()
    dq = to_np(dq)
    check_grads(f"large d={d}", dict(dq=dq[:1], dk=to_np(dk), dv=to_np(dv), dtable=to_np(dtab)),
                dict(dq=gq[:1], dk=gk, dv=gv, dtable=gtab), dt)
    # Head 1's dQ_i = scale sum_j dS_ij k_j sums nearly cancelling terms
    # (parallel keys with norms up to ~230, sum_j dS_ij ~ 0). On the
    # matrix cores dS is rounded to bf16 (relative 2^-9) before that
    # product, which moves dQ by up to scale 2^-9 sum_j |dS_ij| |k_jc|;
    # check it against twice that bound instead of the relative bar.
    q1, k1, v1, do1 = (x[1].astype(np.float64) for x in (q, k, v, do))
    bias = np.where(spd < nb, table[1][np.minimum(spd, nb - 1)], 0.0)
    p1 = np.exp(scale * q1 @ k1.T + bias - l_in[1][:, None].astype(np.float64))
    ds1 = p1 * (do1 @ v1.T - (do1 * o_in[1]).sum(1)[:, None])
    bound = 2.0 * scale * 2.0 ** -9 * (np.abs(ds1) @ np.abs(k1)) + 1e-4
    err = np.abs(dq[1] - gq[1])
    say(f"large d={d}: head-1 dq max err / bound {(err / bound).max():.3f}")
    assert (err <= bound).all()


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_masked_rows_and_neg_inf_table(dt):
    """-inf table entries; rows 0..9 only see -inf buckets: O = 0, LSE = -inf,
    zero gradients from those rows, no NaN anywhere."""
    H, N, d, nb = 2, 300, 64, 9
    q, k, v, do, table, spd = _case(H, N, d, nb, seed=5, dt=dt, neg_inf=True)
    spd[:10] = np.random.default_rng(6).integers(0, nb // 3, size=(10, N))
    scale = 0.125
    say(f"masked rows {dt}")
    got = _run_full(q, k, v, do, table, spd, dt, scale)
    ref = _oracle_full(q, k, v, do, table, spd, scale)
    assert np.isneginf(got["lse"][:, :10]).all() and np.all(got["o"][:, :10] == 0)
    check_fwd("masked", got["o"], got["lse"], ref["o"], ref["lse"], dt)
    check_grads("masked", got, ref, dt)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("Sq,Sk,row_off,col_off,ld,d", [
    (200, 300, 37, 91, 512, 64),      # unaligned slice: byte loads
    (256, 320, 64, 128, 512, 64),     # 16-byte aligned slice: vector loads
    (129, 1, 3, 500, 512, 64),        # single key
    (64, 77, 0, 0, 77, 64),           # ld not a multiple of 16
    (100, 150, 5, 40, 256, 8),        # small head dim (zero-padded 32-wide tiles for bf16)
    (70, 64, 0, 64, 128, 16),
])
def test_ring_step_offsets(Sq, Sk, row_off, col_off, ld, d, dt):
    """One context-parallel step: bias slice spd[row_off + i, col_off + j] of an
    asymmetric spd; partial O (fp32) and LSE against the oracle's ring step."""
    H, nb = 3, 12
    g = np.random.default_rng(Sq + Sk)
    rows = row_off + Sq
    spd = g.integers(0, nb + 2, size=(rows, ld)).astype(np.uint8)
    q = g.standard_normal((H, Sq, d)).astype(np.float32) * 0.125
    k = g.standard_normal((H, Sk, d)).astype(np.float32) * 0.125
    v = g.standard_normal((H, Sk, d)).astype(np.float32)
    if dt == "bf16":
        q, k, v = (synth.round_bf16(x) for x in (q, k, v))
    table = (g.standard_normal((H, nb)) * 0.5).astype(np.float32)
    td = tdtype(dt)
    say(f"ring step {dt} Sq={Sq} Sk={Sk} row_off={row_off} col_off={col_off} ld={ld} d={d}")
    o, l = gt.gt_attn_ring_step(to_dev(q, td), to_dev(k, td), to_dev(v, td),
                                to_dev(spd, torch.uint8), row_off, col_off, to_dev(table),
                                scale=0.125)
    torch.cuda.synchronize()
    o_ref, l_ref = oracle.ring_step(q, k, v, spd, row_off, col_off, table, 0.125)
    check_fwd("ring", to_np(o), to_np(l), o_ref, l_ref, dt)


def test_ring_step_empty_kv_block():
    """Sk = 0: the partial is O = 0, LSE = -inf (null K/V/spd allowed)."""
    q = torch.randn(2, 70, 32, device=DEV).to(torch.bfloat16)
    t = torch.randn(2, 5, device=DEV)
    o, l = gt.gt_attn_ring_step(q, None, None, None, 0, 0, t)
    torch.cuda.synchronize()
    assert torch.all(o == 0) and torch.all(torch.isneginf(l))


@pytest.mark.parametrize("out", ["bf16", "f32"])
@pytest.mark.parametrize("P", [1, 3, 8])
def test_merge(P, out):
    """Merge of partials against the oracle, with some -inf parts and a row
    whose every part is -inf."""
    H, S, d = 3, 333, 64
    g = np.random.default_rng(P)
    o = g.standard_normal((P, H, S, d)).astype(np.float32)
    lse = (g.standard_normal((P, H, S)) * 3).astype(np.float32)
    lse[0, :, ::7] = -np.inf
    lse[:, 0, 5] = -np.inf
    say(f"merge P={P} out={out}")
    O, L = gt.gt_attn_merge(to_dev(o), to_dev(lse), dtype=tdtype(out))
    torch.cuda.synchronize()
    O_ref, L_ref = oracle.merge(o, lse)
    tol = TOL["bf16" if out == "bf16" else "f32"]["o"]
    assert max_abs(to_np(O), O_ref) <= tol
    assert max_abs(to_np(L), L_ref) <= 1e-5
    assert np.isneginf(to_np(L)[0, 5]) and np.all(to_np(O)[0, 5] == 0)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_context_parallel_ring_small(dt):
    """P = 4 uneven shards of N = 1000: every rank runs its ring steps on its
    own spd row shard (row_off = 0, col_off = the block's first node), then
    merges; the result equals the unsharded oracle forward."""
    H, N, d, nb = 2, 1000, 64, 16
    q, k, v, do, table, spd = _case(H, N, d, nb, seed=11, dt=dt)
    bounds = [0, 240, 500, 777, 1000]
    td = tdtype(dt)
    Q, K, V, T = to_dev(q, td), to_dev(k, td), to_dev(v, td), to_dev(table)
    O_ref, L_ref = oracle.forward(q, k, v, spd, table, 0.125)
    P = len(bounds) - 1
    for r in range(P):
        r0, r1 = bounds[r], bounds[r + 1]
        shard = to_dev(spd[r0:r1], torch.uint8)
        parts_o, parts_l = [], []
        for t in range(P):
            b = (r - t) % P
            c0, c1 = bounds[b], bounds[b + 1]
            o_p, l_p = gt.gt_attn_ring_step(Q[:, r0:r1].contiguous(), K[:, c0:c1].contiguous(),
                                            V[:, c0:c1].contiguous(), shard, 0, c0, T, scale=0.125)
            parts_o.append(o_p)
            parts_l.append(l_p)
        O, L = gt.gt_attn_merge(torch.stack(parts_o), torch.stack(parts_l), dtype=td)
        torch.cuda.synchronize()
        say(f"cp small {dt} rank {r}")
        check_fwd(f"cp rank {r}", to_np(O), to_np(L), O_ref[:, r0:r1], L_ref[:, r0:r1], dt)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_context_parallel_ring_accumulate(dt):
    """The same ring with the in-place running merge: the first step's
    partial starts the state, every later step is merged into it by the
    kernel. Equals the unsharded oracle forward and, within fp32 rounding,
    the merge of the separate partials. Rows 0..5 only see -inf buckets in
    block 0 and nowhere else; rows 6..8 see -inf buckets everywhere."""
    H, N, d, nb = 2, 1000, 64, 16
    q, k, v, do, table, spd = _case(H, N, d, nb, seed=13, dt=dt)
    table[:, :4] = -np.inf
    bounds = [0, 240, 500, 777, 1000]
    spd[:6, bounds[0]:bounds[1]] = 1
    spd[6:9] = 2
    td = tdtype(dt)
    Q, K, V, T = to_dev(q, td), to_dev(k, td), to_dev(v, td), to_dev(table)
    O_ref, L_ref = oracle.forward(q, k, v, spd, table, 0.125)
    P = len(bounds) - 1
    for r in range(P):
        r0, r1 = bounds[r], bounds[r + 1]
        shard = to_dev(spd[r0:r1], torch.uint8)
        Qr = Q[:, r0:r1].contiguous()
        parts_o, parts_l, state = [], [], None
        for t in range(P):
            b = (r - t) % P
            c0, c1 = bounds[b], bounds[b + 1]
            Kb, Vb = K[:, c0:c1].contiguous(), V[:, c0:c1].contiguous()
            o_p, l_p = gt.gt_attn_ring_step(Qr, Kb, Vb, shard, 0, c0, T, scale=0.125)
            parts_o.append(o_p)
            parts_l.append(l_p)
            if state is None:
                state = (o_p.clone(), l_p.clone())
            else:
                gt.gt_attn_ring_step_acc(Qr, Kb, Vb, shard, 0, c0, T, state, scale=0.125)
        O_m, L_m = gt.gt_attn_merge(torch.stack(parts_o), torch.stack(parts_l), dtype=torch.float32)
        torch.cuda.synchronize()
        say(f"cp accumulate {dt} rank {r}")
        o_acc, l_acc = to_np(state[0]), to_np(state[1])
        assert np.isfinite(o_acc).all()
        check_fwd(f"cp acc rank {r}", o_acc, l_acc, O_ref[:, r0:r1], L_ref[:, r0:r1], dt)
        assert max_abs(o_acc, to_np(O_m)) <= 1e-5 and max_abs(l_acc, to_np(L_m)) <= 1e-5
        if r == 0:
            assert np.isneginf(l_acc[:, 6:9]).all() and np.all(o_acc[:, 6:9] == 0)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_ring_step_acc_from_empty_state_and_empty_block(dt):
    """A state at O = 0, LSE = -inf plus one step equals that step's partial;
    a step with no keys (Sk = 0) leaves the state bit for bit unchanged."""
    H, Sq, Sk, d, nb = 3, 200, 150, 32, 8
    g = np.random.default_rng(3)
    q = g.standard_normal((H, Sq, d)).astype(np.float32) * 0.2
    k = g.standard_normal((H, Sk, d)).astype(np.float32) * 0.2
    v = g.standard_normal((H, Sk, d)).astype(np.float32)
    spd = g.integers(0, nb, size=(Sq, Sk)).astype(np.uint8)
    table = (g.standard_normal((H, nb)) * 0.5).astype(np.float32)
    td = tdtype(dt)
    Q, K, V, S, T = to_dev(q, td), to_dev(k, td), to_dev(v, td), to_dev(spd, torch.uint8), to_dev(table)
    say(f"ring acc empty state {dt}")
    o_p, l_p = gt.gt_attn_ring_step(Q, K, V, S, 0, 0, T, scale=0.2)
    state = (torch.zeros((H, Sq, d), device=DEV), torch.full((H, Sq), -math.inf, device=DEV))
    gt.gt_attn_ring_step_acc(Q, K, V, S, 0, 0, T, state, scale=0.2)
    torch.cuda.synchronize()
    assert max_abs(to_np(state[0]), to_np(o_p)) <= 1e-6
    assert max_abs(to_np(state[1]), to_np(l_p)) <= 1e-6
    before = (state[0].clone(), state[1].clone())
    gt.gt_attn_ring_step_acc(Q, None, None, None, 0, 0, T, state, scale=0.2)
    torch.cuda.synchronize()
    assert torch.equal(state[0], before[0]) and torch.equal(state[1], before[1])


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("B,N,d,spd_kind", [
    (4, 200, 64, "per_graph"),      # ragged tiles, unaligned spd rows
    (3, 256, 32, "per_graph_t"),    # aligned, with per-graph transposes
    (5, 96, 64, "shared"),          # one spd for every graph (stride 0)
    (16, 65, 8, "per_graph"),       # the paper's head dim: 8 heads over 64 features
    (6, 128, 16, "per_graph_t"),
    (8, 192, 8, "shared"),          # two graphs per forward workgroup, 192 of its 256 rows used
])
def test_batch_of_graphs(B, N, d, spd_kind, dt):
    """A batch of graphs, each with its own spd, sharing the table: every
    graph's O, LSE, dQ, dK, dV equal the oracle on that graph alone, and
    dtable equals the sum of the graphs' oracle dtables."""
    H, nb = 3, 12
    g = np.random.default_rng(B * N + d)
    shape = (B, H, N, d)
    q, k, v = (g.standard_normal(shape).astype(np.float32) / np.float32(math.sqrt(d)) for _ in range(3))
    do = g.standard_normal(shape).astype(np.float32)
    if dt == "bf16":
        q, k, v, do = (synth.round_bf16(x) for x in (q, k, v, do))
    table = (g.standard_normal((H, nb)) * 0.5).astype(np.float32)
    if spd_kind == "shared":
        spd = g.integers(0, nb + 2, size=(N, N)).astype(np.uint8)
        spd_b = [spd] * B
    else:
        spd = g.integers(0, nb + 2, size=(B, N, N)).astype(np.uint8)
        spd_b = list(spd)
    td = tdtype(dt)
    Q, K, V, dO = (to_dev(x, td) for x in (q, k, v, do))
    T = to_dev(table)
    S = to_dev(spd, torch.uint8)
    St = to_dev(np.ascontiguousarray(np.swapaxes(spd, -1, -2)), torch.uint8) if spd_kind == "per_graph_t" else None
    scale = 1.0 / math.sqrt(d)
    say(f"batch {dt} B={B} N={N} d={d} {spd_kind}")
    O, L = gt.gt_attn_fwd_batch(Q, K, V, S, T, scale=scale)
    dq, dk, dv, dtab = gt.gt_attn_bwd_batch(Q, K, V, S, T, O, L, dO, scale=scale, spd_t=St)
    torch.cuda.synchronize()
    dt_ref = np.zeros((H, nb))
    for b in range(B):
        ref = _oracle_full(q[b], k[b], v[b], do[b], table, spd_b[b], scale)
        got = dict(o=to_np(O[b]), lse=to_np(L[b]), dq=to_np(dq[b]), dk=to_np(dk[b]),
                   dv=to_np(dv[b]))
        check_fwd(f"batch graph {b}", got["o"], got["lse"], ref["o"], ref["lse"], dt)
        check_grads(f"batch graph {b}", got, ref, dt)
        dt_ref += ref["dtable"]
    assert rel_l2(to_np(dtab), dt_ref) <= TOL[dt]["grad"]


@pytest.mark.parametrize("B,hpb,N,d,spd_kind", [
    (12, 64, 80, 8, "per_graph"),       # 4 workgroup slots: 3 sequences per workgroup
    (12, 64, 256, 32, "per_graph_t"),
    (64, 8, 33, 16, "shared"),          # 32 slots: 2 sequences per workgroup
    (21, 64, 128, 8, "per_graph"),      # forward: pairs of sequences, 11 pairs on 8 slots
    (19, 128, 50, 16, "shared"),        # forward: 4 sequences at once, last group of 3
    (9, 128, 64, 32, "per_graph_t"),    # forward: 4 at once at d = 32, 3 groups on 2 slots
    (7, 64, 100, 16, "per_graph"),      # forward: pairs with a partial last key block
    (40, 8, 32, 8, "per_graph"),        # forward: 8 sequences at once (backward: 4)
    (37, 16, 20, 16, "per_graph_t"),    # N <= 32 with a partial block, last group of 5
    (64, 8, 12, 32, "shared"),
    (10, 64, 96, 16, "per_graph_t"),    # d = 16, N a multiple of 32: statistics in the products
    (12, 32, 64, 16, "per_graph"),
])
def test_batch_several_graphs_per_workgroup(B, hpb, N, d, spd_kind):
    """Sequences of at most 256 nodes with more sequences than the fused
    backward has workgroup slots, so each workgroup takes several sequences
    of one head in turn (the forward takes 2 or 4 sequences at once at
    N <= 128 or 64, and several such groups in turn). V and dO double every
    third of the batch, so a workgroup's later sequences have larger
    gradient bounds: the fixed-point exponent of its histogram drops and
    the sums accumulated so far are rescaled. Every graph's O, LSE, dQ, dK,
    dV and the summed dtable equal the oracle."""
    nb = 12
    g = np.random.default_rng(B * N + d + hpb)
    shape = (B, hpb, N, d)
    q, k, v = (g.standard_normal(shape).astype(np.float32) / np.float32(math.sqrt(d)) for _ in range(3))
    do = g.standard_normal(shape).astype(np.float32)
    grow = np.float32(2.0) ** ((np.arange(B) * 3) // B).astype(np.float32)
    v *= grow[:, None, None, None]
    do *= grow[:, None, None, None]
    q, k, v, do = (synth.round_bf16(x) for x in (q, k, v, do))
    table = (g.standard_normal((hpb, nb)) * 0.5).astype(np.float32)
    if spd_kind == "shared":
        spd = g.integers(0, nb + 2, size=(N, N)).astype(np.uint8)
        spd_b = [spd] * B
    else:
        spd = g.integers(0, nb + 2, size=(B, N, N)).astype(np.uint8)
        spd_b = list(spd)
    Q, K, V, dO = (to_dev(x, torch.bfloat16) for x in (q, k, v, do))
    T = to_dev(table)
    S = to_dev(spd, torch.uint8)
    St = to_dev(np.ascontiguousarray(np.swapaxes(spd, -1, -2)), torch.uint8) if spd_kind == "per_graph_t" else None
    scale = 1.0 / math.sqrt(d)
    say(f"batch bf16 B={B} hpb={hpb} N={N} d={d} {spd_kind} (several graphs per workgroup)")
    O, L = gt.gt_attn_fwd_batch(Q, K, V, S, T, scale=scale)
    dq, dk, dv, dtab = gt.gt_attn_bwd_batch(Q, K, V, S, T, O, L, dO, scale=scale, spd_t=St)
    torch.cuda.synchronize()
    dt_ref = np.zeros((hpb, nb))
    for b in range(B):
        ref = _oracle_full(q[b], k[b], v[b], do[b], table, spd_b[b], scale)
        got = dict(o=to_np(O[b]), lse=to_np(L[b]), dq=to_np(dq[b]), dk=to_np(dk[b]),
                   dv=to_np(dv[b]))
        check_fwd(f"batch graph {b}", got["o"], got["lse"], ref["o"], ref["lse"], "bf16")
        check_grads(f"batch graph {b}", got, ref, "bf16")
        dt_ref += ref["dtable"]
    err = rel_l2(to_np(dtab), dt_ref)
    say(f"dtable rel-L2 {err:.3e}")
    assert err <= TOL["bf16"]["grad"]


@pytest.mark.parametrize("spd_t_kind", ["none", "transposed"])
@pytest.mark.parametrize("nb,N,d", [(32, 200, 8), (127, 256, 32), (128, 200, 16), (200, 96, 8)])
def test_every_byte_value_short(nb, N, d, spd_t_kind):
    """spd bytes drawn from 0..255 on sequences of at most 256 nodes (the
    short-sequence kernels): bytes at or past n_buckets give bias 0 and no
    gradient, including bytes of 128 or more, which the short forward's
    128-entry table and the fused backward's 128-bucket layout map to a
    padding entry. N = 200 and 96 leave a partial last key block (the
    forward masks those keys through its -inf entry)."""
    H = 3
    q, k, v, do, table, spd = _case(H, N, d, nb, seed=nb * 5 + N + len(spd_t_kind), dt="bf16", hi=256)
    spd_t = np.ascontiguousarray(spd.T) if spd_t_kind == "transposed" else None
    scale = 1.0 / math.sqrt(d)
    tag = f"all bytes short nb={nb} N={N} d={d} spd_t={spd_t_kind}"
    say(tag)
    got = _run_full(q, k, v, do, table, spd, "bf16", scale, spd_t=spd_t)
    ref = _oracle_full(q, k, v, do, table, spd, scale)
    check_fwd(tag, got["o"], got["lse"], ref["o"], ref["lse"], "bf16")
    check_grads(tag, got, ref, "bf16")


def test_forward_is_deterministic():
    H, N, d, nb = 4, 777, 64, 20
    q, k, v, do, table, spd = _case(H, N, d, nb, seed=21, dt="bf16")
    Q, K, V = (to_dev(x, torch.bfloat16) for x in (q, k, v))
    S, T = to_dev(spd, torch.uint8), to_dev(table)
    O1, L1 = gt.gt_attn_fwd(Q, K, V, S, T)
    O2, L2 = gt.gt_attn_fwd(Q, K, V, S, T)
    torch.cuda.synchronize()
    assert torch.equal(O1, O2) and torch.equal(L1, L2)


def test_gradient_invariants_bf16():
    """sum_b dtable = 0, sum_j dK_j = 0, sum_j dV_j = sum_i dO_i (GPU, no oracle)."""
    H, N, d, nb = 2, 2048, 64, 32
    q, k, v, do, table, spd = _case(H, N, d, nb, seed=31, dt="bf16")
    got = _run_full(q, k, v, do, table, spd, "bf16", 0.125)
    scale_dt = np.abs(got["dtable"]).max()
    assert np.abs(got["dtable"].sum(1)).max() <= 1e-2 * scale_dt + 1e-4
    assert rel_l2(got["dk"].sum(1), np.zeros((H, d))) <= 1e-2 * np.linalg.norm(got["dk"])
    assert rel_l2(got["dv"].sum(1), do.sum(1)) <= 1e-2


@pytest.mark.parametrize("kind", ["symmetric", "transposed"])
@pytest.mark.parametrize("N", [64, 400, 1024])
def test_backward_with_spd_transpose(N, kind):
    """The key-stationary stage reading rows of spd_t: a symmetric matrix
    passed as its own transpose, and an asymmetric one with its transpose
    (N = 400 leaves a partial query tile; buckets past the table included)."""
    H, d, nb = 2, 64, 12
    q, k, v, do, table, spd = _case(H, N, d, nb, seed=N + (kind == "symmetric"), dt="bf16", hi=nb + 3)
    if kind == "symmetric":
        spd = np.minimum(spd, spd.T).copy()
        spd_t = spd
    else:
        spd_t = np.ascontiguousarray(spd.T)
    scale = 1.0 / math.sqrt(d)
    say(f"spd_t {kind} N={N}")
    got = _run_full(q, k, v, do, table, spd, "bf16", scale, spd_t=spd_t)
    ref = _oracle_full(q, k, v, do, table, spd, scale)
    check_fwd(f"spd_t {kind} N={N}", got["o"], got["lse"], ref["o"], ref["lse"], "bf16")
    check_grads(f"spd_t {kind} N={N}", got, ref, "bf16")


def test_spd_transpose_ignored_when_unaligned():
    """N = 100 is not a multiple of 16: spd_t is ignored (columns gathered),
    results still match the oracle."""
    H, N, d, nb = 2, 100, 64, 9
    q, k, v, do, table, spd = _case(H, N, d, nb, seed=5, dt="bf16")
    spd_t = np.ascontiguousarray(spd.T)
    scale = 1.0 / math.sqrt(d)
    got = _run_full(q, k, v, do, table, spd, "bf16", scale, spd_t=spd_t)
    ref = _oracle_full(q, k, v, do, table, spd, scale)
    check_grads("spd_t unaligned", got, ref, "bf16")


@pytest.mark.parametrize("spd_t_kind", ["none", "transposed"])
@pytest.mark.parametrize("nb", [32, 127, 128, 200])
def test_every_byte_value(nb, spd_t_kind):
    """spd bytes drawn from the whole range 0..255: bytes at or past
    n_buckets give bias 0 and no gradient. With at most 127 buckets the
    key-stationary stage maps bytes of 128 or more to its padding bucket;
    past that it uses the full 256-entry layout. N = 320 spans several
    query and key tiles with a partial last key block."""
    H, N, d = 2, 320, 64
    q, k, v, do, table, spd = _case(H, N, d, nb, seed=nb * 3 + len(spd_t_kind), dt="bf16", hi=256)
    spd_t = np.ascontiguousarray(spd.T) if spd_t_kind == "transposed" else None
    scale = 1.0 / math.sqrt(d)
    tag = f"all bytes nb={nb} spd_t={spd_t_kind}"
    say(tag)
    got = _run_full(q, k, v, do, table, spd, "bf16", scale, spd_t=spd_t)
    ref = _oracle_full(q, k, v, do, table, spd, scale)
    check_fwd(tag, got["o"], got["lse"], ref["o"], ref["lse"], "bf16")
    check_grads(tag, got, ref, "bf16")
