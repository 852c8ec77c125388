"""GPU parity of the context-parallel backward (Section III-A-1 run in
reverse): one backward ring step through the C ABI against the oracle's
ring_backward_step, and whole simulated rings (forward steps, merge, backward
steps) against the unsharded oracle backward. The accumulators start from
nonzero values, so the tests also check that the step adds rather than
overwrites."""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34420_amd as gt
import synth
from paper_2609_34420_amd import ring
from gpu_common import DEV, TOL, check_fwd, check_grads, rel_l2, say, tdtype, to_dev, to_np

pytestmark = pytest.mark.gpu

NAMES = ("dq", "dk", "dv", "dtable")


def _step_inputs(H, Sq, Sk, d, nb, row_off, col_off, ld, dt, seed, masked_rows=0, zero_v=False,
                 o_scale=1.0):
    """Query shard, KV block, an asymmetric spd of rows row_off + Sq and
    stride ld, and a merged (O, LSE) standing for the whole ring: the block's
    own LSE log-added to a random contribution of the other blocks."""
    g = np.random.default_rng(seed)
    spd = g.integers(0, nb + 2, size=(row_off + Sq, ld)).astype(np.uint8)
    q = g.standard_normal((H, Sq, d)).astype(np.float32) / np.float32(math.sqrt(d))
    k = g.standard_normal((H, Sk, d)).astype(np.float32) / np.float32(math.sqrt(d))
    v = np.zeros((H, Sk, d), np.float32) if zero_v else g.standard_normal((H, Sk, d)).astype(np.float32)
    do = g.standard_normal((H, Sq, d)).astype(np.float32)
    o = (g.standard_normal((H, Sq, d)) * o_scale).astype(np.float32)
    table = (g.standard_normal((H, nb)) * 0.5).astype(np.float32)
    if masked_rows:
        table[:, :3] = -np.inf
        spd[row_off:row_off + masked_rows] = g.integers(0, 3, size=(masked_rows, ld))
    if dt == "bf16":
        q, k, v, do, o = (synth.round_bf16(x) for x in (q, k, v, do, o))
    scale = 1.0 / math.sqrt(d)
    _, lse_blk = oracle.ring_step(q, k, v, spd, row_off, col_off, table, scale)
    other = g.standard_normal((H, Sq)) + 1.0
    if masked_rows:
        other[:, :masked_rows] = -np.inf
    with np.errstate(divide="ignore"):
        lse = np.logaddexp(lse_blk, other).astype(np.float32)
    return q, k, v, do, o, lse, spd, table, scale


def _run_step(q, k, v, do, o, lse, spd, table, row_off, col_off, scale, dt, init):
    td = tdtype(dt)
    acc = tuple(to_dev(x) for x in init)
    gt.gt_attn_bwd_ring_step(to_dev(q, td), to_dev(o, td), to_dev(lse), to_dev(do, td),
                             to_dev(k, td), to_dev(v, td), to_dev(spd, torch.uint8),
                             row_off, col_off, to_dev(table), scale=scale, acc=acc)
    torch.cuda.synchronize()
    return {n: to_np(a) - x.astype(np.float64) for n, a, x in zip(NAMES, acc, init)}


def _init_acc(g, ref):
    """Nonzero starting accumulators of the magnitude of the step's result."""
    return tuple((g.standard_normal(ref[n].shape) * (np.abs(ref[n]).mean() + 1e-3)).astype(np.float32)
                 for n in NAMES)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("Sq,Sk,row_off,col_off,ld", [
    (200, 300, 37, 91, 512),      # unaligned slice: byte loads
    (256, 320, 64, 128, 512),     # 16-byte aligned slice: vector loads, full query tiles
    (256, 256, 0, 256, 512),      # aligned, whole key tiles
    (129, 1, 3, 500, 512),        # single key
    (64, 77, 0, 0, 77),           # ld not a multiple of 16
    (100, 700, 5, 300, 1024),     # more keys than queries (several 256-row blocks)
])
def test_bwd_ring_step_offsets(Sq, Sk, row_off, col_off, ld, dt):
    H, d, nb = 3, 64, 12
    q, k, v, do, o, lse, spd, table, scale = _step_inputs(H, Sq, Sk, d, nb, row_off, col_off, ld,
                                                          dt, seed=Sq * 3 + Sk)
    ref = dict(zip(NAMES, oracle.ring_backward_step(q, o, lse, do, k, v, spd, row_off, col_off,
                                                    table, scale)))
    init = _init_acc(np.random.default_rng(Sk), ref)
    say(f"bwd ring step {dt} Sq={Sq} Sk={Sk} row_off={row_off} col_off={col_off} ld={ld}")
    got = _run_step(q, k, v, do, o, lse, spd, table, row_off, col_off, scale, dt, init)
    check_grads(f"bwd ring step Sq={Sq} Sk={Sk}", got, ref, dt)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("d", [8, 16, 32, 64])
def test_bwd_ring_step_masked_rows(d, dt):
    """Rows whose every bucket is -inf have LSE = -inf over the whole ring:
    P = 0, so they add nothing (their dQ accumulator rows stay as they were)."""
    H, Sq, Sk, nb, m = 2, 150, 200, 9, 6
    q, k, v, do, o, lse, spd, table, scale = _step_inputs(H, Sq, Sk, d, nb, 10, 40, 256, dt,
                                                          seed=d, masked_rows=m)
    assert np.isneginf(lse[:, :m]).all()
    ref = dict(zip(NAMES, oracle.ring_backward_step(q, o, lse, do, k, v, spd, 10, 40, table, scale)))
    init = _init_acc(np.random.default_rng(1), ref)
    say(f"bwd ring step masked rows {dt} d={d}")
    got = _run_step(q, k, v, do, o, lse, spd, table, 10, 40, scale, dt, init)
    assert np.all(got["dq"][:, :m] == 0.0)
    check_grads("bwd ring step masked", got, ref, dt)


def test_bwd_ring_step_zero_values_large_output():
    """A KV block whose values are all zero while the merged O (from the other
    blocks) is large: dS = -P Dlt is set by O alone. The bf16 kernel's
    fixed-point range must come from |Dlt| here, not from |V|."""
    H, Sq, Sk, d, nb = 2, 200, 128, 64, 16
    q, k, v, do, o, lse, spd, table, scale = _step_inputs(H, Sq, Sk, d, nb, 0, 64, 256, "bf16",
                                                          seed=77, zero_v=True, o_scale=10.0)
    ref = dict(zip(NAMES, oracle.ring_backward_step(q, o, lse, do, k, v, spd, 0, 64, table, scale)))
    assert np.abs(ref["dtable"]).max() > 0 and np.all(ref["dv"] != 0)
    init = _init_acc(np.random.default_rng(2), ref)
    say("bwd ring step zero V, |O| ~ 10 (bf16)")
    got = _run_step(q, k, v, do, o, lse, spd, table, 0, 64, scale, "bf16", init)
    check_grads("bwd ring step zero V", got, ref, "bf16")


def test_bwd_ring_step_empty_block_leaves_accumulators():
    q = torch.randn(2, 70, 32, device=DEV).to(torch.bfloat16)
    lse = torch.randn(2, 70, device=DEV)
    t = torch.randn(2, 5, device=DEV)
    acc = (torch.randn(2, 70, 32, device=DEV), torch.zeros(2, 0, 32, device=DEV),
           torch.zeros(2, 0, 32, device=DEV), torch.randn(2, 5, device=DEV))
    before = [a.clone() for a in acc]
    gt.gt_attn_bwd_ring_step(q, q, lse, q, None, None, None, 0, 0, t, acc=acc)
    torch.cuda.synchronize()
    for a, b in zip(acc, before):
        assert torch.equal(a, b)


def _ring_case(H, N, d, nb, seed, dt):
    g = np.random.default_rng(seed)
    q, k, v = (g.standard_normal((H, N, d)).astype(np.float32) / np.float32(math.sqrt(d))
               for _ in range(3))
    do = g.standard_normal((H, N, d)).astype(np.float32)
    if dt == "bf16":
        q, k, v, do = (synth.round_bf16(x) for x in (q, k, v, do))
    table = (g.standard_normal((H, nb)) * 0.5).astype(np.float32)
    spd = g.integers(0, nb, size=(N, N)).astype(np.uint8)
    return q, k, v, do, table, spd


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("N,bounds", [
    (1000, [0, 240, 500, 777, 1000]),        # uneven shards, unaligned spd columns
    (1024, [0, 256, 512, 768, 1024]),        # even shards, 16-byte aligned slices
    (700, [0, 700]),                         # one rank: the ring is the full backward
])
def test_context_parallel_ring_backward(N, bounds, dt):
    """Every rank keeps its query rows and spd rows: forward ring steps and a
    merge give its (O, LSE); then it visits the KV blocks in ring order and
    adds each step's gradients (dQ locally, dK/dV into the block's
    accumulators that travel with it, dtable everywhere). The sums equal the
    unsharded oracle backward."""
    H, d, nb = 2, 64, 16
    q, k, v, do, table, spd = _ring_case(H, N, d, nb, seed=N, dt=dt)
    scale = 1.0 / math.sqrt(d)
    td = tdtype(dt)
    Q, K, V, dO, T = to_dev(q, td), to_dev(k, td), to_dev(v, td), to_dev(do, td), to_dev(table)
    P = len(bounds) - 1
    dq = torch.zeros(H, N, d, device=DEV)
    dk = torch.zeros(H, N, d, device=DEV)
    dv = torch.zeros(H, N, d, device=DEV)
    dtab = torch.zeros(H, nb, device=DEV)
    dk_blk = [torch.zeros(H, bounds[b + 1] - bounds[b], d, device=DEV) for b in range(P)]
    dv_blk = [torch.zeros(H, bounds[b + 1] - bounds[b], d, device=DEV) for b in range(P)]
    for r in range(P):
        r0, r1 = bounds[r], bounds[r + 1]
        shard = to_dev(spd[r0:r1], torch.uint8)
        q_r, do_r = Q[:, r0:r1].contiguous(), dO[:, r0:r1].contiguous()
        parts_o, parts_l = [], []
        for t in range(P):
            b = (r - t) % P
            c0, c1 = bounds[b], bounds[b + 1]
            o_p, l_p = gt.gt_attn_ring_step(q_r, K[:, c0:c1].contiguous(), V[:, c0:c1].contiguous(),
                                            shard, 0, c0, T, scale=scale)
            parts_o.append(o_p)
            parts_l.append(l_p)
        O_r, L_r = gt.gt_attn_merge(torch.stack(parts_o), torch.stack(parts_l), dtype=td)
        dq_r = torch.zeros(H, r1 - r0, d, device=DEV)
        for t in range(P):
            b = (r - t) % P
            c0, c1 = bounds[b], bounds[b + 1]
            gt.gt_attn_bwd_ring_step(q_r, O_r, L_r, do_r, K[:, c0:c1].contiguous(),
                                     V[:, c0:c1].contiguous(), shard, 0, c0, T, scale=scale,
                                     acc=(dq_r, dk_blk[b], dv_blk[b], dtab))
        dq[:, r0:r1] = dq_r
    for b in range(P):
        dk[:, bounds[b]:bounds[b + 1]] = dk_blk[b]
        dv[:, bounds[b]:bounds[b + 1]] = dv_blk[b]
    torch.cuda.synchronize()
    say(f"cp ring backward {dt} N={N} P={P}")
    ref = dict(zip(NAMES, oracle.backward(q, k, v, spd, table, scale, do)))
    got = dict(dq=to_np(dq), dk=to_np(dk), dv=to_np(dv), dtable=to_np(dtab))
    check_grads(f"cp ring backward N={N} P={P}", got, ref, dt)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("n_reg,n_super,bounds,d", [
    (900, 37, [0, 300, 612, 900], 64),       # uneven shards, unaligned spd columns
    (960, 64, [0, 320, 640, 960], 64),       # N = 1024: 16-byte aligned slices
    (500, 1, [0, 130, 250, 380, 500], 8),    # the paper's end-to-end shape: one global node, d = 8
])
def test_context_parallel_super_nodes(n_reg, n_super, bounds, d, dt):
    """Super nodes (Section III-A-1 parts 1-2): each rank's query shard is
    its regular rows plus every super-node row, with those spd rows only.
    Forward: the running merge over the P regular KV blocks in ring order and
    the super-node block once. Backward: the same steps, rank 0 carrying the
    super rows' dO (zero on the other ranks), dK/dV per block, the super
    block's accumulated by every rank. Both equal the unsharded oracle over
    all N = N' + N_s nodes, and every rank computes the same super rows."""
    H, nb = 2, 16
    N = n_reg + n_super
    q, k, v, do, table, spd = _ring_case(H, N, d, nb, seed=N + 1, dt=dt)
    scale = 1.0 / math.sqrt(d)
    td = tdtype(dt)
    Q, K, V, dO, T = to_dev(q, td), to_dev(k, td), to_dev(v, td), to_dev(do, td), to_dev(table)
    P = len(bounds) - 1
    blocks = [(bounds[j], bounds[j + 1]) for j in range(P)]
    O_ref, L_ref = oracle.forward(q, k, v, spd, table, scale)
    dq = torch.zeros(H, N, d, device=DEV)
    dk = torch.zeros(H, N, d, device=DEV)
    dv = torch.zeros(H, N, d, device=DEV)
    dtab = torch.zeros(H, nb, device=DEV)
    acc_k = {c: torch.zeros(H, e - c, d, device=DEV) for c, e in blocks + [(n_reg, N)]}
    acc_v = {c: torch.zeros(H, e - c, d, device=DEV) for c, e in blocks + [(n_reg, N)]}
    o_sup = []
    for r in range(P):
        # the schedule of the documented calling convention
        rows = np.array(ring.shard_rows(bounds, r, n_super))
        assert np.array_equal(rows, oracle.super_shard_rows(bounds, N, n_super, r))
        nr = bounds[r + 1] - bounds[r]
        idx = torch.from_numpy(rows).to(DEV)
        shard = to_dev(spd[rows], torch.uint8)
        q_r = Q[:, idx].contiguous()
        steps = ring.ring_steps(bounds, r, n_super)
        assert steps == [blocks[(r - t) % P] for t in range(P)] + [(n_reg, N)]
        state = None
        for c0, c1 in steps:
            Kb, Vb = K[:, c0:c1].contiguous(), V[:, c0:c1].contiguous()
            if state is None:
                state = gt.gt_attn_ring_step(q_r, Kb, Vb, shard, 0, c0, T, scale=scale)
            else:
                gt.gt_attn_ring_step_acc(q_r, Kb, Vb, shard, 0, c0, T, state, scale=scale)
        O_r, L_r = gt.gt_attn_merge(state[0][None].contiguous(), state[1][None].contiguous(), dtype=td)
        torch.cuda.synchronize()
        say(f"super nodes {dt} N'={n_reg} Ns={n_super} rank {r}: forward")
        check_fwd(f"super rank {r}", to_np(state[0]), to_np(state[1]), O_ref[:, rows], L_ref[:, rows], dt)
        o_sup.append(to_np(state[0])[:, nr:])
        do_r = dO[:, idx].contiguous()
        if not ring.carries_super_rows(r):
            do_r[:, nr:] = 0
        dq_r = torch.zeros(H, len(rows), d, device=DEV)
        for c0, c1 in steps:
            gt.gt_attn_bwd_ring_step(q_r, O_r, L_r, do_r, K[:, c0:c1].contiguous(),
                                     V[:, c0:c1].contiguous(), shard, 0, c0, T, scale=scale,
                                     acc=(dq_r, acc_k[c0], acc_v[c0], dtab))
        dq[:, bounds[r]:bounds[r + 1]] += dq_r[:, :nr]
        dq[:, n_reg:] += dq_r[:, nr:]
    for c0, c1 in blocks + [(n_reg, N)]:
        dk[:, c0:c1] = acc_k[c0]
        dv[:, c0:c1] = acc_v[c0]
    torch.cuda.synchronize()
    for o_s in o_sup[1:]:
        assert np.abs(o_s - o_sup[0]).max() <= 1e-5
    say(f"super nodes {dt} N'={n_reg} Ns={n_super}: backward")
    ref = dict(zip(NAMES, oracle.backward(q, k, v, spd, table, scale, do)))
    got = dict(dq=to_np(dq), dk=to_np(dk), dv=to_np(dv), dtable=to_np(dtab))
    check_grads(f"super nodes N'={n_reg} Ns={n_super}", got, ref, dt)
