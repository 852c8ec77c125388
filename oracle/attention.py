"""Reference (oracle) biased graph attention in fp64 NumPy. TEST INFRASTRUCTURE.

Parity status: every function here is pinned by CPU tests to things other
than itself (a library routine, closed forms, invariants, finite
differences, hand-derived values); see tests/test_oracle_pins.py.

Notation follows the paper (MegaGraph): H heads, N nodes, head dim d.
Section II-A, Eq. (1) defines the attention

    Attention(Q, K, V) = softmax(Q K^T / sqrt(d) + b_attn) V,

where b_attn is the structural-encoding bias (Section II-A: topology turned
into additive per-pair terms, e.g. from shortest-path distances, Section
III-A-1 part 2). Here the bias is a learned scalar per (head, SPD bucket):

    b_attn[h, i, j] = table[h, spd[i, j]]     (0 if spd[i, j] >= n_buckets).

Readings taken where the paper is silent (each is listed in the design
notes): the scale multiplies Q K^T only, never the bias; LSE is in natural
log; a row whose every score is -inf yields O = 0, LSE = -inf and zero
gradients; an out-of-range bucket contributes bias 0 and no gradient.

All arithmetic is fp64 on exactly the values the GPU receives (bf16 inputs
upcast exactly). Score blocks are materialised whole; nothing is tiled,
fused or reordered.
"""
from __future__ import annotations

import numpy as np

__all__ = ["bias_block", "block_attention", "block_backward", "forward", "backward",
           "ring_step", "merge", "ring_forward", "ring_backward_step", "ring_backward",
           "super_shard_rows", "ring_forward_super", "ring_backward_super", "lse_bias_only"]


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def bias_block(spd: np.ndarray, table_h: np.ndarray) -> np.ndarray:
    """Structural bias of one head for a block of node pairs.

    B[i, j] = table_h[spd[i, j]] when spd[i, j] < n_buckets, else 0
    (Section III-A-1 part 2; Eq. (2) adds the sliced bias b_i[:, Indices(K_j)]
    to the block's scores)."""
    spd = np.asarray(spd)
    table_h = _f64(table_h)
    idx = spd.astype(np.int64)
    inside = idx < table_h.shape[0]
    out = np.zeros(spd.shape, dtype=np.float64)
    out[inside] = table_h[idx[inside]]
    return out


def _scores(q_h, k_h, spd, table_h, scale):
    """S = scale * Q K^T + B (Eq. (1) for one head; Eq. (2) for a block)."""
    return scale * (_f64(q_h) @ _f64(k_h).T) + bias_block(spd, table_h)


def _row_lse(S: np.ndarray) -> np.ndarray:
    """Log-sum-exp of every row, natural log; -inf for an all -inf row."""
    m = S.max(axis=1) if S.shape[1] else np.full(S.shape[0], -np.inf)
    finite = np.isfinite(m)
    m0 = np.where(finite, m, 0.0)
    with np.errstate(under="ignore"):
        ssum = np.exp(S - m0[:, None]).sum(axis=1)
    with np.errstate(divide="ignore"):
        return np.where(finite, m0 + np.log(ssum), -np.inf)


def _probs(S: np.ndarray, lse: np.ndarray) -> np.ndarray:
    """Row softmax P = exp(S - LSE); rows with LSE = -inf are all zero."""
    finite = np.isfinite(lse)
    with np.errstate(under="ignore", invalid="ignore"):
        P = np.exp(S - np.where(finite, lse, 0.0)[:, None])
    P[~finite] = 0.0
    return P


def block_attention(q, k, v, spd, table, scale):
    """Biased attention of a query block against a key/value block.

    q [H, Sq, d], k and v [H, Sk, d], spd [Sq, Sk] (the bias slice aligned
    with these rows and columns), table [H, n_buckets].
    Returns O [H, Sq, d] (normalised within the block) and LSE [H, Sq].

    With the full node set this is Eq. (1); with a query shard and one KV
    block it is the per-step partial of the ring (Eq. (2) plus the
    bias-aware softmax statistics of Section III-A-1 part 3)."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    H, Sq, d = q.shape
    O = np.zeros((H, Sq, v.shape[2]), dtype=np.float64)
    L = np.zeros((H, Sq), dtype=np.float64)
    for h in range(H):
        S = _scores(q[h], k[h], spd, table[h], scale)
        lse = _row_lse(S)
        P = _probs(S, lse)
        O[h] = P @ v[h]
        L[h] = lse
    return O, L


def forward(q, k, v, spd, table, scale):
    """Eq. (1) over all N nodes: O [H, N, d], LSE [H, N]."""
    return block_attention(q, k, v, spd, table, scale)


def block_backward(q, k, v, spd, table, scale, d_out):
    """Gradients of L = sum(O * dO) for a query block against all keys.

    The paper does not write the backward out; it follows from Eq. (1) by
    the chain rule through the row softmax:
      P = softmax(S), dV = P^T dO, dP = dO V^T, Dlt_i = sum_c dO_ic O_ic,
      dS = P * (dP - Dlt), dQ = scale dS K, dK = scale dS^T Q,
      dTable[h, b] = sum of dS_ij over pairs with spd_ij = b (< n_buckets).
    No gradient reaches spd (an integer index).

    Given only some query rows (with their spd rows), dQ is exact for those
    rows, and dK, dV, dTable are exactly the full gradients of a dO that is
    zero outside them."""
    q, k, v, d_out = _f64(q), _f64(k), _f64(v), _f64(d_out)
    H, Sq, d = q.shape
    nb = table.shape[1]
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    dt = np.zeros((H, nb), dtype=np.float64)
    idx = np.asarray(spd).astype(np.int64)
    inside = idx < nb
    for h in range(H):
        S = _scores(q[h], k[h], spd, table[h], scale)
        lse = _row_lse(S)
        P = _probs(S, lse)
        O = P @ v[h]
        dv[h] = P.T @ d_out[h]
        dP = d_out[h] @ v[h].T
        dlt = (d_out[h] * O).sum(axis=1)
        dS = P * (dP - dlt[:, None])
        dq[h] = scale * (dS @ k[h])
        dk[h] = scale * (dS.T @ q[h])
        dt[h] = np.bincount(idx[inside], weights=dS[inside], minlength=nb)[:nb]
    return dq, dk, dv, dt


def backward(q, k, v, spd, table, scale, d_out):
    """Full backward over all N nodes: dQ, dK, dV [H, N, d], dTable [H, nb]."""
    return block_backward(q, k, v, spd, table, scale, d_out)


def ring_step(q_shard, k_shard, v_shard, spd, row_off, col_off, table, scale):
    """One graph-aware context-parallel step (Section III-A-1, parts 1-3).

    The rank holds the bias rows of its query shard (query-dimension bias
    sharding); for the incoming KV block it slices the bias columns of that
    block, spd[row_off:row_off+Sq, col_off:col_off+Sk], adds them to the
    block's scores (Eq. (2)) and returns the block-normalised partial
    (O_p, LSE_p). spd is any 2-D array whose element (r, c) is the SPD
    bucket of global query row r and global key column c."""
    Sq = q_shard.shape[1]
    Sk = k_shard.shape[1]
    blk = np.asarray(spd)[row_off:row_off + Sq, col_off:col_off + Sk]
    return block_attention(q_shard, k_shard, v_shard, blk, table, scale)


def merge(o_parts, lse_parts):
    """Combine block partials into the attention over all blocks.

    LSE = log sum_p exp(LSE_p); O = sum_p exp(LSE_p - LSE) O_p. The softmax
    statistics of every part already include that part's bias slice
    (Section III-A-1 part 3), so the combination is exact. Parts with
    LSE_p = -inf contribute nothing; if all are -inf, O = 0 and LSE = -inf.
    o_parts [P, H, S, d], lse_parts [P, H, S]."""
    o_parts = _f64(o_parts)
    lse_parts = _f64(lse_parts)
    m = lse_parts.max(axis=0)
    finite = np.isfinite(m)
    m0 = np.where(finite, m, 0.0)
    with np.errstate(under="ignore", invalid="ignore"):
        w = np.exp(lse_parts - m0[None])
    w[:, ~finite] = 0.0
    tot = w.sum(axis=0)
    with np.errstate(divide="ignore"):
        lse = np.where(finite, m0 + np.log(np.where(finite, tot, 1.0)), -np.inf)
    with np.errstate(invalid="ignore", divide="ignore"):
        wn = np.where(finite[None], w / np.where(finite, tot, 1.0)[None], 0.0)
    O = (wn[..., None] * o_parts).sum(axis=0)
    return O, lse


def ring_forward(q, k, v, spd, table, scale, bounds):
    """Simulate every rank of the ring on the CPU.

    bounds: shard boundaries [0 = b_0 < b_1 < ... < b_P = N] (shards may be
    uneven). Rank r keeps query rows [b_r, b_{r+1}) and only those spd rows;
    at step t it holds KV block (r - t) mod P (each rank passes its KV block
    downstream and receives the next from upstream, Section III-A-1 part 1).
    Returns the merged O [H, N, d] and LSE [H, N]."""
    P = len(bounds) - 1
    H, N, d = np.asarray(q).shape
    O = np.zeros((H, N, np.asarray(v).shape[2]))
    L = np.zeros((H, N))
    for r in range(P):
        r0, r1 = bounds[r], bounds[r + 1]
        spd_rows = np.asarray(spd)[r0:r1]           # this rank's bias shard
        parts_o, parts_l = [], []
        for t in range(P):
            blk = (r - t) % P
            c0, c1 = bounds[blk], bounds[blk + 1]
            o_p, l_p = ring_step(np.asarray(q)[:, r0:r1], np.asarray(k)[:, c0:c1],
                                 np.asarray(v)[:, c0:c1], spd_rows, 0, c0, table, scale)
            parts_o.append(o_p)
            parts_l.append(l_p)
        O[:, r0:r1], L[:, r0:r1] = merge(np.stack(parts_o), np.stack(parts_l))
    return O, L


def lse_bias_only(spd_rows, table):
    """LSE when Q = 0: every score of row i is its bias, so
    LSE_i = ln sum_b cnt_i[b] exp(table[b]) with cnt_i the bucket counts of
    spd row i (out-of-range buckets count with bias 0). [H, R]."""
    spd_rows = np.asarray(spd_rows)
    table = _f64(table)
    H, nb = table.shape
    out = np.zeros((H, spd_rows.shape[0]))
    for r in range(spd_rows.shape[0]):
        cnt = np.bincount(spd_rows[r].astype(np.int64), minlength=256)
        inside = cnt[:nb].astype(np.float64)
        outside = float(cnt[nb:].sum())
        for h in range(H):
            terms = [np.log(inside[b]) + table[h, b] for b in range(nb) if inside[b] > 0]
            if outside > 0:
                terms.append(np.log(outside))
            terms = np.array(terms)
            mx = terms.max()
            out[h, r] = mx + np.log(np.exp(terms - mx).sum())
    return out


def ring_backward_step(q_shard, o_shard, lse_shard, d_out_shard, k_blk, v_blk, spd, row_off,
                       col_off, table, scale):
    """Backward of one graph-aware context-parallel step: the rank's query
    shard against the KV block it holds (Section III-A-1 parts 1-3 run in
    reverse). The softmax of a query row spans every KV block, so P comes
    from the merged forward's LSE and Dlt from its merged O (never from the
    block's own partial):
      P = exp(S - LSE), S = scale Q K_blk^T + table[spd slice] (Eq. (2)),
      Dlt_i = sum_c dO_ic O_ic, dS = P * (dO V_blk^T - Dlt),
      dQ_part = scale dS K_blk, dK_part = scale dS^T Q, dV_part = P^T dO,
      dTable_part[h, b] = sum of dS_ij over the block's pairs with spd = b.
    The parts of all KV blocks add up to the full gradients; dK_part and
    dV_part belong to the KV block and travel with it around the ring.
    spd: any 2-D array whose element (r, c) is the bucket of global query
    row r and global key column c."""
    q, o, do = _f64(q_shard), _f64(o_shard), _f64(d_out_shard)
    k, v = _f64(k_blk), _f64(v_blk)
    lse = _f64(lse_shard)
    H, Sq, d = q.shape
    Sk = k.shape[1]
    nb = table.shape[1]
    blk = np.asarray(spd)[row_off:row_off + Sq, col_off:col_off + Sk]
    idx = blk.astype(np.int64)
    inside = idx < nb
    dq = np.zeros_like(q)
    dk = np.zeros_like(k)
    dv = np.zeros_like(v)
    dt = np.zeros((H, nb), dtype=np.float64)
    for h in range(H):
        S = _scores(q[h], k[h], blk, table[h], scale)
        P = _probs(S, lse[h])
        dP = do[h] @ v[h].T
        dlt = (do[h] * o[h]).sum(axis=1)
        dS = P * (dP - dlt[:, None])
        dq[h] = scale * (dS @ k[h])
        dk[h] = scale * (dS.T @ q[h])
        dv[h] = P.T @ do[h]
        dt[h] = np.bincount(idx[inside], weights=dS[inside], minlength=nb)[:nb]
    return dq, dk, dv, dt


def ring_backward(q, k, v, spd, table, scale, d_out, bounds):
    """Simulate the backward of every rank of the ring on the CPU: each rank
    keeps its query rows and spd rows, runs ring_forward's merged (O, LSE)
    for them, and visits the KV blocks in ring order, accumulating dQ
    locally and each block's dK/dV parts and dTable across ranks.
    Returns dQ, dK, dV [H, N, d] and dTable [H, nb]."""
    P = len(bounds) - 1
    q, k, v, d_out = np.asarray(q), np.asarray(k), np.asarray(v), np.asarray(d_out)
    O, L = ring_forward(q, k, v, spd, table, scale, bounds)
    dq = np.zeros(q.shape)
    dk = np.zeros(k.shape)
    dv = np.zeros(v.shape)
    dt = np.zeros(table.shape)
    for r in range(P):
        r0, r1 = bounds[r], bounds[r + 1]
        spd_rows = np.asarray(spd)[r0:r1]
        for t in range(P):
            blk = (r - t) % P
            c0, c1 = bounds[blk], bounds[blk + 1]
            a, b, c, e = ring_backward_step(q[:, r0:r1], O[:, r0:r1], L[:, r0:r1], d_out[:, r0:r1],
                                            k[:, c0:c1], v[:, c0:c1], spd_rows, 0, c0, table, scale)
            dq[:, r0:r1] += a
            dk[:, c0:c1] += b
            dv[:, c0:c1] += c
            dt += e
    return dq, dk, dv, dt


def super_shard_rows(bounds, n_total, n_super, r):
    """Global node ids of rank r's query shard when the batch holds
    N' = n_total - n_super regular nodes (ids 0..N'-1, split by bounds over
    [0, N']) and n_super global super nodes (ids N'..n_total-1): the rank's
    regular nodes followed by every super node (Section III-A-1 part 1: the
    regular nodes are partitioned, the super nodes replicated)."""
    n_reg = n_total - n_super
    return np.concatenate([np.arange(bounds[r], bounds[r + 1]), np.arange(n_reg, n_total)])


def ring_forward_super(q, k, v, spd, table, scale, bounds, n_super):
    """Simulate every rank of the ring when the batch has super nodes.

    Rank r keeps the query rows super_shard_rows(...) and only those spd rows
    (its bias shard [N'/P + N_s, N' + N_s], Section III-A-1 part 2). It visits
    the P regular KV blocks in ring order (block (r - t) mod P, columns
    [b_j, b_{j+1})) and, once, the super-node KV block (columns [N', N)),
    then merges the P + 1 partials. Every super-node key thus enters each
    query's softmax exactly once (the reading taken where the paper puts the
    super nodes in every KV block). Returns O [H, N, d] and LSE [H, N] (the
    super rows from rank 0) and, per rank, the super rows' (O, LSE), which
    every rank computes."""
    q, k, v, spd = np.asarray(q), np.asarray(k), np.asarray(v), np.asarray(spd)
    P = len(bounds) - 1
    H, N, _ = q.shape
    n_reg = N - n_super
    O = np.zeros((H, N, v.shape[2]))
    L = np.zeros((H, N))
    per_rank_super = []
    for r in range(P):
        rows = super_shard_rows(bounds, N, n_super, r)
        spd_rows = spd[rows]
        qs = q[:, rows]
        parts_o, parts_l = [], []
        for t in range(P):
            blk = (r - t) % P
            c0, c1 = bounds[blk], bounds[blk + 1]
            o_p, l_p = ring_step(qs, k[:, c0:c1], v[:, c0:c1], spd_rows, 0, c0, table, scale)
            parts_o.append(o_p)
            parts_l.append(l_p)
        if n_super > 0:
            o_p, l_p = ring_step(qs, k[:, n_reg:], v[:, n_reg:], spd_rows, 0, n_reg, table, scale)
            parts_o.append(o_p)
            parts_l.append(l_p)
        o_r, l_r = merge(np.stack(parts_o), np.stack(parts_l))
        nr = bounds[r + 1] - bounds[r]
        O[:, bounds[r]:bounds[r + 1]] = o_r[:, :nr]
        L[:, bounds[r]:bounds[r + 1]] = l_r[:, :nr]
        per_rank_super.append((o_r[:, nr:], l_r[:, nr:]))
        if r == 0:
            O[:, n_reg:] = o_r[:, nr:]
            L[:, n_reg:] = l_r[:, nr:]
    return O, L, per_rank_super


def ring_backward_super(q, k, v, spd, table, scale, d_out, bounds, n_super):
    """Backward of ring_forward_super on every rank. The super-node query rows
    are replicated, so their loss terms must be counted once: rank 0 carries
    their dO and every other rank passes dO = 0 for them (then their dS is 0
    there: dP = 0 and Dlt = 0). Each rank visits the regular KV blocks and the
    super block with ring_backward_step, accumulating its rows' dQ and each
    block's dK, dV and dTable. Returns dQ, dK, dV [H, N, d] and dTable."""
    q, k, v, spd, d_out = (np.asarray(x) for x in (q, k, v, spd, d_out))
    P = len(bounds) - 1
    H, N, _ = q.shape
    n_reg = N - n_super
    O, L, _ = ring_forward_super(q, k, v, spd, table, scale, bounds, n_super)
    dq = np.zeros(q.shape)
    dk = np.zeros(k.shape)
    dv = np.zeros(v.shape)
    dt = np.zeros(table.shape)
    blocks = [(bounds[j], bounds[j + 1]) for j in range(P)]
    for r in range(P):
        rows = super_shard_rows(bounds, N, n_super, r)
        spd_rows = spd[rows]
        do_r = d_out[:, rows].copy()
        nr = bounds[r + 1] - bounds[r]
        if r != 0:
            do_r[:, nr:] = 0.0
        steps = [blocks[(r - t) % P] for t in range(P)]
        if n_super > 0:
            steps.append((n_reg, N))
        for c0, c1 in steps:
            a, b, c, e = ring_backward_step(q[:, rows], O[:, rows], L[:, rows], do_r,
                                            k[:, c0:c1], v[:, c0:c1], spd_rows, 0, c0, table, scale)
            dq[:, rows] += a
            dk[:, c0:c1] += b
            dv[:, c0:c1] += c
            dt += e
    return dq, dk, dv, dt
