"""Host-side schedule of one rank's context-parallel ring (Section III-A-1).

These helpers only compute node ranges; every step of the attention runs in
the library's kernels through gt_attn_ring_step, gt_attn_ring_step_acc and
gt_attn_bwd_ring_step. The convention (stated in include/gt_attn.h beside
the ring-step entry points):

  * P ranks split the N' regular nodes into contiguous blocks
    [bounds[r], bounds[r + 1]); N_s super nodes (ids N' .. N' + N_s - 1) are
    replicated on every rank.
  * Rank r's query shard is its regular rows followed by every super-node
    row (shard_rows); it holds only those spd rows.
  * At step t the rank holds regular KV block (r - t) mod P; with N_s > 0 one
    more step visits the super-node block, so every key counts once
    (ring_steps).
  * In the backward, rank 0 carries the replicated super-node rows' dO and
    every other rank passes zeros for them (carries_super_rows).
"""
from __future__ import annotations

from typing import Sequence


def _check(bounds: Sequence[int], rank: int, n_super: int) -> int:
    P = len(bounds) - 1
    if P < 1:
        raise ValueError("bounds must hold at least two entries")
    if bounds[0] != 0 or any(bounds[i] > bounds[i + 1] for i in range(P)):
        raise ValueError("bounds must start at 0 and be non-decreasing")
    if not 0 <= rank < P:
        raise ValueError(f"rank must be in [0, {P}), got {rank}")
    if n_super < 0:
        raise ValueError("n_super must be >= 0")
    return P


def shard_rows(bounds: Sequence[int], rank: int, n_super: int = 0) -> list[int]:
    """Global node ids of rank `rank`'s query shard, in shard order: its
    regular nodes, then every super node."""
    _check(bounds, rank, n_super)
    n_reg = bounds[-1]
    return list(range(bounds[rank], bounds[rank + 1])) + list(range(n_reg, n_reg + n_super))


def ring_steps(bounds: Sequence[int], rank: int, n_super: int = 0) -> list[tuple[int, int]]:
    """KV blocks (first node id, end node id) that rank `rank` visits, in
    order: at step t regular block (rank - t) mod P (it receives each block
    from its upstream neighbour), then, if there are super nodes, the
    super-node block once. The first id of each block is the ring step's
    col_off."""
    P = _check(bounds, rank, n_super)
    steps = []
    for t in range(P):
        b = (rank - t) % P
        steps.append((bounds[b], bounds[b + 1]))
    if n_super > 0:
        n_reg = bounds[-1]
        steps.append((n_reg, n_reg + n_super))
    return steps


def carries_super_rows(rank: int) -> bool:
    """Whether rank `rank` passes the super-node rows' dO in the backward
    (the other ranks pass zeros for those rows, so their loss counts once)."""
    return rank == 0
