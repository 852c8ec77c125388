"""The ring schedule helpers (host logic, CPU): each rank's query shard and
the KV blocks it visits, against the ring order of Section III-A-1 and the
oracle's super-node shards."""
import numpy as np
import pytest

import oracle
from paper_2609_34420_amd import ring


@pytest.mark.parametrize("bounds,n_super", [([0, 40], 0), ([0, 11, 40], 7), ([0, 5, 19, 33, 40], 1),
                                            ([0, 8, 16, 24, 32, 40, 48, 56, 64], 3)])
def test_schedule(bounds, n_super):
    P = len(bounds) - 1
    n_reg = bounds[-1]
    seen = {}
    for r in range(P):
        rows = ring.shard_rows(bounds, r, n_super)
        assert np.array_equal(rows, oracle.super_shard_rows(bounds, n_reg + n_super, n_super, r))
        steps = ring.ring_steps(bounds, r, n_super)
        assert len(steps) == P + (1 if n_super else 0)
        # step t holds block (r - t) mod P: each rank receives from upstream
        for t in range(P):
            assert steps[t] == (bounds[(r - t) % P], bounds[(r - t) % P + 1])
        # every key is visited exactly once per rank
        cols = [c for a, b in steps for c in range(a, b)]
        assert sorted(cols) == list(range(n_reg + n_super))
        for t, blk in enumerate(steps[:P]):
            seen.setdefault(t, set()).add(blk)
        assert ring.carries_super_rows(r) == (r == 0)
    # at every step the P ranks hold P distinct blocks (a ring rotation)
    for t, blks in seen.items():
        assert len(blks) == len(set(zip(bounds[:-1], bounds[1:])))


def test_rank_three_of_eight_visits_blocks_in_ring_order():
    bounds = [i * 32768 for i in range(9)]
    steps = ring.ring_steps(bounds, 3)
    assert [a // 32768 for a, _ in steps] == [3, 2, 1, 0, 7, 6, 5, 4]


@pytest.mark.parametrize("bounds,rank,n_super", [([0], 0, 0), ([1, 4], 0, 0), ([0, 5, 3], 0, 0),
                                                 ([0, 4], 1, 0), ([0, 4], 0, -1)])
def test_schedule_rejects(bounds, rank, n_super):
    with pytest.raises(ValueError):
        ring.ring_steps(bounds, rank, n_super)
