"""Seeded input generators: graphs, clipped BFS spd, Zipf spd, bf16 rounding."""
import hashlib

import numpy as np
import pytest
import scipy.sparse as sp
import torch
from scipy.sparse.csgraph import shortest_path

import synth
from synth import graphs


def _scipy_spd(g: graphs.Graph, rows, clip):
    m = sp.csr_matrix((np.ones(g.indices.size), g.indices, g.indptr), shape=(g.n, g.n))
    if g.n <= 64:  # Floyd-Warshall on the whole graph, then pick rows
        D = shortest_path(m, method="FW", unweighted=True)[np.asarray(rows)]
    else:
        D = shortest_path(m, method="D", unweighted=True, indices=rows)
    return np.where(np.isinf(D), clip + 1, np.minimum(D, clip)).astype(np.uint8)


@pytest.mark.parametrize("kind", ["er", "ba", "sbm"])
def test_bfs_spd_matches_shortest_path(kind):
    g0 = np.random.default_rng(3)
    if kind == "er":
        ip, ix = graphs.erdos_renyi(60, 2.0, g0)       # sparse: several components
    elif kind == "ba":
        ip, ix = graphs.barabasi_albert(64, 2, g0)
    else:
        ip, ix = graphs.planted_partition(64, 4, 0.2, 0.01, g0)
    g = graphs.Graph(ip.size - 1, ip, ix)
    for clip in (1, 2, 3, 20):
        rows = np.arange(g.n)
        mine = g.spd_rows(rows, clip)
        ref = _scipy_spd(g, rows, clip)
        np.testing.assert_array_equal(mine, ref)
        assert np.all(np.diag(mine) == 0)
    # a row subset in arbitrary order (more than one 64-source block)
    rows = np.random.default_rng(4).permutation(g.n)[:50]
    np.testing.assert_array_equal(g.spd_rows(rows, 5), _scipy_spd(g, rows, 5))


def test_tiny_workload_spd_and_determinism():
    w = synth.workload("tiny")
    spd = w.spd_block(0, w.N)
    assert spd.shape == (512, 512) and spd.dtype == np.uint8
    assert np.all(np.diag(spd) == 0)
    assert spd.max() <= 21
    np.testing.assert_array_equal(spd, spd.T)          # undirected graph
    ref = _scipy_spd(w.graph_obj(), np.arange(w.N), 20)
    np.testing.assert_array_equal(spd, ref)
    h1 = hashlib.sha256(spd.tobytes()).hexdigest()
    h2 = hashlib.sha256(synth.workload("tiny").spd_block(0, w.N).tobytes()).hexdigest()
    assert h1 == h2
    # ER average degree 8
    assert 6.5 < 2 * w.graph_obj().n_edges / w.N < 9.5


def test_ba_edge_count():
    ip, ix = graphs.barabasi_albert(500, 4, np.random.default_rng(0))
    assert ix.size // 2 == 10 + (500 - 5) * 4


def test_sbm_edge_statistics():
    g = np.random.default_rng(5)
    n, c, pin, pout = 8192, 8, 2e-3, 1e-5
    ip, ix = graphs.planted_partition(n, c, pin, pout, g)
    src = np.repeat(np.arange(n), np.diff(ip))
    comm = src // (n // c)
    intra = (comm == ix // (n // c)).sum() // 2
    inter = ix.size // 2 - intra
    e_intra = c * (n // c) * (n // c - 1) / 2 * pin
    e_inter = (n * (n - 1) / 2 - c * (n // c) * (n // c - 1) / 2) * pout
    assert abs(intra - e_intra) < 5 * np.sqrt(e_intra)
    assert abs(inter - e_inter) < 5 * np.sqrt(e_inter) + 5


def test_zipf_spd_distribution_and_counter_based():
    probs = graphs.zipf_probs(256, 1.2)
    n = 4096
    a = graphs.iid_spd_rows(n, 0, 64, probs, seed=99)
    b = graphs.iid_spd_rows(n, 32, 16, probs, seed=99)
    np.testing.assert_array_equal(a[32:48], b)          # any row range, same bytes
    assert all(a[r, r] == 0 for r in range(64))
    off = a[~np.eye(64, n, dtype=bool)]
    freq = np.bincount(off, minlength=256) / off.size
    assert abs(freq[0] - probs[0]) < 0.01               # ~25 % in bucket 0
    assert abs(freq[1] - probs[1]) < 0.01
    assert 0.2 < probs[0] < 0.3


def test_round_bf16_is_round_to_nearest_even():
    """Against the bit-level definition: add 0x7FFF plus the lowest kept bit,
    then truncate the low 16 bits (finite inputs)."""
    x = np.random.default_rng(6).standard_normal(100000).astype(np.float32) * 3
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 0.0]   # ties round to even
    mine = synth.round_bf16(x)
    u = x.view(np.uint32).astype(np.uint64)
    ref = ((u + ((u >> 16) & 1) + 0x7FFF) & 0xFFFF0000).astype(np.uint32).view(np.float32)
    np.testing.assert_array_equal(mine, ref)
    assert mine[0] == 1.0 and mine[1] == 1.0 + 2 ** -6


def test_workload_tensors_are_seeded_and_bf16_exact():
    w = synth.workload("ba16k")
    w.N = 256
    q, k, v = w.qkv(0)
    q2, _, _ = w.qkv(0)
    np.testing.assert_array_equal(q, q2)
    assert not np.array_equal(q, k)
    assert np.array_equal(synth.round_bf16(q), q)
    t = w.table(0)
    assert t.shape == (8, 32) and t.dtype == np.float32
    assert 0.01 < t.std() < 0.03


def test_bfs_spd_is_symmetric_and_iid_is_not():
    """The bench passes spd as its own transpose for BFS workloads: pin that
    their distance matrices are symmetric (undirected graphs), and that the
    i.i.d. law is not (it takes the column-gather path)."""
    w = synth.workload("tiny")
    assert w.spd_symmetric
    spd = w.spd_block(0, w.N)
    assert (spd == spd.T).all()
    b = synth.workload("ba16k")
    rows = b.spd_block(0, 64)
    cols = b.spd_rows(np.arange(64))        # rows 0..63 again, by id
    assert (rows == cols).all()
    sub = b.spd_rows(np.arange(64))[:, :64]
    assert (sub == sub.T).all()
    d = synth.workload("deep32k")
    assert not d.spd_symmetric
    blk = d.spd_block(0, 64)[:, :64]
    assert not (blk == blk.T).all()
