"""Seeded synthetic graph generators and the SPD index matrix built from them.

Input construction only: the attention method takes the spd matrix as given
(structural encoding is built on the CPU during data loading, Section II-A).
Nothing in this module computes any part of the attention.

Graphs are undirected, simple (no self-loops, no multi-edges) and returned as
CSR arrays ``(indptr int64 [n+1], indices int32 [nnz])`` with both directions
stored.
"""
from __future__ import annotations

import ctypes
import os
from pathlib import Path

import numpy as np
import scipy.sparse as sp
from scipy.sparse.csgraph import connected_components

_HERE = Path(__file__).resolve().parent
_LIB_PATH = _HERE / "libspdgen.so"
_lib = None


def build_native(verbose: bool = False) -> Path:
    """Compile the native SPD generator (gcc + OpenMP) in place."""
    import subprocess

    cmd = ["gcc", "-O3", "-march=x86-64-v2", "-fopenmp", "-shared", "-fPIC",
           str(_HERE / "spdgen.c"), "-o", str(_LIB_PATH) + ".tmp"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(str(_LIB_PATH) + ".tmp", _LIB_PATH)
    return _LIB_PATH


def _native():
    global _lib
    if _lib is None:
        if not _LIB_PATH.exists():
            build_native()
        lib = ctypes.CDLL(str(_LIB_PATH))
        lib.spd_bfs_rows.restype = ctypes.c_int
        lib.spd_bfs_rows.argtypes = [
            ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
            ctypes.c_int64, ctypes.c_int32]
        lib.spd_iid_rows.restype = ctypes.c_int
        lib.spd_iid_rows.argtypes = [
            ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
            ctypes.c_int32, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int64,
            ctypes.c_int32]
        _lib = lib
    return _lib


def _threads() -> int:
    return int(os.environ.get("GT_SYNTH_THREADS", "0") or 0)


# --------------------------------------------------------------------------
# Graph generators
# --------------------------------------------------------------------------

def _csr_from_edges(n: int, src: np.ndarray, dst: np.ndarray):
    """Symmetric, deduplicated CSR without self-loops."""
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    keep = src != dst
    src, dst = src[keep], dst[keep]
    lo, hi = np.minimum(src, dst), np.maximum(src, dst)
    key = np.unique(lo * n + hi)
    lo, hi = key // n, key % n
    rows = np.concatenate([lo, hi])
    cols = np.concatenate([hi, lo])
    m = sp.csr_matrix((np.ones(rows.size, dtype=np.int8), (rows, cols)), shape=(n, n))
    m.sort_indices()
    return m.indptr.astype(np.int64), m.indices.astype(np.int32)


def erdos_renyi(n: int, avg_degree: float, rng: np.random.Generator):
    """G(n, p) with p = avg_degree / (n - 1): every pair independently."""
    p = avg_degree / max(n - 1, 1)
    iu, ju = np.triu_indices(n, k=1)
    keep = rng.random(iu.size) < p
    return _csr_from_edges(n, iu[keep], ju[keep])


def barabasi_albert(n: int, m: int, rng: np.random.Generator):
    """Preferential attachment: a clique on m+1 seed nodes, then every new
    node links to m distinct existing nodes drawn with probability
    proportional to degree (the repeated-endpoint list method)."""
    if n <= m + 1:
        iu, ju = np.triu_indices(n, k=1)
        return _csr_from_edges(n, iu, ju)
    iu, ju = np.triu_indices(m + 1, k=1)
    src = [iu.astype(np.int64)]
    dst = [ju.astype(np.int64)]
    # endpoint list: every edge contributes both ends
    cap = 2 * (iu.size + (n - m - 1) * m)
    ends = np.empty(cap, dtype=np.int64)
    ne = 2 * iu.size
    ends[:iu.size] = iu
    ends[iu.size:ne] = ju
    new_src = np.empty((n - m - 1) * m, dtype=np.int64)
    new_dst = np.empty((n - m - 1) * m, dtype=np.int64)
    w = 0
    # draw in batches, reject duplicates per node
    for v in range(m + 1, n):
        chosen = set()
        while len(chosen) < m:
            cand = ends[rng.integers(0, ne, size=2 * m)]
            for c in cand.tolist():
                if len(chosen) < m:
                    chosen.add(c)
        for c in chosen:
            new_src[w] = v
            new_dst[w] = c
            w += 1
            ends[ne] = v
            ends[ne + 1] = c
            ne += 2
    src.append(new_src[:w])
    dst.append(new_dst[:w])
    return _csr_from_edges(n, np.concatenate(src), np.concatenate(dst))


def planted_partition(n: int, n_comm: int, p_in: float, p_out: float,
                      rng: np.random.Generator):
    """Stochastic block model with n_comm equal contiguous communities:
    pairs inside a community link with p_in, pairs across with p_out.
    Edge counts are drawn binomially and endpoints uniformly (duplicates,
    which are rare at these densities, are merged)."""
    size = n // n_comm
    comm = np.minimum(np.arange(n) // size, n_comm - 1)
    srcs, dsts = [], []
    for c in range(n_comm):
        lo = c * size
        hi = n if c == n_comm - 1 else lo + size
        s = hi - lo
        pairs = s * (s - 1) // 2
        k = rng.binomial(pairs, p_in)
        a = rng.integers(lo, hi, size=k)
        b = rng.integers(lo, hi, size=k)
        srcs.append(a)
        dsts.append(b)
    total_pairs = n * (n - 1) // 2
    intra_pairs = sum(((n if c == n_comm - 1 else (c + 1) * size) - c * size) *
                      ((n if c == n_comm - 1 else (c + 1) * size) - c * size - 1) // 2
                      for c in range(n_comm))
    k = rng.binomial(total_pairs - intra_pairs, p_out)
    a = rng.integers(0, n, size=2 * k + 16)
    b = rng.integers(0, n, size=2 * k + 16)
    cross = comm[a] != comm[b]
    a, b = a[cross][:k], b[cross][:k]
    srcs.append(a)
    dsts.append(b)
    return _csr_from_edges(n, np.concatenate(srcs), np.concatenate(dsts))


def components(n: int, indptr: np.ndarray, indices: np.ndarray) -> np.ndarray:
    m = sp.csr_matrix((np.ones(indices.size, dtype=np.int8), indices, indptr), shape=(n, n))
    _, labels = connected_components(m, directed=False)
    return labels.astype(np.int32)


# --------------------------------------------------------------------------
# SPD rows
# --------------------------------------------------------------------------

class Graph:
    """A CSR graph plus its component labels; produces SPD rows on demand."""

    def __init__(self, n: int, indptr: np.ndarray, indices: np.ndarray):
        self.n = int(n)
        self.indptr = np.ascontiguousarray(indptr, dtype=np.int64)
        self.indices = np.ascontiguousarray(indices, dtype=np.int32)
        self.comp = components(self.n, self.indptr, self.indices)

    @property
    def n_edges(self) -> int:
        return int(self.indices.size // 2)

    def spd_rows(self, sources, clip: int, out: np.ndarray | None = None) -> np.ndarray:
        """uint8 [len(sources), n]: clipped BFS distance from each source."""
        src = np.ascontiguousarray(np.asarray(sources, dtype=np.int64).reshape(-1))
        if out is None:
            out = np.empty((src.size, self.n), dtype=np.uint8)
        assert out.dtype == np.uint8 and out.shape[0] == src.size and out.shape[1] >= self.n
        assert out.strides[1] == 1
        if src.size == 0:
            return out
        rc = _native().spd_bfs_rows(
            self.n, self.indptr.ctypes.data, self.indices.ctypes.data,
            self.comp.ctypes.data, src.ctypes.data, src.size, int(clip),
            out.ctypes.data, out.strides[0], _threads())
        if rc != 0:
            raise RuntimeError(f"spd_bfs_rows failed ({rc})")
        return out


def iid_spd_rows(n: int, row0: int, nrows: int, probs: np.ndarray, seed: int,
                 out: np.ndarray | None = None) -> np.ndarray:
    """Rows [row0, row0+nrows) of an n x n matrix of i.i.d. bucket draws with
    the given probabilities, diagonal 0 (counter-based: any row range of the
    same (n, probs, seed) gives identical bytes)."""
    probs = np.asarray(probs, dtype=np.float64)
    cdf = np.cumsum(probs / probs.sum())
    cdf[-1] = 1.0
    cdf = np.ascontiguousarray(cdf)
    if out is None:
        out = np.empty((nrows, n), dtype=np.uint8)
    assert out.dtype == np.uint8 and out.shape[0] == nrows and out.strides[1] == 1
    rc = _native().spd_iid_rows(n, row0, nrows, cdf.ctypes.data, cdf.size,
                                np.uint64(seed & 0xFFFFFFFFFFFFFFFF), out.ctypes.data,
                                out.strides[0], _threads())
    if rc != 0:
        raise RuntimeError(f"spd_iid_rows failed ({rc})")
    return out


def zipf_probs(n_buckets: int, s: float) -> np.ndarray:
    """Truncated Zipf: P(b) proportional to (b+1)^-s for b in [0, n_buckets)."""
    w = (np.arange(n_buckets, dtype=np.float64) + 1.0) ** (-s)
    return w / w.sum()
