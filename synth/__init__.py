"""Seeded synthetic workloads for biased graph attention.

This package is the ONLY code shared between the CPU oracle and the HIP path.
It builds inputs (graphs, the uint8 SPD index matrix, Q/K/V/dO, bias tables)
and holds none of the attention arithmetic.

Every workload is a deterministic function of (name, seed). Random draws use
numpy PCG64 streams keyed by (seed, stream name, layer), so any tensor can be
regenerated on its own. bf16 workloads round their float tensors to the
nearest bf16 value (round-to-nearest-even) here, so both sides receive the
identical values: the oracle upcasts them exactly, the GPU side stores them
as bfloat16 without a further rounding step.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

from . import graphs
from .graphs import Graph, iid_spd_rows, zipf_probs

_STREAMS = {"graph": 1, "q": 2, "k": 3, "v": 4, "do": 5, "table": 6, "rows": 7,
            "spd": 8, "perm": 9, "misc": 10}


def rng(seed: int, stream: str, layer: int = 0) -> np.random.Generator:
    """Independent named substream of the master seed (numpy)."""
    ss = np.random.SeedSequence(entropy=int(seed), spawn_key=(_STREAMS[stream], int(layer)))
    return np.random.Generator(np.random.PCG64(ss))


def stream_seed(seed: int, stream: str, layer: int = 0) -> int:
    """63-bit seed of a named substream (for torch CPU generators)."""
    ss = np.random.SeedSequence(entropy=int(seed), spawn_key=(_STREAMS[stream], int(layer)))
    return int(ss.generate_state(1, np.uint64)[0] >> np.uint64(1))


def normal(seed: int, stream: str, shape, layer: int = 0) -> np.ndarray:
    """float32 N(0, 1) draws of a named substream. torch's CPU generator is
    used for speed; its output does not depend on the thread count."""
    import torch

    g = torch.Generator().manual_seed(stream_seed(seed, stream, layer))
    return torch.randn(tuple(shape), generator=g, dtype=torch.float32).numpy()


def round_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest bf16 value (ties to even), returned as float32.
    Input quantisation, not arithmetic of the method."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


@dataclass
class Workload:
    """One synthetic configuration (all sizes of one run)."""
    name: str
    N: int                      # nodes
    H: int                      # heads
    d: int                      # head dim
    dtype: str                  # "f32" | "bf16"
    graph: tuple                # ("er", avg_deg) | ("ba", m) | ("sbm", n_comm, p_in, p_out)
    clip: int                   # SPD clip D; unreachable -> D+1
    n_buckets: int              # table width D+2 (or the Zipf bucket count)
    qkv_std: float              # Q,K,V ~ N(0, qkv_std^2)
    table_std: float = 0.02
    layers: int = 1
    spd_law: tuple | None = None    # ("zipf", s): i.i.d. buckets instead of BFS
    shards: int = 1             # context-parallel split of N
    shard: int = 0              # the query shard this device owns
    note: str = ""
    _graph: Graph | None = field(default=None, repr=False)

    # ---- sizes ------------------------------------------------------------
    @property
    def spd_symmetric(self) -> bool:
        """BFS distances on an undirected graph: spd[i, j] == spd[j, i]."""
        return self.spd_law is None

    @property
    def S(self) -> int:
        return self.N // self.shards

    @property
    def flops_fwd_bwd(self) -> float:
        """4 N^2 d H forward + 10 N^2 d H backward, per layer."""
        return 14.0 * self.N * self.N * self.d * self.H * self.layers

    # ---- graph / spd ------------------------------------------------------
    def graph_obj(self, seed: int = 0) -> Graph:
        if self._graph is None:
            g = rng(seed, "graph")
            kind = self.graph[0]
            if kind == "er":
                ip, ix = graphs.erdos_renyi(self.N, self.graph[1], g)
            elif kind == "ba":
                ip, ix = graphs.barabasi_albert(self.N, self.graph[1], g)
            elif kind == "sbm":
                ip, ix = graphs.planted_partition(self.N, self.graph[1], self.graph[2],
                                                  self.graph[3], g)
            else:
                raise ValueError(kind)
            self._graph = Graph(self.N, ip, ix)
        return self._graph

    def spd_rows(self, rows, seed: int = 0, out: np.ndarray | None = None) -> np.ndarray:
        """uint8 [len(rows), N]: the spd rows for the given global node ids."""
        rows = np.asarray(rows, dtype=np.int64).reshape(-1)
        if self.spd_law is not None:
            assert self.spd_law[0] == "zipf"
            probs = zipf_probs(self.n_buckets, self.spd_law[1])
            if out is None:
                out = np.empty((rows.size, self.N), dtype=np.uint8)
            # counter-based: contiguous runs are generated row by row
            for t, r in enumerate(rows.tolist()):
                iid_spd_rows(self.N, r, 1, probs, _spd_seed(seed), out=out[t:t + 1])
            return out
        return self.graph_obj(seed).spd_rows(rows, self.clip, out=out)

    def spd_block(self, row0: int, nrows: int, seed: int = 0,
                  out: np.ndarray | None = None) -> np.ndarray:
        """uint8 [nrows, N]: contiguous spd rows [row0, row0+nrows)."""
        if self.spd_law is not None:
            probs = zipf_probs(self.n_buckets, self.spd_law[1])
            return iid_spd_rows(self.N, row0, nrows, probs, _spd_seed(seed), out=out)
        return self.graph_obj(seed).spd_rows(np.arange(row0, row0 + nrows), self.clip, out=out)

    # ---- dense tensors ----------------------------------------------------
    def _normal(self, seed, stream, shape, std, layer=0):
        x = normal(seed, stream, shape, layer)
        if std != 1.0:
            x *= np.float32(std)
        return round_bf16(x) if self.dtype == "bf16" else x

    def qkv(self, seed: int = 0, layer: int = 0, rows: slice | None = None):
        shp = (self.H, self.N, self.d)
        q = self._normal(seed, "q", shp, self.qkv_std, layer)
        k = self._normal(seed, "k", shp, self.qkv_std, layer)
        v = self._normal(seed, "v", shp, self.qkv_std, layer)
        return q, k, v

    def d_out(self, seed: int = 0, layer: int = 0):
        return self._normal(seed, "do", (self.H, self.N, self.d), 1.0, layer)

    def table(self, seed: int = 0, layer: int = 0) -> np.ndarray:
        """fp32 [H, n_buckets]; the bias table is always fp32."""
        t = rng(seed, "table", layer).standard_normal(size=(self.H, self.n_buckets),
                                                      dtype=np.float32)
        return (t * np.float32(self.table_std)).astype(np.float32)

    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    def sample_rows(self, count: int, seed: int = 0, lo: int = 0, hi: int | None = None):
        """Sorted seeded row sample in [lo, hi) that always holds both ends."""
        hi = self.N if hi is None else hi
        g = rng(seed, "rows")
        k = min(count, hi - lo)
        r = g.choice(np.arange(lo, hi), size=k, replace=False)
        r = np.unique(np.concatenate([r, [lo, hi - 1]]))
        return r.astype(np.int64)

    def stratified_rows(self, count: int, block: int = 256, seed: int = 0, lo: int = 0,
                        hi: int | None = None):
        """Sorted seeded row sample in [lo, hi): the range is cut into blocks
        of `block` rows and each block contributes the same number of rows
        (at least one, at most the block's size), drawn without replacement,
        plus both ends of the range. Every block of the kernels' row tiles
        (any multiple of `block`) then holds a sampled row."""
        hi = self.N if hi is None else hi
        g = rng(seed, "rows")
        nblk = (hi - lo + block - 1) // block
        per = max(1, -(-count // nblk))
        picks = [np.array([lo, hi - 1])]
        for b in range(nblk):
            a, e = lo + b * block, min(hi, lo + (b + 1) * block)
            picks.append(g.choice(np.arange(a, e), size=min(per, e - a), replace=False))
        return np.unique(np.concatenate(picks)).astype(np.int64)


def _spd_seed(seed: int) -> int:
    return int(np.random.SeedSequence(entropy=int(seed),
                                      spawn_key=(_STREAMS["spd"],)).generate_state(1, np.uint64)[0])


def _mk():
    return {
        # Erdos-Renyi, average degree 8, BFS spd clipped to 20, unreachable 21.
        "tiny": Workload("tiny", N=512, H=4, d=32, dtype="f32", graph=("er", 8.0),
                         clip=20, n_buckets=22, qkv_std=1.0),
        # Barabasi-Albert m=4, clip 30, unreachable 31.
        "ba16k": Workload("ba16k", N=16384, H=8, d=64, dtype="bf16", graph=("ba", 4),
                          clip=30, n_buckets=32, qkv_std=1.0 / 8.0),
        # Clustered graph: 64 contiguous communities, p_in 1e-3, p_out 1e-6,
        # clip 62, unreachable 63 (N^2 = 17.2e9 spd bytes).
        "sbm128k": Workload("sbm128k", N=131072, H=8, d=64, dtype="bf16",
                            graph=("sbm", 64, 1e-3, 1e-6), clip=62, n_buckets=64,
                            qkv_std=1.0 / 8.0),
        # Context-parallel share: N=262144 in 8 shards of 32768, query shard 3.
        "cp256k": Workload("cp256k", N=262144, H=8, d=64, dtype="bf16", graph=("ba", 4),
                           clip=30, n_buckets=32, qkv_std=1.0 / 8.0, shards=8, shard=3),
        # 12 layers, N=32768, H=16, 256 Zipf(1.2) buckets shared by all layers.
        "deep32k": Workload("deep32k", N=32768, H=16, d=64, dtype="bf16", graph=("ba", 8),
                            clip=254, n_buckets=256, qkv_std=1.0 / 8.0, layers=12,
                            spd_law=("zipf", 1.2)),
    }


WORKLOADS = _mk()


def workload(name: str) -> Workload:
    """A fresh Workload (graph caches are per instance)."""
    return _mk()[name]

