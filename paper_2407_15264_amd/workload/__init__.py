"""Seeded synthetic workloads for the feature-gather cache.

Inputs only: an R-MAT graph (CSR by source), the in-degree static score, raw
request streams from GraphSAGE-style uniform neighbour sampling, and N(0,1)
feature rows.  The arithmetic lives in ``gen.c`` (C + OpenMP, counter-based
SplitMix64 draws, so results do not depend on thread count).  Nothing in here
computes any part of the cache method; both the CPU oracle's tests and the GPU
path's tests and benchmark draw their inputs from this module.

The five workload shapes mirror the paper's evaluation datasets (Sec. 5,
dataset table) at synthetic stand-in scale; the paper's own datasets are not
available, so these R-MAT graphs replace them.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libworkload.so")
GIB = 1 << 30


@dataclasses.dataclass(frozen=True)
class CacheShape:
    num_sets: int
    victim_rows: int
    lookahead: int
    near_threshold: int = 0  # 0 -> max(1, L // 8)


@dataclasses.dataclass(frozen=True)
class WorkloadConfig:
    name: str
    num_nodes: int
    num_edges: int
    dim: int
    elt_bytes: int  # 4 = fp32, 2 = fp16
    batches: int
    batch_size: int
    fanout: tuple
    cache: CacheShape
    rmat: tuple = (0.57, 0.19, 0.19)  # (a, b, c); d = 1 - a - b - c
    seed: int = 0

    @property
    def row_bytes(self) -> int:
        return self.dim * self.elt_bytes

    @property
    def feature_dtype(self) -> str:
        return "fp32" if self.elt_bytes == 4 else "fp16"

    def describe(self) -> dict:
        return {
            "workload": self.name,
            "num_nodes": self.num_nodes,
            "num_edges": self.num_edges,
            "feature": f"{self.feature_dtype}x{self.dim}",
            "row_bytes": self.row_bytes,
            "batch_size": self.batch_size,
            "fanout": list(self.fanout),
            "num_sets": self.cache.num_sets,
            "ways": 8,
            "victim_rows": self.cache.victim_rows,
            "lookahead": self.cache.lookahead,
        }


def _cache_lines_for(bytes_budget: int, row_bytes: int) -> int:
    return bytes_budget // row_bytes


# Workload names, smallest to largest.
RMAT14 = "rmat-s14-e18-f32x128"
RMAT20 = "rmat-s20-deg16-f32x256"
RMAT10M = "rmat-10M-e120M-f32x1024"
TYPED20M = "rmat-20M-e250M-4types"
RMAT100M = "rmat-100M-e1.6B-f16x1024"

# The homogeneous workload shapes, by name.  Cache/ring budgets in GiB; cache
# sets are the budget in rows divided by the 8 ways.
CONFIGS = {
    RMAT14: WorkloadConfig(RMAT14, 1 << 14, 1 << 18, 128, 4, 20, 256, (10, 5),
                      CacheShape(num_sets=2048, victim_rows=1024, lookahead=2)),
    RMAT20: WorkloadConfig(RMAT20, 1 << 20, 1 << 24, 256, 4, 200, 1024, (15, 10, 5),
                      CacheShape(num_sets=int(0.10 * (1 << 20)) // 8, victim_rows=int(0.05 * (1 << 20)),
                                 lookahead=4)),
    RMAT10M: WorkloadConfig(RMAT10M, 10_000_000, 120_000_000, 1024, 4, 500, 4096, (10, 5, 5),
                      CacheShape(num_sets=_cache_lines_for(8 * GIB, 4096) // 8,
                                 victim_rows=_cache_lines_for(4 * GIB, 4096), lookahead=8)),
    RMAT100M: WorkloadConfig(RMAT100M, 100_000_000, 1_600_000_000, 1024, 2, 1000, 8192, (15, 10, 5),
                      CacheShape(num_sets=_cache_lines_for(96 * GIB, 2048) // 8,
                                 victim_rows=_cache_lines_for(32 * GIB, 2048), lookahead=16)),
}


@dataclasses.dataclass(frozen=True)
class HeteroConfig:
    """A typed graph: one homogeneous R-MAT graph over all nodes, each node given
    a type by a seeded permutation (the first type_share[0] of the permuted
    order is type 0, and so on; a node's local ID is its position within its
    type), each type with its own feature width and its own cache.  The cache
    and victim-ring budgets are split in proportion to each type's store bytes.
    Edge types play no part in sampling."""
    name: str
    num_nodes: int
    num_edges: int
    type_share: tuple
    dims: tuple
    elt_bytes: int
    batches: int
    batch_size: int
    fanout: tuple
    cache_bytes: int
    ring_bytes: int
    lookahead: int
    rmat: tuple = (0.57, 0.19, 0.19)
    seed: int = 0

    @property
    def num_types(self) -> int:
        return len(self.dims)

    def type_counts(self) -> list:
        c = [int(round(f * self.num_nodes)) for f in self.type_share[:-1]]
        return c + [self.num_nodes - sum(c)]

    def row_bytes(self, t: int) -> int:
        return self.dims[t] * self.elt_bytes

    def store_bytes(self, t: int) -> int:
        return self.type_counts()[t] * self.row_bytes(t)

    def cache_shape(self, t: int) -> CacheShape:
        total = sum(self.store_bytes(k) for k in range(self.num_types))
        share = self.store_bytes(t) / total
        return CacheShape(num_sets=int(self.cache_bytes * share) // self.row_bytes(t) // 8,
                          victim_rows=int(self.ring_bytes * share) // self.row_bytes(t),
                          lookahead=self.lookahead)

    def describe(self) -> dict:
        return {
            "workload": self.name,
            "num_nodes": self.num_nodes,
            "num_edges": self.num_edges,
            "types": [{"nodes": n, "feature": f"fp32x{d}" if self.elt_bytes == 4 else f"fp16x{d}",
                       "row_bytes": self.row_bytes(t), "num_sets": self.cache_shape(t).num_sets,
                       "victim_rows": self.cache_shape(t).victim_rows}
                      for t, (n, d) in enumerate(zip(self.type_counts(), self.dims))],
            "batch_size": self.batch_size,
            "fanout": list(self.fanout),
            "ways": 8,
            "lookahead": self.lookahead,
        }


# The heterogeneous workload shape: 4 node types (40/30/20/10 %), fp32 widths
# 1024/768/256/128, caches totalling 32 GiB of HBM, rings totalling 16 GiB.
HETERO = {
    TYPED20M: HeteroConfig(TYPED20M, 20_000_000, 250_000_000, (0.4, 0.3, 0.2, 0.1), (1024, 768, 256, 128), 4,
                    500, 8192, (10, 5, 5), 32 * GIB, 16 * GIB, 8),
}

# every workload, smallest to largest
WORKLOADS = {n: {**CONFIGS, **HETERO}[n] for n in (RMAT14, RMAT20, RMAT10M, TYPED20M, RMAT100M)}

# key offset of the node-type permutation (distinct from the seed-node permutation)
TYPE_PERM_SEED = 0x54595045


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O3", "-std=c11", "-ffp-contract=off", "-fno-math-errno", "-fopenmp", "-fPIC", "-shared", "-Wall",
           os.path.join(HERE, "gen.c"), "-o", LIB_PATH + ".tmp", "-lm"]
    subprocess.run(cmd, check=True, capture_output=not verbose)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            build()
        L = ctypes.CDLL(LIB_PATH)
        u64, i32, vp, f64 = ctypes.c_uint64, ctypes.c_int, ctypes.c_void_p, ctypes.c_double
        L.wl_splitmix_at.restype = u64
        L.wl_splitmix_at.argtypes = [u64, u64]
        L.wl_rmat_csr.restype = i32
        L.wl_rmat_csr.argtypes = [u64, u64, f64, f64, f64, u64, vp, vp, vp]
        L.wl_perm_prefix.restype = i32
        L.wl_perm_prefix.argtypes = [u64, u64, u64, vp]
        L.wl_sample.restype = i32
        L.wl_sample.argtypes = [vp, vp, vp, u64, vp, i32, u64, u64, u64, vp, vp]
        L.wl_features.restype = None
        L.wl_features.argtypes = [u64, i32, u64, u64, u64, vp]
        _lib = L
    return _lib


def splitmix_at(key: int, k: int) -> int:
    return int(lib().wl_splitmix_at(key, k))


class Graph:
    def __init__(self, offsets, adj, indeg):
        self.offsets, self.adj, self.indeg = offsets, adj, indeg

    @property
    def num_nodes(self):
        return self.offsets.size - 1


def rmat_graph(num_nodes: int, num_edges: int, abc=(0.57, 0.19, 0.19), seed: int = 0) -> Graph:
    offsets = np.empty(num_nodes + 1, np.int64)
    adj = np.empty(max(num_edges, 1), np.uint32)
    indeg = np.empty(num_nodes, np.uint32)
    rc = lib().wl_rmat_csr(num_nodes, num_edges, abc[0], abc[1], abc[2], seed,
                           offsets.ctypes.data, adj.ctypes.data, indeg.ctypes.data)
    if rc:
        raise MemoryError("wl_rmat_csr failed")
    return Graph(offsets, adj[:num_edges], indeg)


def seed_permutation(num_nodes: int, count: int, seed: int = 0) -> np.ndarray:
    out = np.empty(max(count, 1), np.int64)
    rc = lib().wl_perm_prefix(num_nodes, count, seed, out.ctypes.data)
    if rc:
        raise MemoryError("wl_perm_prefix failed")
    return out[:count]


def sample_batches(graph: Graph, seeds: np.ndarray, batch_size: int, fanout, b0: int, b1: int,
                   seed: int = 0):
    """Raw request lists of minibatches [b0, b1): (ids int64 concatenated,
    offsets int64 of length b1-b0+1)."""
    assert seeds.size >= b1 * batch_size
    fan = np.ascontiguousarray(fanout, dtype=np.uint32)
    lens = np.empty(b1 - b0, np.uint64)
    L = lib()
    args = (graph.offsets.ctypes.data, graph.adj.ctypes.data, seeds.ctypes.data, batch_size,
            fan.ctypes.data, fan.size, seed, b0, b1, lens.ctypes.data)
    rc = L.wl_sample(*args, None)
    if rc:
        raise RuntimeError(f"wl_sample failed ({rc})")
    offs = np.zeros(b1 - b0 + 1, np.int64)
    np.cumsum(lens.astype(np.int64), out=offs[1:])
    ids = np.empty(max(int(offs[-1]), 1), np.int64)
    rc = L.wl_sample(*args, ids.ctypes.data)
    if rc:
        raise RuntimeError(f"wl_sample failed ({rc})")
    return ids[: offs[-1]], offs


def fill_features(out_ptr: int, dim: int, elt_bytes: int, v0: int, v1: int, seed: int = 0) -> None:
    """Write rows [v0, v1) of the N(0,1) feature table to host memory at out_ptr."""
    lib().wl_features(dim, elt_bytes, seed, v0, v1, out_ptr)


def features(num_nodes: int, dim: int, elt_bytes: int = 4, seed: int = 0) -> np.ndarray:
    a = np.empty((num_nodes, dim), np.float32 if elt_bytes == 4 else np.float16)
    fill_features(a.ctypes.data, dim, elt_bytes, 0, num_nodes, seed)
    return a


class Workload:
    """Graph + request streams for one config (features are filled separately,
    usually straight into pinned host memory)."""

    def __init__(self, cfg: WorkloadConfig, batches: int | None = None):
        self.cfg = cfg
        self.num_batches = cfg.batches if batches is None else batches
        self.graph = rmat_graph(cfg.num_nodes, cfg.num_edges, cfg.rmat, cfg.seed)
        self.static = self.graph.indeg
        self.seeds = seed_permutation(cfg.num_nodes, self.num_batches * cfg.batch_size, cfg.seed)
        self.ids, self.offsets = sample_batches(self.graph, self.seeds, cfg.batch_size, cfg.fanout,
                                                0, self.num_batches, cfg.seed)

    def batch(self, b: int) -> np.ndarray:
        return self.ids[self.offsets[b]: self.offsets[b + 1]]

    @property
    def max_batch(self) -> int:
        return int(np.diff(self.offsets).max()) if self.num_batches else 0


class HeteroWorkload:
    """Graph + request streams of a typed workload, split by node type.  The
    raw request list of a minibatch (global IDs, as the sampler produced them)
    is split into one list per type, in request order, of local IDs."""

    def __init__(self, cfg: HeteroConfig, batches: int | None = None):
        self.cfg = cfg
        self.num_batches = cfg.batches if batches is None else batches
        N = cfg.num_nodes
        self.graph = rmat_graph(N, cfg.num_edges, cfg.rmat, cfg.seed)
        self.seeds = seed_permutation(N, self.num_batches * cfg.batch_size, cfg.seed)
        self.ids, self.offsets = sample_batches(self.graph, self.seeds, cfg.batch_size, cfg.fanout,
                                                0, self.num_batches, cfg.seed)
        perm = seed_permutation(N, N, cfg.seed + TYPE_PERM_SEED)
        counts = cfg.type_counts()
        self.type_offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
        self.node_type = np.empty(N, np.uint8)
        self.node_local = np.empty(N, np.int64)
        self.static = []
        for t in range(cfg.num_types):
            nodes = perm[self.type_offsets[t]: self.type_offsets[t + 1]]
            self.node_type[nodes] = t
            self.node_local[nodes] = np.arange(nodes.size, dtype=np.int64)
            self.static.append(np.ascontiguousarray(self.graph.indeg[nodes]))
        del perm
        self._split = {}

    def batch(self, b: int, t: int) -> np.ndarray:
        """Local IDs of type t in minibatch b, in request order."""
        if b not in self._split:
            g = self.ids[self.offsets[b]: self.offsets[b + 1]]
            ty = self.node_type[g]
            loc = self.node_local[g]
            self._split = {b: [loc[ty == k] for k in range(self.cfg.num_types)]}
        return self._split[b][t]

    def type_batches(self, t: int) -> list:
        out = []
        for b in range(self.num_batches):
            g = self.ids[self.offsets[b]: self.offsets[b + 1]]
            out.append(self.node_local[g][self.node_type[g] == t])
        return out


# Pinned host memory a process may hold is limited (64 GiB on the MI355X hosts
# measured); the victim rings, the pinned stores and the bounce buffers of
# pageable stores must fit together.
PINNED_BUDGET = 52 * GIB


def pin_plan(store_bytes, ring_bytes_total, budget=PINNED_BUDGET):
    """Which stores to keep in pinned memory: the largest first, while the
    rings and the pinned stores fit the budget; the rest stay pageable."""
    pinned = [False] * len(store_bytes)
    used = ring_bytes_total
    for i in sorted(range(len(store_bytes)), key=lambda k: -store_bytes[k]):
        if used + store_bytes[i] <= budget:
            pinned[i] = True
            used += store_bytes[i]
    return pinned


def scaled_cache(cfg: WorkloadConfig) -> CacheShape:
    return cfg.cache


def near_threshold_default(lookahead: int) -> int:
    return max(1, lookahead // 8)


__all__ = ["RMAT14", "RMAT20", "RMAT10M", "TYPED20M", "RMAT100M", "WORKLOADS", "CONFIGS", "HETERO", "HeteroConfig", "HeteroWorkload", "WorkloadConfig", "CacheShape", "Workload", "Graph", "rmat_graph",
           "seed_permutation", "sample_batches", "features", "fill_features", "build", "splitmix_at",
           "near_threshold_default", "pin_plan", "PINNED_BUDGET", "math"]
