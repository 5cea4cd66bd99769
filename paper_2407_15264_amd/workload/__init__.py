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


# The homogeneous workload shapes.  Cache/ring budgets in GiB; cache sets are
# the budget in rows divided by the 8 ways.
CONFIGS = {
    1: WorkloadConfig("rmat-s14-e18-f32x128", 1 << 14, 1 << 18, 128, 4, 20, 256, (10, 5),
                      CacheShape(num_sets=2048, victim_rows=1024, lookahead=2)),
    2: WorkloadConfig("rmat-s20-deg16-f32x256", 1 << 20, 1 << 24, 256, 4, 200, 1024, (15, 10, 5),
                      CacheShape(num_sets=int(0.10 * (1 << 20)) // 8, victim_rows=int(0.05 * (1 << 20)),
                                 lookahead=4)),
    3: WorkloadConfig("rmat-10M-e120M-f32x1024", 10_000_000, 120_000_000, 1024, 4, 500, 4096, (10, 5, 5),
                      CacheShape(num_sets=_cache_lines_for(8 * GIB, 4096) // 8,
                                 victim_rows=_cache_lines_for(4 * GIB, 4096), lookahead=8)),
    5: WorkloadConfig("rmat-100M-e1.6B-f16x1024", 100_000_000, 1_600_000_000, 1024, 2, 1000, 8192, (15, 10, 5),
                      CacheShape(num_sets=_cache_lines_for(96 * GIB, 2048) // 8,
                                 victim_rows=_cache_lines_for(32 * GIB, 2048), lookahead=16)),
}


def build(verbose: bool = False) -> str:
    cmd = ["gcc", "-O3", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall",
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


def scaled_cache(cfg: WorkloadConfig) -> CacheShape:
    return cfg.cache


def near_threshold_default(lookahead: int) -> int:
    return max(1, lookahead // 8)


__all__ = ["CONFIGS", "WorkloadConfig", "CacheShape", "Workload", "Graph", "rmat_graph",
           "seed_permutation", "sample_batches", "features", "fill_features", "build", "splitmix_at",
           "near_threshold_default", "math"]
