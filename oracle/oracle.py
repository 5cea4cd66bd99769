"""CPU oracle binding -- TEST INFRASTRUCTURE ONLY.

ctypes wrapper around ``liboracle.so`` (built from ``oracle.c`` with gcc).  Only
the tests, the smoke check and the benchmark's CPU-baseline leg import this
module; the GPU library never does.  See ``oracle.c`` for the definition and
the paper passages each step follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "liboracle.so")

HIT, VICTIM_HIT, MISS = 0, 1, 2
STATUS = {0: "OK", 1: "E_INVAL", 2: "E_RANGE", 3: "E_WINDOW", 4: "E_NOMEM"}
STAT_FIELDS = ("batch", "requests", "unique", "hits", "victim_hits", "misses",
               "evictions", "enqueued", "dropped", "request_hits", "request_victim_hits")


class OracleError(RuntimeError):
    def __init__(self, code: int, where: str):
        super().__init__(f"{where}: {STATUS.get(code, code)}")
        self.code = code
        self.status = STATUS.get(code, str(code))


class _Stats(ctypes.Structure):
    _fields_ = [(f, ctypes.c_uint64) for f in STAT_FIELDS]


def build(verbose: bool = False) -> str:
    """Compile liboracle.so (plain C, -O2, single-threaded)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-Wall", "-Wextra",
           os.path.join(HERE, "oracle.c"), os.path.join(HERE, "pagerank.c"), "-lm", "-o", LIB_PATH + ".tmp"]
    subprocess.run(cmd, check=True, capture_output=not verbose)
    os.replace(LIB_PATH + ".tmp", LIB_PATH)
    return LIB_PATH


def stale() -> bool:
    """True when liboracle.so is missing or older than its sources."""
    if not os.path.exists(LIB_PATH):
        return True
    built = os.path.getmtime(LIB_PATH)
    return any(os.path.getmtime(os.path.join(HERE, f)) > built for f in ("oracle.c", "pagerank.c", "oracle.h"))


_lib = None


def lib():
    global _lib
    if _lib is None:
        if stale():
            build()
        L = ctypes.CDLL(LIB_PATH)
        u64, u32, i32, vp = ctypes.c_uint64, ctypes.c_uint32, ctypes.c_int, ctypes.c_void_p
        L.orc_set_of.restype = u64
        L.orc_set_of.argtypes = [u64, u64]
        L.orc_create.restype = i32
        L.orc_create.argtypes = [u64, u32, vp, vp, u64, u32, u64, u32, u32, u32, u32, u32, ctypes.POINTER(vp)]
        L.orc_pagerank.restype = i32
        L.orc_pagerank.argtypes = [u64, vp, vp, ctypes.c_double, u32, vp]
        L.orc_rank_scores.restype = i32
        L.orc_rank_scores.argtypes = [u64, vp, vp]
        L.orc_destroy.restype = None
        L.orc_destroy.argtypes = [vp]
        L.orc_advance.restype = i32
        L.orc_advance.argtypes = [vp, vp, u64]
        L.orc_gather.restype = i32
        L.orc_gather.argtypes = [vp, vp, u64, vp, vp, vp, vp, ctypes.POINTER(u64)]
        L.orc_stats.restype = i32
        L.orc_stats.argtypes = [vp, ctypes.POINTER(_Stats), ctypes.POINTER(_Stats)]
        L.orc_export_state.restype = i32
        L.orc_export_state.argtypes = [vp, vp, vp, ctypes.POINTER(u64), ctypes.POINTER(u64)]
        L.orc_near_threshold.restype = u32
        L.orc_near_threshold.argtypes = [vp]
        _lib = L
    return _lib


def set_of(x: int, num_sets: int) -> int:
    return int(lib().orc_set_of(int(x), int(num_sets)))


def _ptr(a):
    return None if a is None else a.ctypes.data


# eviction policies of the paper's evaluation (Sec. 5): hybrid (Sec. 4.2),
# static information only, dynamic information only, round-robin
POLICIES = {"hybrid": 0, "static": 1, "dynamic": 2, "round_robin": 3}
# victim buffer forms: one FIFO ring, or per-reuse-iteration queues (Sec. 4.3.1)
VICTIM_MODES = {"fifo": 0, "queues": 1}


class Oracle:
    """Sequential reference cache.  ``store`` is a (num_nodes, row_bytes) uint8
    view of the backing feature table, or None for metadata-only runs.
    ``policy`` is a name in POLICIES (or its number)."""

    def __init__(self, num_nodes, row_bytes, static_score, num_sets, victim_rows,
                 lookahead, near_threshold=0, ways=8, store=None, policy="hybrid", victim_mode="fifo",
                 refresh_period=1):
        self.num_nodes = int(num_nodes)
        self.row_bytes = int(row_bytes)
        self.num_sets = int(num_sets)
        self.ways = int(ways)
        self.victim_rows = int(victim_rows)
        self.static = np.ascontiguousarray(static_score, dtype=np.uint32)
        self.store = None
        if store is not None:
            self.store = np.ascontiguousarray(store).view(np.uint8).reshape(self.num_nodes, self.row_bytes)
        h = ctypes.c_void_p()
        rc = lib().orc_create(self.num_nodes, self.row_bytes, _ptr(self.store), _ptr(self.static),
                              self.num_sets, self.ways, self.victim_rows, int(lookahead),
                              int(near_threshold), POLICIES.get(policy, policy),
                              VICTIM_MODES.get(victim_mode, victim_mode), int(refresh_period), ctypes.byref(h))
        if rc:
            raise OracleError(rc, "orc_create")
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            lib().orc_destroy(self._h)
            self._h = None

    __del__ = close

    @property
    def near_threshold(self) -> int:
        return int(lib().orc_near_threshold(self._h))

    def advance(self, ids):
        ids = np.ascontiguousarray(ids, dtype=np.int64)
        rc = lib().orc_advance(self._h, _ptr(ids), ids.size)
        if rc:
            raise OracleError(rc, "orc_advance")

    def gather(self, ids, rows: bool = True, out=None):
        """Returns dict(uniq, inv, outcome, out, stats).  `out`: optional
        caller buffer for the rows (a C-contiguous uint8 array of at least
        len(ids) * row_bytes bytes), used instead of a new array."""
        ids = np.ascontiguousarray(ids, dtype=np.int64)
        n = ids.size
        uniq = np.empty(max(n, 1), np.int64)
        inv = np.empty(max(n, 1), np.int64)
        outcome = np.empty(max(n, 1), np.uint8)
        if not (rows and self.store is not None):
            out = None
        elif out is None:
            out = np.empty((max(n, 1), self.row_bytes), np.uint8)
        else:
            if out.dtype != np.uint8 or not out.flags.c_contiguous or out.size < n * self.row_bytes:
                raise ValueError("out must be a C-contiguous uint8 array of at least n * row_bytes bytes")
            out = out.reshape(-1)[: max(n, 1) * self.row_bytes].reshape(max(n, 1), self.row_bytes)
        nu = ctypes.c_uint64()
        rc = lib().orc_gather(self._h, _ptr(ids), n, _ptr(out), _ptr(uniq), _ptr(inv),
                              _ptr(outcome), ctypes.byref(nu))
        if rc:
            raise OracleError(rc, "orc_gather")
        U = nu.value
        return dict(uniq=uniq[:U], inv=inv[:n], outcome=outcome[:U],
                    out=None if out is None else out[:U], stats=self.stats()[0])

    def stats(self):
        last, total = _Stats(), _Stats()
        rc = lib().orc_stats(self._h, ctypes.byref(last), ctypes.byref(total))
        if rc:
            raise OracleError(rc, "orc_stats")
        return ({f: getattr(last, f) for f in STAT_FIELDS},
                {f: getattr(total, f) for f in STAT_FIELDS})

    def export_state(self):
        tags = np.empty(self.num_sets * self.ways, np.uint32)
        ring = np.empty(max(self.victim_rows, 1), np.uint32)
        tail, t = ctypes.c_uint64(), ctypes.c_uint64()
        rc = lib().orc_export_state(self._h, _ptr(tags), _ptr(ring), ctypes.byref(tail), ctypes.byref(t))
        if rc:
            raise OracleError(rc, "orc_export_state")
        return dict(tags=tags.reshape(self.num_sets, self.ways),
                    ring_tags=ring[:self.victim_rows], ring_tail=tail.value, t=t.value)


def pagerank(offsets, adj, damping=0.85, iterations=20):
    """Reverse-PageRank ranks (float64, one per node) of a CSR graph whose node u
    lists the neighbours it samples; see pagerank.c for the definition."""
    offsets = np.ascontiguousarray(offsets, np.int64)
    adj = np.ascontiguousarray(adj, np.uint32)
    n = offsets.size - 1
    rank = np.empty(max(n, 1), np.float64)
    rc = lib().orc_pagerank(n, _ptr(offsets), _ptr(adj) if adj.size else None, float(damping), int(iterations),
                            _ptr(rank))
    if rc:
        raise OracleError(rc, "orc_pagerank")
    return rank[:n]


def rank_scores(rank):
    """32-bit static scores: floor(rank / max rank * (2^32 - 1))."""
    rank = np.ascontiguousarray(rank, np.float64)
    out = np.empty(max(rank.size, 1), np.uint32)
    rc = lib().orc_rank_scores(rank.size, _ptr(rank), _ptr(out))
    if rc:
        raise OracleError(rc, "orc_rank_scores")
    return out[:rank.size]
