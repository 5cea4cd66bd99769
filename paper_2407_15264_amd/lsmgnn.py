"""Python binding of the MI355X feature-gather cache (C ABI in include/lsmgnn.h).

Argument marshalling only: every step of a gather runs in the gfx950 kernels of
liblsmgnn.so.  PyTorch supplies device memory (tensors) and the stream.  There
is no CPU fallback: if the library is missing this module raises.
"""
from __future__ import annotations

import atexit
import ctypes
import os
import weakref

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "liblsmgnn.so")

OK, E_INVAL, E_RANGE, E_WINDOW, E_NOMEM, E_DEVICE, E_STATE = range(7)
STATUS_NAMES = {0: "OK", 1: "E_INVAL", 2: "E_RANGE", 3: "E_WINDOW", 4: "E_NOMEM", 5: "E_DEVICE", 6: "E_STATE"}
HIT, VICTIM_HIT, MISS = 0, 1, 2
EMPTY = 0xFFFFFFFF
COUNT_FIELDS = ("batch", "requests", "unique", "hits", "victim_hits", "misses", "evictions", "enqueued",
                "dropped", "request_hits", "request_victim_hits", "victim_rows_ring", "victim_rows_staged",
                "victim_rows_cache", "victim_rows_prefetched")


class LsmgnnError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        self.status = STATUS_NAMES.get(code, str(code))
        msg = lib().lsmgnn_strerror(code).decode() if _lib is not None else self.status
        super().__init__(f"{where}: {self.status} ({msg})")


class Config(ctypes.Structure):
    _fields_ = [("num_nodes", ctypes.c_uint64), ("row_bytes", ctypes.c_uint64), ("num_sets", ctypes.c_uint64),
                ("victim_rows", ctypes.c_uint64), ("max_batch", ctypes.c_uint64), ("lookahead", ctypes.c_uint32),
                ("near_threshold", ctypes.c_uint32), ("device", ctypes.c_int32), ("flags", ctypes.c_uint32),
                ("host_threads", ctypes.c_uint32), ("policy", ctypes.c_uint32), ("victim_mode", ctypes.c_uint32),
                ("refresh_period", ctypes.c_uint32), ("host_store", ctypes.c_void_p),
                ("static_score", ctypes.c_void_p)]


FLAG_PAGEABLE_STORE = 1
# lsmgnn_config.policy values: the method's hybrid order and the evaluation's
# alternatives (static score only, next announced use only, round-robin)
POLICY = {"hybrid": 0, "static": 1, "dynamic": 2, "round_robin": 3}
# lsmgnn_config.victim_mode values: one FIFO ring, or per-reuse-iteration
# queues prefetched into HBM before their iteration
VICTIM_MODE = {"fifo": 0, "queues": 1}


class Counts(ctypes.Structure):
    _fields_ = [(f, ctypes.c_uint64) for f in COUNT_FIELDS]


class Profile(ctypes.Structure):
    _fields_ = [("hbm_copy_ms", ctypes.c_double), ("hbm_copy_launches", ctypes.c_uint64),
                ("hbm_copy_rows", ctypes.c_uint64),
                ("host_fetch_ms", ctypes.c_double), ("host_fetch_launches", ctypes.c_uint64),
                ("host_fetch_rows", ctypes.c_uint64),
                ("enqueue_ms", ctypes.c_double), ("enqueue_launches", ctypes.c_uint64),
                ("enqueue_rows", ctypes.c_uint64),
                ("fill_ms", ctypes.c_double), ("fill_launches", ctypes.c_uint64), ("fill_rows", ctypes.c_uint64),
                ("host_copy_ms", ctypes.c_double), ("host_copy_rows", ctypes.c_uint64),
                ("prefetch_ms", ctypes.c_double), ("prefetch_launches", ctypes.c_uint64),
                ("prefetch_rows", ctypes.c_uint64),
                ("gather_ms", ctypes.c_double), ("gathers", ctypes.c_uint64)]


_lib = None

# Library objects still open, closed at interpreter exit before module
# teardown begins: caches first (their host threads read the stores and their
# streams may still move rows), then samplers, then pinned buffers.  A
# finalizer that ran during teardown would find the module's globals gone.
_LIVE = {"cache": weakref.WeakSet(), "sampler": weakref.WeakSet(), "pinned": weakref.WeakSet()}


def _close_all():
    for kind in ("cache", "sampler", "pinned"):
        for obj in list(_LIVE[kind]):
            obj.close()


atexit.register(_close_all)


def lib():
    """Load liblsmgnn.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(hipcc --offload-arch=gfx950); there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        vp, u64, i32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int
        L.lsmgnn_cache_create.restype = i32
        L.lsmgnn_cache_create.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(vp)]
        L.lsmgnn_cache_destroy.restype = None
        L.lsmgnn_cache_destroy.argtypes = [vp]
        L.lsmgnn_advance.restype = i32
        L.lsmgnn_advance.argtypes = [vp, vp, u64, vp]
        L.lsmgnn_gather.restype = i32
        L.lsmgnn_gather.argtypes = [vp, vp, u64, vp, vp, vp, vp, ctypes.POINTER(u64), vp]
        L.lsmgnn_gather_async.restype = i32
        L.lsmgnn_gather_async.argtypes = [vp, vp, u64, vp, u64, vp, vp, vp, vp, ctypes.POINTER(u64),
                                          ctypes.POINTER(u64), vp]
        L.lsmgnn_gather_wait.restype = i32
        L.lsmgnn_gather_wait.argtypes = [vp, u64, vp]
        L.lsmgnn_sync.restype = i32
        L.lsmgnn_sync.argtypes = [vp]
        L.lsmgnn_stats.restype = i32
        L.lsmgnn_stats.argtypes = [vp, ctypes.POINTER(Counts), ctypes.POINTER(Counts)]
        L.lsmgnn_export_state.restype = i32
        L.lsmgnn_export_state.argtypes = [vp, vp, vp, ctypes.POINTER(u64), ctypes.POINTER(u64)]
        L.lsmgnn_set_profiling.restype = i32
        L.lsmgnn_set_profiling.argtypes = [vp, i32]
        L.lsmgnn_get_profile.restype = i32
        L.lsmgnn_get_profile.argtypes = [vp, ctypes.POINTER(Profile)]
        L.lsmgnn_host_alloc.restype = i32
        L.lsmgnn_host_alloc.argtypes = [u64, ctypes.POINTER(vp)]
        L.lsmgnn_host_free.restype = None
        L.lsmgnn_host_free.argtypes = [vp]
        L.lsmgnn_set_of.restype = u64
        L.lsmgnn_set_of.argtypes = [u64, u64]
        L.lsmgnn_copy_bytes.restype = i32
        L.lsmgnn_copy_bytes.argtypes = [vp, vp, u64, vp]
        L.lsmgnn_pagerank_scores.restype = i32
        L.lsmgnn_pagerank_scores.argtypes = [vp, vp, u64, ctypes.c_double, ctypes.c_uint32, vp, vp, i32, vp]
        L.lsmgnn_expand.restype = i32
        L.lsmgnn_expand.argtypes = [vp, vp, u64, u64, vp, vp]
        L.lsmgnn_sampler_create.restype = i32
        L.lsmgnn_sampler_create.argtypes = [vp, vp, u64, vp, ctypes.c_uint32, u64, i32, ctypes.POINTER(vp)]
        L.lsmgnn_sampler_destroy.restype = None
        L.lsmgnn_sampler_destroy.argtypes = [vp]
        L.lsmgnn_sample.restype = i32
        L.lsmgnn_sample.argtypes = [vp, vp, u64, u64, vp, u64, ctypes.POINTER(u64), vp]
        L.lsmgnn_sample_async.restype = i32
        L.lsmgnn_sample_async.argtypes = [vp, vp, u64, u64, vp, u64, vp, vp]
        L.lsmgnn_split_work_bytes.restype = u64
        L.lsmgnn_split_work_bytes.argtypes = [u64, ctypes.c_uint32]
        L.lsmgnn_split_by_type_async.restype = i32
        L.lsmgnn_split_by_type_async.argtypes = [vp, u64, u64, vp, vp, ctypes.c_uint32, ctypes.POINTER(vp), u64,
                                                 vp, u64, vp, vp]
        L.lsmgnn_split_by_type_noalloc_async.restype = i32
        L.lsmgnn_split_by_type_noalloc_async.argtypes = [vp, u64, u64, vp, vp, ctypes.c_uint32, ctypes.POINTER(vp),
                                                         u64, vp, vp]
        L.lsmgnn_strerror.restype = ctypes.c_char_p
        L.lsmgnn_strerror.argtypes = [i32]
        _lib = L
    return _lib


def _check(rc: int, where: str):
    if rc != OK:
        raise LsmgnnError(rc, where)


def set_of(x: int, num_sets: int) -> int:
    return int(lib().lsmgnn_set_of(int(x), int(num_sets)))


def copy_bytes(dst_ptr: int, src_ptr: int, nbytes: int, stream=None, device=0):
    """Calibration copy (device or pinned host pointers), synchronous."""
    _check(lib().lsmgnn_copy_bytes(ctypes.c_void_p(dst_ptr), ctypes.c_void_p(src_ptr), int(nbytes),
                                   _stream_handle(stream, device)), "lsmgnn_copy_bytes")


def expand(rows, inverse, row_bytes, out=None, stream=None, device=0):
    """Rows in request order (lsmgnn_expand): out[i] = rows[inverse[i]].  rows:
    a gather's unique-row output (uint8 device tensor), inverse: its int64
    inverse index (n entries).  Returns `out` (uint8, n * row_bytes), allocated
    when not given."""
    import torch
    n = inverse.numel()
    if out is None:
        out = torch.empty(max(n, 1) * row_bytes, dtype=torch.uint8, device=inverse.device)
    _check(lib().lsmgnn_expand(ctypes.c_void_p(rows.data_ptr()), ctypes.c_void_p(inverse.data_ptr()), n,
                               int(row_bytes), ctypes.c_void_p(out.data_ptr()), _stream_handle(stream, device)),
           "lsmgnn_expand")
    return out[: n * row_bytes]


def pagerank_scores(offsets, adj, damping=0.85, iterations=20, rank=False, device=0, stream=None):
    """Reverse-PageRank static scores (lsmgnn_pagerank_scores) of a CSR graph
    given as device tensors (offsets int64 [N+1], adj int32/uint32 [E]).
    Returns a device uint32-valued int32 tensor of scores (viewed as uint32 by
    callers through .cpu().numpy().view(np.uint32)), and the float64 ranks
    when rank=True."""
    import torch
    dev = torch.device("cuda", device)
    n = offsets.numel() - 1
    scores = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
    rk = torch.empty(max(n, 1), dtype=torch.float64, device=dev) if rank else None
    _check(lib().lsmgnn_pagerank_scores(ctypes.c_void_p(offsets.data_ptr()),
                                        ctypes.c_void_p(adj.data_ptr()) if adj.numel() else None, n,
                                        float(damping), int(iterations), ctypes.c_void_p(scores.data_ptr()),
                                        ctypes.c_void_p(rk.data_ptr()) if rank else None, int(device),
                                        _stream_handle(stream, device)), "lsmgnn_pagerank_scores")
    return (scores[:n], rk[:n]) if rank else scores[:n]


class GpuSampler:
    """GraphSAGE request lists sampled on the GPU (lsmgnn_sampler_create /
    lsmgnn_sample) from a CSR graph in device memory (offsets int64 [N+1],
    adj int32/uint32 [E]); the tensors must outlive the sampler."""

    def __init__(self, offsets, adj, fanout, seed=0, device=0):
        import torch
        self.device = torch.device("cuda", device)
        off_p = _dev_ptr(offsets, torch.int64, "offsets")
        adj_p = _dev_ptr(adj, (torch.int32, torch.uint32), "adj") if adj.numel() else None
        self._graph = (offsets, adj)  # keeps the borrowed graph alive
        self.num_nodes = offsets.numel() - 1
        fan = (ctypes.c_uint32 * len(fanout))(*[int(f) for f in fanout])
        self.hops = len(fanout)
        h = ctypes.c_void_p()
        _check(lib().lsmgnn_sampler_create(off_p, adj_p, self.num_nodes, fan, self.hops, int(seed), int(device),
                                           ctypes.byref(h)), "lsmgnn_sampler_create")
        self._destroy = lib().lsmgnn_sampler_destroy  # kept: module globals may be gone when the finalizer runs
        self._h = h
        _LIVE["sampler"].add(self)

    def close(self):
        if getattr(self, "_h", None):
            self._destroy(self._h)
            self._h = None

    __del__ = close

    def sample(self, seeds, batch, out, stream=None):
        """Request list of minibatch `batch` from its seeds (int64 device
        tensor) into `out` (int64 device tensor); returns out[:length]."""
        import torch
        sp = _dev_ptr(seeds, torch.int64, "seeds") if seeds.numel() else None
        op = _dev_ptr(out, torch.int64, "out")
        n = ctypes.c_uint64(0)
        _check(lib().lsmgnn_sample(self._h, sp, seeds.numel(), int(batch), op, out.numel(), ctypes.byref(n),
                                   _stream_handle(stream, self.device.index)), "lsmgnn_sample")
        return out[: n.value]

    def sample_async(self, seeds, batch, out, result_ptr, stream=None):
        """Queue the sampling of minibatch `batch` into `out`; once `stream`
        has run it, the two uint64 at result_ptr (pinned host memory) hold
        the list's length and its status code."""
        import torch
        sp = _dev_ptr(seeds, torch.int64, "seeds") if seeds.numel() else None
        op = _dev_ptr(out, torch.int64, "out")
        _check(lib().lsmgnn_sample_async(self._h, sp, seeds.numel(), int(batch), op, out.numel(),
                                         ctypes.c_void_p(result_ptr), _stream_handle(stream, self.device.index)),
               "lsmgnn_sample_async")


def split_work_bytes(n, num_types):
    """Device work memory split_by_type_async needs for n requests."""
    return int(lib().lsmgnn_split_work_bytes(int(n), int(num_types)))


def split_by_type_async(ids, node_type, local, outs, work, result_ptr, stream=None, device=0):
    """Queue the split of a global request list (int64 device tensor) into one
    list of within-type indices per node type (lsmgnn_split_by_type_async):
    node_type (uint8 device tensor), local (int32/uint32 device tensor), outs
    (int64 device tensors of equal length, one per type), work (a device
    tensor of at least split_work_bytes bytes); result_ptr: pinned host
    memory for the len(outs) lengths and the status."""
    import torch
    T = len(outs)
    if T == 0:
        raise ValueError("outs must hold one tensor per node type")
    ids_p = _dev_ptr(ids, torch.int64, "ids") if ids.numel() else None
    type_p = _dev_ptr(node_type, torch.uint8, "node_type")
    local_p = _dev_ptr(local, (torch.int32, torch.uint32), "local")
    if local.numel() != node_type.numel():
        raise ValueError("local and node_type must have one entry per node")
    ptrs = (ctypes.c_void_p * T)(*[_dev_ptr(o, torch.int64, f"outs[{t}]").value for t, o in enumerate(outs)])
    cap = min(o.numel() for o in outs)  # every list may be written up to the capacity
    work_p = _dev_ptr(work, work.dtype, "work")
    _check(lib().lsmgnn_split_by_type_async(ids_p, ids.numel(), node_type.numel(), type_p, local_p, T, ptrs, cap,
                                            work_p, work.numel() * work.element_size(),
                                            ctypes.c_void_p(result_ptr), _stream_handle(stream, device)),
           "lsmgnn_split_by_type_async")


def split_by_type_noalloc_async(ids, node_type, local, outs, result_ptr, stream=None, device=0):
    """split_by_type_async without the work tensor
    (lsmgnn_split_by_type_noalloc_async): the library's own device array is
    the work memory, so the call allocates nothing; calls that may overlap on
    one device must be ordered by the caller."""
    import torch
    T = len(outs)
    if T == 0:
        raise ValueError("outs must hold one tensor per node type")
    ids_p = _dev_ptr(ids, torch.int64, "ids") if ids.numel() else None
    type_p = _dev_ptr(node_type, torch.uint8, "node_type")
    local_p = _dev_ptr(local, (torch.int32, torch.uint32), "local")
    if local.numel() != node_type.numel():
        raise ValueError("local and node_type must have one entry per node")
    ptrs = (ctypes.c_void_p * T)(*[_dev_ptr(o, torch.int64, f"outs[{t}]").value for t, o in enumerate(outs)])
    cap = min(o.numel() for o in outs)
    _check(lib().lsmgnn_split_by_type_noalloc_async(ids_p, ids.numel(), node_type.numel(), type_p, local_p, T, ptrs,
                                                    cap, ctypes.c_void_p(result_ptr), _stream_handle(stream, device)),
           "lsmgnn_split_by_type_noalloc_async")


class PinnedBuffer:
    """Exact-size pinned, device-mapped host memory (lsmgnn_host_alloc)."""

    def __init__(self, nbytes: int):
        p = ctypes.c_void_p()
        _check(lib().lsmgnn_host_alloc(int(nbytes), ctypes.byref(p)), "lsmgnn_host_alloc")
        self.ptr = p.value
        self.nbytes = int(nbytes)
        self._free = lib().lsmgnn_host_free  # kept: module globals may be gone when the finalizer runs
        _LIVE["pinned"].add(self)

    def numpy(self, dtype=np.uint8, shape=None) -> np.ndarray:
        raw = (ctypes.c_uint8 * self.nbytes).from_address(self.ptr)
        a = np.frombuffer(raw, dtype=np.uint8).view(dtype)
        return a if shape is None else a.reshape(shape)

    def close(self):
        if getattr(self, "ptr", None):
            self._free(self.ptr)
            self.ptr = None

    __del__ = close


def _stream_handle(stream, device):
    import torch
    s = torch.cuda.current_stream(device) if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev_ptr(t, dtype, name):
    """Device address of a contiguous tensor of `dtype` (or one of a tuple of
    dtypes); raises TypeError for anything else."""
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    ok = t.dtype in dtype if isinstance(dtype, tuple) else t.dtype == dtype
    if not ok or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous {dtype} tensor")
    return ctypes.c_void_p(t.data_ptr())


class GatherResult:
    """Outputs of one gather as views of the caller's buffers (built on first
    access, so the hot loop pays nothing for them):
    out (n_unique, row_bytes) uint8, unique (n_unique,) int64, inverse (n,)
    int64 or None, outcome (n_unique,) uint8 or None."""

    __slots__ = ("n_unique", "n", "row_bytes", "_out", "_unique", "_inverse", "_outcome")

    def __init__(self, n_unique, n, row_bytes, out, unique, inverse, outcome):
        self.n_unique, self.n, self.row_bytes = n_unique, n, row_bytes
        self._out, self._unique, self._inverse, self._outcome = out, unique, inverse, outcome

    @property
    def out(self):
        import torch
        U = self.n_unique
        return self._out.view(torch.uint8).reshape(-1)[: U * self.row_bytes].view(U, self.row_bytes)

    @property
    def unique(self):
        return self._unique[: self.n_unique]

    @property
    def inverse(self):
        return None if self._inverse is None else self._inverse[: self.n]

    @property
    def outcome(self):
        return None if self._outcome is None else self._outcome[: self.n_unique]


class FeatureCache:
    """GPU feature-gather cache on one device.

    host_store: num_nodes * row_bytes bytes of host memory that must outlive
    the cache: pinned (a PinnedBuffer, its ptr, or a pinned torch tensor), or
    with pageable=True ordinary memory (a numpy array or an address), whose
    rows the library's host threads (host_threads, 0 = 8) copy for the GPU.
    static_score: num_nodes unsigned scores.
    policy: a name in POLICY (or its number); victim_mode: a name in
    VICTIM_MODE (or its number); refresh_period: the update period of the
    dynamic information (1 = exact at every gather)."""

    def __init__(self, num_nodes, row_bytes, host_store, static_score, num_sets, victim_rows, lookahead,
                 max_batch, near_threshold=0, device=0, pageable=False, host_threads=0, policy="hybrid",
                 victim_mode="fifo", refresh_period=1):
        import torch
        self.device = torch.device("cuda", device)
        self.num_nodes, self.row_bytes = int(num_nodes), int(row_bytes)
        self.num_sets, self.victim_rows = int(num_sets), int(victim_rows)
        self.lookahead, self.max_batch = int(lookahead), int(max_batch)
        if isinstance(host_store, PinnedBuffer):
            host_store = host_store.ptr
        elif isinstance(host_store, torch.Tensor):
            host_store = host_store.data_ptr()
        elif isinstance(host_store, np.ndarray):
            if not host_store.flags.c_contiguous or host_store.nbytes < self.num_nodes * self.row_bytes:
                raise ValueError("host_store array must be C-contiguous and hold num_nodes * row_bytes bytes")
            self._store_ref = host_store
            host_store = host_store.ctypes.data
        stat = np.ascontiguousarray(np.asarray(static_score), dtype=np.uint32)
        cfg = Config(self.num_nodes, self.row_bytes, self.num_sets, self.victim_rows, self.max_batch,
                     self.lookahead, int(near_threshold), int(device), FLAG_PAGEABLE_STORE if pageable else 0,
                     int(host_threads), int(POLICY.get(policy, policy)),
                     int(VICTIM_MODE.get(victim_mode, victim_mode)), int(refresh_period),
                     ctypes.c_void_p(int(host_store)),
                     ctypes.c_void_p(stat.ctypes.data))
        h = ctypes.c_void_p()
        _check(lib().lsmgnn_cache_create(ctypes.byref(cfg), ctypes.byref(h)), "lsmgnn_cache_create")
        self._destroy = lib().lsmgnn_cache_destroy  # kept: module globals may be gone when the finalizer runs
        self._h = h
        self._scratch = {}
        _LIVE["cache"].add(self)

    def close(self):
        if getattr(self, "_h", None):
            self._destroy(self._h)
            self._h = None

    __del__ = close

    def _buf(self, name, n, dtype):
        import torch
        b = self._scratch.get(name)
        if b is None or b.numel() < n:
            b = torch.empty(max(n, 1), dtype=dtype, device=self.device)
            self._scratch[name] = b
        return b

    def advance(self, ids, stream=None):
        import torch
        n = ids.numel()
        p = _dev_ptr(ids, torch.int64, "ids") if n else None
        _check(lib().lsmgnn_advance(self._h, p, n, _stream_handle(stream, self.device)), "lsmgnn_advance")

    def _gather_args(self, ids, out, unique, inverse, outcome):
        import torch
        n = ids.numel()
        if out is None:
            out = self._buf("out", n * self.row_bytes, torch.uint8)
        if unique is None:
            unique = self._buf("unique", n, torch.int64)

        def pick(arg, name, dtype):
            if isinstance(arg, torch.Tensor):
                if arg.numel() < n:
                    raise ValueError(f"{name} buffer too small")
                return arg
            return self._buf(name, n, dtype) if arg else None

        inv_t = pick(inverse, "inverse", torch.int64)
        oc_t = pick(outcome, "outcome", torch.uint8)
        if out.numel() * out.element_size() < n * self.row_bytes or unique.numel() < n:
            raise ValueError("out/unique buffers too small")
        args = (self._h, _dev_ptr(ids, torch.int64, "ids") if n else None, n,
                ctypes.c_void_p(out.data_ptr()), _dev_ptr(unique, torch.int64, "unique"),
                _dev_ptr(inv_t, torch.int64, "inverse") if inv_t is not None else None,
                _dev_ptr(oc_t, torch.uint8, "outcome") if oc_t is not None else None)
        return n, out, unique, inv_t, oc_t, args

    def _result(self, U, n, out, unique, inv_t, oc_t):
        return GatherResult(U, n, self.row_bytes, out, unique, inv_t, oc_t)

    def gather(self, ids, out=None, unique=None, inverse=True, outcome=False, stream=None) -> GatherResult:
        """Gather one minibatch (returns when everything is complete).  `out`
        (uint8, >= n*row_bytes bytes) and `unique` (int64, >= n) may be passed
        to reuse caller buffers; `inverse`/`outcome` may be True (allocate), a
        tensor, or False/None."""
        n, out, unique, inv_t, oc_t, args = self._gather_args(ids, out, unique, inverse, outcome)
        nu = ctypes.c_uint64()
        _check(lib().lsmgnn_gather(*args, ctypes.byref(nu), _stream_handle(stream, self.device)), "lsmgnn_gather")
        return self._result(nu.value, n, out, unique, inv_t, oc_t)

    def gather_async(self, ids, out, unique, inverse=None, outcome=None, stream=None, announce=None):
        """Pipelined gather: returns (ticket, GatherResult) once the unique
        count is known.  `announce` (int64 device tensor, or None) is the next
        minibatch to announce after this gather, as advance() would.  The
        buffers must be caller-owned tensors (not reused until wait(ticket) and
        a synchronisation of the stream)."""
        import torch
        n, out, unique, inv_t, oc_t, args = self._gather_args(ids, out, unique, inverse, outcome)
        if announce is None:
            ann = (None, 0)
        else:
            an = announce.numel()
            # any non-NULL pointer announces, even an empty list (then it is
            # not read): the unique buffer's address serves
            ann = (_dev_ptr(announce, torch.int64, "announce") if an else args[4], an)
        nu, tk = ctypes.c_uint64(), ctypes.c_uint64()
        _check(lib().lsmgnn_gather_async(*args[:3], *ann, *args[3:], ctypes.byref(nu), ctypes.byref(tk),
                                         _stream_handle(stream, self.device)), "lsmgnn_gather_async")
        return tk.value, self._result(nu.value, n, out, unique, inv_t, oc_t)

    def wait(self, ticket, stream=None):
        """Make `stream` wait (on the device) for gather `ticket`."""
        _check(lib().lsmgnn_gather_wait(self._h, int(ticket), _stream_handle(stream, self.device)),
               "lsmgnn_gather_wait")

    def sync(self):
        _check(lib().lsmgnn_sync(self._h), "lsmgnn_sync")

    def stats(self):
        last, total = Counts(), Counts()
        _check(lib().lsmgnn_stats(self._h, ctypes.byref(last), ctypes.byref(total)), "lsmgnn_stats")
        return ({f: getattr(last, f) for f in COUNT_FIELDS}, {f: getattr(total, f) for f in COUNT_FIELDS})

    def export_state(self):
        tags = np.empty(self.num_sets * 8, np.uint32)
        ring = np.empty(max(self.victim_rows, 1), np.uint32)
        tail, t = ctypes.c_uint64(), ctypes.c_uint64()
        _check(lib().lsmgnn_export_state(self._h, tags.ctypes.data, ring.ctypes.data, ctypes.byref(tail),
                                         ctypes.byref(t)), "lsmgnn_export_state")
        return dict(tags=tags.reshape(self.num_sets, 8), ring_tags=ring[: self.victim_rows],
                    ring_tail=tail.value, t=t.value)

    def set_profiling(self, on: bool):
        _check(lib().lsmgnn_set_profiling(self._h, 1 if on else 0), "lsmgnn_set_profiling")

    def profile(self) -> dict:
        p = Profile()
        _check(lib().lsmgnn_get_profile(self._h, ctypes.byref(p)), "lsmgnn_get_profile")
        return {f: getattr(p, f) for f, _ in Profile._fields_}
