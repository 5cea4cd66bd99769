"""Side-by-side driver: the GPU library (through its C ABI) and the CPU oracle
consume the same seeded request stream and are compared after every gather.

Compared per gather: the ascending unique IDs, the inverse index, the outcome
of every unique ID (hit / victim hit / miss), all counters, and the gathered
rows (bit-exact).  Compared at the end: every cache tag, every ring tag, the
ring tail and the gather count.  Integer work, so everything must match
exactly.
"""
from __future__ import annotations

import sys
import time

import numpy as np

from oracle.oracle import Oracle
from paper_2407_15264_amd import lsmgnn
from paper_2407_15264_amd import workload as W

COUNT_KEYS = ("batch", "requests", "unique", "hits", "victim_hits", "misses", "evictions", "enqueued", "dropped",
              "request_hits", "request_victim_hits")


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


class Store:
    """A host feature table (num_nodes x row_bytes): pinned (read by the GPU
    directly), or with pinned=False ordinary pageable memory (rows copied by
    the library's host threads)."""

    def __init__(self, num_nodes, dim, elt_bytes=4, seed=0, fill=None, pinned=True):
        self.num_nodes, self.row_bytes = num_nodes, dim * elt_bytes
        self._alloc(pinned)
        if fill is None:
            W.fill_features(self.np.ctypes.data, dim, elt_bytes, 0, num_nodes, seed)
        else:
            self.np[:] = fill

    def _alloc(self, pinned):
        self.pinned = pinned
        if pinned:
            self.buf = lsmgnn.PinnedBuffer(self.num_nodes * self.row_bytes)
            self.np = self.buf.numpy(np.uint8, (self.num_nodes, self.row_bytes))
        else:
            self.np = np.empty((self.num_nodes, self.row_bytes), np.uint8)
            self.buf = self.np

    @classmethod
    def random_bytes(cls, num_nodes, row_bytes, seed=0, pinned=True):
        rng = np.random.default_rng(seed)
        s = cls.__new__(cls)
        s.num_nodes, s.row_bytes = num_nodes, row_bytes
        s._alloc(pinned)
        s.np[:] = rng.integers(0, 256, (num_nodes, row_bytes), dtype=np.uint8)
        return s


def compare_state(cache, orc, where=""):
    g, o = cache.export_state(), orc.export_state()
    if not np.array_equal(g["tags"], o["tags"]):
        bad = np.argwhere(g["tags"] != o["tags"])[:5]
        raise AssertionError(f"{where}: cache tags differ at {bad.tolist()}: gpu {g['tags'][tuple(bad[0])]} "
                             f"oracle {o['tags'][tuple(bad[0])]}")
    if not np.array_equal(g["ring_tags"], o["ring_tags"]):
        bad = np.flatnonzero(g["ring_tags"] != o["ring_tags"])[:5]
        raise AssertionError(f"{where}: ring tags differ at {bad.tolist()}")
    assert g["ring_tail"] == o["ring_tail"], (where, g["ring_tail"], o["ring_tail"])
    assert g["t"] == o["t"], (where, g["t"], o["t"])


def run_parity(store: Store, static, num_sets, victim_rows, lookahead, batches, announce=None,
               near_threshold=0, rows="all", max_batch=None, device=0, state_every=0, label="parity",
               store_gpu=None, policy="hybrid", victim_mode="fifo", refresh_period=1, per_gather_stats=True):
    """rows: 'all' -> compare every gathered row with the oracle's; an int k ->
    compare with the oracle on every k-th gather and, on every gather, with the
    backing-store rows indexed on the GPU (store_gpu, a device copy).

    per_gather_stats=False: the counters are compared only as totals at the
    end, so no call waits for the library's internal streams between gathers
    (a blocking gather waits only for its own rows); the rows, unique IDs,
    inverse and outcomes are still compared after every gather."""
    import torch
    dev = torch.device("cuda", device)
    announce = batches if announce is None else announce
    mb = max_batch or max(1, max((len(b) for b in list(batches) + list(announce)), default=1))
    L = lookahead
    cache = lsmgnn.FeatureCache(store.num_nodes, store.row_bytes, store.buf, static, num_sets, victim_rows, L, mb,
                                near_threshold=near_threshold, device=device, pageable=not store.pinned,
                                policy=policy, victim_mode=victim_mode, refresh_period=refresh_period)
    orc = Oracle(store.num_nodes, store.row_bytes, static, num_sets, victim_rows, L,
                 near_threshold=near_threshold, store=store.np, policy=policy, victim_mode=victim_mode,
                 refresh_period=refresh_period)
    dev_ann = [torch.as_tensor(np.asarray(a, np.int64)).to(dev) for a in announce]
    dev_bat = [torch.as_tensor(np.asarray(b, np.int64)).to(dev) for b in batches]
    for j in range(min(L + 1, len(announce))):
        cache.advance(dev_ann[j])
        orc.advance(announce[j])
    t0 = time.time()
    o_tot = {k: 0 for k in COUNT_KEYS}
    for b, ids in enumerate(batches):
        where = f"{label} gather {b}"
        r = cache.gather(dev_bat[b], inverse=True, outcome=True)
        full_rows = rows == "all" or (isinstance(rows, int) and b % rows == 0)
        o = orc.gather(np.asarray(ids, np.int64), rows=full_rows)
        U = r.n_unique
        assert U == o["uniq"].size, (where, U, o["uniq"].size)
        uq = r.unique.cpu().numpy()
        if not np.array_equal(uq, o["uniq"]):
            raise AssertionError(f"{where}: unique IDs differ")
        if not np.array_equal(r.inverse.cpu().numpy(), o["inv"]):
            raise AssertionError(f"{where}: inverse differs")
        oc = r.outcome.cpu().numpy()
        if not np.array_equal(oc, o["outcome"]):
            bad = np.flatnonzero(oc != o["outcome"])[:5]
            raise AssertionError(f"{where}: outcome differs at unique idx {bad.tolist()} "
                                 f"(ids {o['uniq'][bad].tolist()}): gpu {oc[bad].tolist()} "
                                 f"oracle {o['outcome'][bad].tolist()}")
        if per_gather_stats:
            last, _ = cache.stats()
            for k in COUNT_KEYS:
                if last[k] != o["stats"][k]:
                    raise AssertionError(f"{where}: counter {k}: gpu {last[k]} oracle {o['stats'][k]}")
        else:
            for k in COUNT_KEYS:
                if k != "batch":
                    o_tot[k] += o["stats"][k]
        if full_rows:
            if not np.array_equal(r.out.cpu().numpy(), o["out"]):
                bad = np.flatnonzero((r.out.cpu().numpy() != o["out"]).any(axis=1))[:5]
                raise AssertionError(f"{where}: gathered rows differ at unique idx {bad.tolist()} "
                                     f"outcomes {oc[bad].tolist()}")
        elif store_gpu is not None:
            ref = store_gpu.index_select(0, r.unique)
            if not torch.equal(r.out, ref):
                raise AssertionError(f"{where}: gathered rows differ from the backing store")
        if state_every and (b + 1) % state_every == 0:
            compare_state(cache, orc, where)
        if b + L + 1 < len(announce):
            cache.advance(dev_ann[b + L + 1])
            orc.advance(announce[b + L + 1])
    compare_state(cache, orc, f"{label} end")
    tot = cache.stats()[1]
    if not per_gather_stats:
        for k, v in o_tot.items():
            if k != "batch" and tot[k] != v:
                raise AssertionError(f"{label}: total {k}: gpu {tot[k]} oracle {v}")
    cache.close()
    orc.close()
    return dict(total=tot, seconds=time.time() - t0)


def device_store(store: Store, device=0):
    """A device copy of the backing store, for checking gathered rows on the GPU."""
    import torch
    dev = torch.device("cuda", device)
    if not store.pinned:
        return torch.from_numpy(store.np).to(dev)
    t = torch.empty((store.num_nodes, store.row_bytes), dtype=torch.uint8, device=dev)
    lsmgnn.copy_bytes(t.data_ptr(), store.buf.ptr, store.num_nodes * store.row_bytes)
    return t


class _Lane:
    """One cache driven in the launch configuration of bench.py
    (lsmgnn_gather_async with the next minibatch's announcement, or a separate
    lsmgnn_advance; two gathers in flight; three rotating output-buffer sets),
    with its oracle beside it.  Each gather's unique IDs, inverse, outcomes and
    rows are compared once it has been waited for."""

    def __init__(self, store, static, num_sets, victim_rows, lookahead, batches, rows, store_gpu, label,
                 combined, near_threshold, device, row_sample=0, policy="hybrid", victim_mode="fifo",
                 refresh_period=1, mixed_seed=None):
        import torch
        self.torch = torch
        self.store, self.row_sample = store, row_sample
        self.rng = np.random.default_rng(12345)
        # mixed_seed: each gather goes through the blocking call (then a
        # separate advance) or the pipelined one, by a seeded coin
        self.mixed = None if mixed_seed is None else np.random.default_rng(mixed_seed)
        dev = torch.device("cuda", device)
        self.mb = max(1, max(len(b) for b in batches))
        self.L, self.batches, self.rows, self.store_gpu, self.label = lookahead, batches, rows, store_gpu, label
        self.combined = combined
        self.cache = lsmgnn.FeatureCache(store.num_nodes, store.row_bytes, store.buf, static, num_sets, victim_rows,
                                         lookahead, self.mb, near_threshold=near_threshold, device=device,
                                         pageable=not store.pinned, policy=policy, victim_mode=victim_mode,
                                         refresh_period=refresh_period)
        self.orc = Oracle(store.num_nodes, store.row_bytes, static, num_sets, victim_rows, lookahead,
                          near_threshold=near_threshold, store=store.np, policy=policy, victim_mode=victim_mode,
                          refresh_period=refresh_period)
        self.db = [torch.as_tensor(np.asarray(b, np.int64)).to(dev) for b in batches]
        if rows is not None and rows != 0:
            # the oracle writes its rows into pinned memory; they are compared
            # with the gathered rows on the GPU
            nbytes = self.mb * store.row_bytes
            self.ref_host = torch.empty(nbytes, dtype=torch.uint8).pin_memory()
            self.ref_np = self.ref_host.numpy()
            self.ref_dev = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        self.bufs = [(torch.empty(self.mb * store.row_bytes, dtype=torch.uint8, device=dev),
                      torch.empty(self.mb, dtype=torch.int64, device=dev),
                      torch.empty(self.mb, dtype=torch.int64, device=dev),
                      torch.empty(self.mb, dtype=torch.uint8, device=dev)) for _ in range(3)]
        for j in range(min(lookahead + 1, len(batches))):
            self.cache.advance(self.db[j])
            self.orc.advance(batches[j])
        self.pending = []

    def issue(self, b):
        out, uq, inv, oc = self.bufs[b % 3]
        L = self.L
        nxt = self.db[b + L + 1] if b + L + 1 < len(self.batches) else None
        if self.mixed is not None and self.mixed.random() < 0.5:
            r = self.cache.gather(self.db[b], out=out, unique=uq, inverse=inv, outcome=oc)
            if nxt is not None:
                self.cache.advance(nxt)
            self.pending.append((None, r, b))
            return
        if self.combined:
            ticket, r = self.cache.gather_async(self.db[b], out, uq, inverse=inv, outcome=oc, announce=nxt)
        else:
            ticket, r = self.cache.gather_async(self.db[b], out, uq, inverse=inv, outcome=oc)
            if nxt is not None:
                self.cache.advance(nxt)
        self.pending.append((ticket, r, b))

    def check_oldest(self):
        torch = self.torch
        ticket, r, b = self.pending.pop(0)
        if ticket is not None:  # a blocking gather has completed already
            self.cache.wait(ticket)
        torch.cuda.current_stream().synchronize()
        where = f"{self.label} gather {b}"
        rows = self.rows
        full_rows = rows == "all" or (isinstance(rows, int) and b % rows == 0)
        o = self.orc.gather(np.asarray(self.batches[b], np.int64), rows=full_rows,
                            out=self.ref_np if full_rows else None)
        assert r.n_unique == o["uniq"].size, (where, r.n_unique, o["uniq"].size)
        if not np.array_equal(r.unique.cpu().numpy(), o["uniq"]):
            raise AssertionError(f"{where}: unique IDs differ")
        if not np.array_equal(r.inverse.cpu().numpy(), o["inv"]):
            raise AssertionError(f"{where}: inverse differs")
        oc = r.outcome.cpu().numpy()
        if not np.array_equal(oc, o["outcome"]):
            bad = np.flatnonzero(oc != o["outcome"])[:5]
            raise AssertionError(f"{where}: outcome differs at unique idx {bad.tolist()}")
        if full_rows:
            nb = r.n_unique * self.store.row_bytes
            ref = self.ref_dev[:nb]
            ref.copy_(self.ref_host[:nb], non_blocking=True)
            got = r.out.reshape(-1)
            if not torch.equal(got, ref):
                bad = torch.nonzero((got != ref).view(r.n_unique, -1).any(dim=1)).flatten()[:5].tolist()
                raise AssertionError(f"{where}: gathered rows differ from the oracle's at unique idx {bad} "
                                     f"(outcomes {oc[bad].tolist()})")
        elif self.store_gpu is not None:
            if not torch.equal(r.out, self.store_gpu.index_select(0, r.unique)):
                raise AssertionError(f"{where}: gathered rows differ from the backing store")
        elif self.row_sample and r.n_unique:
            # a seeded sample of the gathered rows against the host store
            k = min(self.row_sample, r.n_unique)
            u = np.sort(self.rng.choice(r.n_unique, size=k, replace=False))
            got = r.out[torch.as_tensor(u, device=r.out.device)].cpu().numpy()
            if not np.array_equal(got, self.store.np[o["uniq"][u]]):
                raise AssertionError(f"{where}: sampled gathered rows differ from the backing store")
        if b + self.L + 1 < len(self.batches):
            self.orc.advance(self.batches[b + self.L + 1])

    def drain(self):
        while self.pending:
            self.check_oldest()

    def finish(self):
        self.drain()
        tot_gpu = self.cache.stats()[1]
        tot_orc = self.orc.stats()[1]
        for k in COUNT_KEYS:
            assert tot_gpu[k] == tot_orc[k], (self.label, k, tot_gpu[k], tot_orc[k])
        compare_state(self.cache, self.orc, f"{self.label} end")
        self.cache.close()
        self.orc.close()
        return tot_gpu


def _run_lanes(lanes, nb, state_every, label):
    t0 = time.time()
    for b in range(nb):
        for ln in lanes:
            ln.issue(b)
        if state_every and (b + 1) % state_every == 0:
            # the exported state is the one after every issued gather: drain first
            for ln in lanes:
                ln.drain()
                compare_state(ln.cache, ln.orc, f"{ln.label} gather {b}")
            log(f"  {label}: {b + 1} gathers checked ({time.time() - t0:.1f} s)")
        else:
            for ln in lanes:
                if len(ln.pending) == 2:
                    ln.check_oldest()
    totals = [ln.finish() for ln in lanes]
    return totals, time.time() - t0


def run_async_parity(store: Store, static, num_sets, victim_rows, lookahead, batches, rows="all", store_gpu=None,
                     state_every=0, label="async", combined=True, near_threshold=0, device=0, row_sample=0,
                     policy="hybrid", victim_mode="fifo", refresh_period=1):
    """One cache in the launch configuration of bench.py, against the oracle:
    unique IDs, inverse, outcomes and rows of every gather (rows as in
    run_parity), counters as totals, the cache and ring state every
    `state_every` gathers and at the end."""
    ln = _Lane(store, static, num_sets, victim_rows, lookahead, batches, rows, store_gpu, label, combined,
               near_threshold, device, row_sample, policy, victim_mode, refresh_period)
    totals, seconds = _run_lanes([ln], len(batches), state_every, label)
    return dict(total=totals[0], seconds=seconds)


def run_mixed_parity(store: Store, static, num_sets, victim_rows, lookahead, batches, seed, state_every=0,
                     label="mixed", near_threshold=0, policy="hybrid", victim_mode="fifo", refresh_period=1):
    """Blocking and pipelined gathers interleaved on one cache (a seeded coin
    per gather), with no call in between that waits for the library's
    streams except the checks' own waits: every gather's unique IDs, inverse,
    outcomes and rows, the counters as totals, the state every `state_every`
    gathers and at the end."""
    ln = _Lane(store, static, num_sets, victim_rows, lookahead, batches, "all", None, label, True, near_threshold,
               0, 0, policy, victim_mode, refresh_period, mixed_seed=seed)
    totals, seconds = _run_lanes([ln], len(batches), state_every, label)
    return dict(total=totals[0], seconds=seconds)


def run_typed_async_parity(stores, statics, shapes, type_batches, rows=50, stores_gpu=None, state_every=0,
                           label="typed", device=0):
    """A typed workload: one cache per node type, all driven together, minibatch
    by minibatch (each type's gather of minibatch b is issued before any check
    of minibatch b-1), each against its own oracle."""
    lanes = [_Lane(stores[t], statics[t], shapes[t].num_sets, shapes[t].victim_rows, shapes[t].lookahead,
                   type_batches[t], rows, None if stores_gpu is None else stores_gpu[t], f"{label} type {t}", True,
                   shapes[t].near_threshold, device) for t in range(len(stores))]
    totals, seconds = _run_lanes(lanes, len(type_batches[0]), state_every, label)
    return dict(totals=totals, seconds=seconds)


def config_stream(cfg, batches=None):
    wl = W.Workload(cfg, batches)
    return wl, [wl.batch(b) for b in range(wl.num_batches)]
