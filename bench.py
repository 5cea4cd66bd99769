#!/usr/bin/env python3
"""Benchmark of the per-minibatch feature gather through the MI355X cache.

One step = one pass of the whole hot path over one minibatch: a gather of the
minibatch's raw request IDs (dedup, set walk with hybrid eviction, victim ring,
hit/miss/victim-hit row movement, fills) and the announcement of the minibatch
L+1 ahead.  By default both go through one lsmgnn_gather_async call with two
minibatches in flight; --sync uses lsmgnn_gather then lsmgnn_advance.  All
request streams are on the GPU and the feature table is in pinned host memory
before the timed region starts.

Default workload: R-MAT graph with 2^20 nodes and 2^24 edges (a, b, c, d =
0.57, 0.19, 0.19, 0.05), fp32 x 256 features (1 GiB pinned host store), GraphSAGE
sampling of 1024 seeds per minibatch with fanout (15, 10, 5), an 8-way cache
holding 10% of the nodes, a victim ring of 5% of the nodes, lookahead 4.
--workload picks another shape by name; the typed graph (rmat-20M-e250M-4types)
runs one cache per node type and a step gathers the minibatch's IDs of every
type.

Prints one JSON line.  `value` is gathered feature bytes (unique rows x row
bytes) per second over the timed steps; `roofline` rates the dominant data
kernel against its bound, timed with HIP events on the gather's stream.  The
timed steps run over the same minibatches three times, each time from fresh
caches: without the library's timing events (`value`), with them (the
per-kernel figures, and `profiled_pass`), and untimed with every gather's
counts read (`per_minibatch`).
"""
import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "gathered feature GB/s per minibatch stream (% HBM/host-link roofline) + hit rate"
HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E, published
SAMPLE_AHEAD = 2                # --gpu-sampler: minibatches sampled before their announcement
PCIE5_X16_PEAK_GBPS = 64.0      # host link, published per direction
HIT_PATH_TARGET_FRAC = 0.70     # hit-path goal: this fraction of the HBM peak


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def copy_kernels_hash():
    src = open(os.path.join(ROOT, "paper_2407_15264_amd", "csrc", "gather_kernels.hip")).read()
    a = src.index("// -------------------------------------------------------------- row copies")
    b = src.index("// ------------------------------------------------------------ calibration")
    return hashlib.sha256(src[a:b].encode()).hexdigest()


def recorded_traffic(workload, kernel):
    """HBM/link bytes per launch of `kernel` from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE passes, each scaled by its reading for a copy of
    known size; None when absent or when the row-copy kernels have changed
    since the counters were taken."""
    path = os.path.join(ROOT, "profiles", f"counters_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("copy_kernels_source_sha256") != copy_kernels_hash() or kernel not in rec["kernels"]:
        return None
    k, cal = rec["kernels"][kernel], rec["calibration"]
    fetch = k["fetch_kib"] * 1024 * cal["fetch_scale"]
    write = k["write_kib"] * 1024 * cal["write_scale"]
    return {"bytes": fetch + write, "fetch_bytes": fetch, "write_bytes": write,
            "source": os.path.relpath(path, ROOT)}


def duplex_probe(nbytes=1 << 30):
    """Both link directions at once, as in the pipeline (which sends about half
    as many bytes out as it reads in): the runtime's copies, nbytes host to
    device on one stream and nbytes/2 device to host on another, from and to
    pinned memory.  Runs in a process of its own: the two extra streams would
    otherwise take hardware queues that the library's streams need."""
    import torch
    dev = torch.device("cuda", 0)
    half = nbytes // 32 * 16
    h_in = torch.ones(nbytes, dtype=torch.uint8).pin_memory()
    h_out = torch.empty(half, dtype=torch.uint8).pin_memory()
    d_in = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    d_out = torch.zeros(half, dtype=torch.uint8, device=dev)
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    best = None
    for it in range(9):  # the first three warm the link and the copy path up, untimed
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        with torch.cuda.stream(sa):
            ev[0].record()
            d_in.copy_(h_in, non_blocking=True)
            ev[1].record()
        with torch.cuda.stream(sb):
            ev[2].record()
            h_out.copy_(d_out, non_blocking=True)
            ev[3].record()
        torch.cuda.synchronize()
        ta, tb = ev[0].elapsed_time(ev[1]) / 1e3, ev[2].elapsed_time(ev[3]) / 1e3
        span = max(ev[0].elapsed_time(ev[1]), ev[0].elapsed_time(ev[3])) / 1e3
        r = {"h2d_GBps": nbytes / ta / 1e9, "d2h_GBps": half / tb / 1e9,
             "total_GBps": (nbytes + half) / span / 1e9, "bytes_in": nbytes, "bytes_out": half,
             "how": "runtime copies from and to pinned memory on two streams, started together; best of 6 "
                    "after 3 untimed"}
        if it >= 3 and (best is None or r["total_GBps"] > best["total_GBps"]):
            best = r
    print(json.dumps(best), flush=True)


def child_probe(flag):
    """A probe (--duplex-probe, --hbm-probe) in a child process: its JSON
    result, or None if it fails."""
    import subprocess
    try:
        out = subprocess.run([sys.executable, os.path.abspath(__file__), flag], capture_output=True,
                             text=True, timeout=300)
        return json.loads(out.stdout.strip().splitlines()[-1]) if out.returncode == 0 else None
    except (subprocess.SubprocessError, ValueError, IndexError, OSError):
        return None


def measure_ceilings(torch, lsmgnn, store_ptr, nbytes, duplex, hbm):
    """Host-link and HBM ceilings in this run: pinned H2D DMA, zero-copy reads
    and writes by the 128-bit copy kernel; `duplex` and `hbm` are
    duplex_probe()'s and hbm_probe()'s results, measured in child processes
    beforehand."""
    dev = torch.device("cuda", 0)
    nbytes = min(nbytes, 1 << 30) // 16 * 16
    d0 = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    d1 = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    pinned = torch.empty(nbytes, dtype=torch.uint8).pin_memory()
    res = {}

    def best(fn, reps=5):
        ts = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            ts.append(time.perf_counter() - t0)
        return min(ts)

    res["dma_h2d_GBps"] = nbytes / best(lambda: d0.copy_(pinned, non_blocking=True)) / 1e9
    res["dma_d2h_GBps"] = nbytes / best(lambda: pinned.copy_(d0, non_blocking=True)) / 1e9
    res["zero_copy_read_GBps"] = nbytes / best(lambda: lsmgnn.copy_bytes(d0.data_ptr(), store_ptr, nbytes)) / 1e9
    res["zero_copy_write_GBps"] = nbytes / best(
        lambda: lsmgnn.copy_bytes(pinned.data_ptr(), d0.data_ptr(), nbytes)) / 1e9
    del d0, d1, pinned
    rates = [v for k, v in (hbm or {}).items() if k.endswith("MiB")]
    res["hbm_copy_GBps"] = max(rates) if rates else None
    res["hbm_copy_detail"] = hbm
    res["duplex"] = duplex
    res["bytes"] = nbytes
    return res


def hbm_probe():
    """The HBM ceiling: the best device-to-device copy over sizes and copy
    engines (the library's 128-bit copy kernel, and the runtime's copy behind
    torch's copy_), read + write bytes per second.  The runtime's copy is timed
    with GPU events; the library's calibration call synchronises, so its time is
    taken on the host less that of a 16-byte call (the launch and the wait).
    Runs in a process of its own: in the bench process, the runtime's
    device-to-device copies and the buffers left the ring writes of the gathers
    measured afterwards about a quarter slower."""
    import torch
    from paper_2407_15264_amd import lsmgnn
    dev = torch.device("cuda", 0)

    def best_host(fn, reps=7):
        ts = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            ts.append(time.perf_counter() - t0)
        return min(ts)

    def best_events(fn, reps=7):
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            e1.synchronize()
            ts.append(e0.elapsed_time(e1) / 1e3)
        return min(ts)

    hbm = {}
    small_a = torch.ones(16, dtype=torch.uint8, device=dev)
    small_b = torch.empty(16, dtype=torch.uint8, device=dev)
    call = best_host(lambda: lsmgnn.copy_bytes(small_b.data_ptr(), small_a.data_ptr(), 16), reps=21)
    hbm["call_overhead_us"] = round(1e6 * call, 1)
    # at least 1 GiB: a smaller copy runs partly out of the 256 MB MALL
    for size in (1 << 30, 4 << 30, 8 << 30):
        a = torch.empty(size, dtype=torch.uint8, device=dev)
        b = torch.empty(size, dtype=torch.uint8, device=dev)
        a.fill_(1)
        t = best_host(lambda: lsmgnn.copy_bytes(b.data_ptr(), a.data_ptr(), size)) - call
        hbm[f"copy_kernel_{size >> 20}MiB"] = round(2 * size / t / 1e9, 1)
        hbm[f"runtime_copy_{size >> 20}MiB"] = round(2 * size / best_events(lambda: b.copy_(a)) / 1e9, 1)
        del a, b
    print(json.dumps(hbm), flush=True)


def make_parts(W, cfg, nb):
    """One part per cache: a homogeneous workload has one, a typed workload one
    per node type (each with its own feature width, store, cache and ring)."""
    import numpy as np
    if isinstance(cfg, W.HeteroConfig):
        wl = W.HeteroWorkload(cfg, nb)
        parts = [dict(label=f"type {t}", num_nodes=n, dim=d, elt=cfg.elt_bytes, seed=cfg.seed + 1 + t,
                      static=wl.static[t], shape=cfg.cache_shape(t), batches=wl.type_batches(t))
                 for t, (n, d) in enumerate(zip(cfg.type_counts(), cfg.dims))]
        # what a GPU sampler needs: the global graph and seeds, each node's type and index within it
        parts[0].update(graph=wl.graph, seeds=wl.seeds, node_type=wl.node_type, node_local=wl.node_local,
                        global_max=int(np.diff(wl.offsets).max()))
        requests = float(sum(b.size for p in parts for b in p["batches"])) / nb
    else:
        wl = W.Workload(cfg, nb)
        parts = [dict(label="all", num_nodes=cfg.num_nodes, dim=cfg.dim, elt=cfg.elt_bytes, seed=cfg.seed,
                      static=wl.static, shape=cfg.cache, batches=[wl.batch(b) for b in range(nb)],
                      graph=wl.graph, seeds=wl.seeds)]
        requests = float(wl.ids.size) / nb
    for p in parts:
        p["R"] = p["dim"] * p["elt"]
    return parts, requests


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def steady_start(cfg, L):
    """First timed minibatch: after max(L+1, 10 %) of the configured run, past
    the cold start (at first nearly every request misses).  A cache much
    larger than a minibatch keeps filling after that, and its hit rate keeps
    rising over the run."""
    return max(L + 1, -(-cfg.batches // 10))


def cpu_baseline(parts, budget_s, first, policy="hybrid", victim_rows=None, victim_mode="fifo", refresh_period=1):
    """The CPU oracle (single-threaded C, one instance per part) on the same
    stream: gathers 0 .. first-1 untimed without rows (the cold-start fill),
    then the timed minibatches from `first` with rows, stopped after about
    budget_s seconds."""
    from oracle.oracle import Oracle
    orcs = []
    for p in parts:
        sh = p["shape"]
        o = Oracle(p["num_nodes"], p["R"], p["static"], sh.num_sets,
                   sh.victim_rows if victim_rows is None else victim_rows, sh.lookahead,
                   near_threshold=sh.near_threshold, store=p["store_np"], policy=policy, victim_mode=victim_mode,
                   refresh_period=refresh_period)
        for j in range(sh.lookahead + 1):
            o.advance(p["batches"][j])
        orcs.append(o)
    L = parts[0]["shape"].lookahead
    nb = len(parts[0]["batches"])
    for b in range(first):
        for p, o in zip(parts, orcs):
            o.gather(p["batches"][b], rows=False)
            o.advance(p["batches"][b + L + 1])
    t0 = time.perf_counter()
    done, rows, nbytes = first, 0, 0
    while done < nb - L - 1 and time.perf_counter() - t0 < budget_s:
        for p, o in zip(parts, orcs):
            r = o.gather(p["batches"][done], rows=True)
            o.advance(p["batches"][done + L + 1])
            rows += r["uniq"].size
            nbytes += r["uniq"].size * p["R"]
        done += 1
    dt = time.perf_counter() - t0
    for o in orcs:
        o.close()
    return {"value": nbytes / dt / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"gathers {first}..{done - 1} of the same stream ({done - first} minibatches from the first "
                      f"timed one, {rows} unique rows, {dt:.1f} s; gathers 0..{first - 1} run before, untimed), "
                      "rows copied with memcpy from the host store",
            "rows_per_s": rows / dt,
            "parts": len(parts), "seconds_per_minibatch": dt / max(done - first, 1),
            "cpu": _cpu_model(), "host_cpus": os.cpu_count()}


def gpu_sampler_check(torch, lsmgnn, W, parts, cfg, L, nb, warmup, steps, dev):
    """The GPU lists against the host-generated ones (every minibatch of the
    run and every part, element by element), and their rate alone: the timed
    minibatches sampled (and split) back to back, against the host sampler on
    the same minibatches."""
    import numpy as np
    first, typed = parts[0], len(parts) > 1
    max_len = max(1, max(b.size for p in parts for b in p["batches"]))
    lists = GpuLists(torch, lsmgnn, first, cfg, L, max_len, dev, typed=typed)
    mismatched = sum(int(not np.array_equal(lists.get(b, t).cpu().numpy(), p["batches"][b]))
                     for b in range(nb) for t, p in enumerate(parts))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for b in range(warmup, warmup + steps):
        lists.get(b, 0)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    requests = sum(int(p["batches"][b].size) for p in parts for b in range(warmup, warmup + steps))
    t0 = time.perf_counter()
    W.sample_batches(first["graph"], first["seeds"], cfg.batch_size, cfg.fanout, warmup, warmup + steps, cfg.seed)
    dh = time.perf_counter() - t0
    lists.close()
    return {"identical_to_host_lists": mismatched == 0, "minibatches_compared": nb, "parts": len(parts),
            "alone_ms_per_minibatch": 1e3 * dt / steps, "alone_requests_per_s": requests / dt,
            "split_by_type": typed,
            "host_sampler_ms_per_minibatch": 1e3 * dh / steps,
            "host_sampler_threads": int(os.environ.get("OMP_NUM_THREADS", os.cpu_count()))}


def hit_path_alone(parts, b, reps=5):
    """The hit copy with no host fetch running beside it: minibatch b gathered
    again (once to make its rows resident, then `reps` timed passes that find
    nearly all of them in the cache), with the same per-launch events.  Run
    after the timed region; it changes the caches' state."""
    ms = rows = nbytes = launches = uniq = hits = 0
    for p in parts:
        c, db = p["cache"], p["dev_batches"]
        out, uq, inv = p["bufs"][0]
        c.gather(db[b], out=out, unique=uq, inverse=inv)
        _, before = c.stats()
        c.set_profiling(True)
        for _ in range(reps):
            c.gather(db[b], out=out, unique=uq, inverse=inv)
        pr = c.profile()
        c.set_profiling(False)
        _, after = c.stats()
        ms += pr["hbm_copy_ms"]
        launches += pr["hbm_copy_launches"]
        rows += pr["hbm_copy_rows"]
        nbytes += 2 * pr["hbm_copy_rows"] * p["R"]
        uniq += after["unique"] - before["unique"]
        hits += after["hits"] - before["hits"]
    gbps = nbytes / (ms / 1e3) / 1e9 if ms > 0 else 0.0
    return {"achieved": gbps, "frac": gbps / HBM_PEAK_GBPS, "avg_launch_us": 1e3 * ms / max(launches, 1),
            "bytes_per_launch": nbytes / max(launches, 1), "hit_rate": hits / max(uniq, 1),
            "how": f"minibatch {b} gathered again {reps} times after the timed region (blocking calls); "
                   "bytes = hit rows x row bytes x 2 (read + write)"}


def side_stream(torch):
    """One more HIP stream, at default priority, from the runtime PyTorch
    loaded (a torch.cuda.Stream would instantiate PyTorch's whole stream pool)."""
    import ctypes
    hip = ctypes.CDLL(os.path.join(os.path.dirname(torch.__file__), "lib", "libamdhip64.so"))
    s = ctypes.c_void_p()
    rc = hip.hipStreamCreateWithFlags(ctypes.byref(s), ctypes.c_uint(1))  # hipStreamNonBlocking
    if rc != 0:
        raise RuntimeError(f"hipStreamCreateWithFlags failed ({rc})")
    return torch.cuda.ExternalStream(s.value)


class GpuLists:
    """Request lists sampled on the GPU on demand (lsmgnn_sample_async, then
    for a typed workload lsmgnn_split_by_type_async), for parts that index
    them like the resident host-generated lists (part_view).  The sampler runs
    on `stream` (a training loop's data-loading stream); prefetch(b) queues
    minibatch b's lists, and indexing waits only for them.  A ring of
    L+3+ahead buffers: the lists prefetched at step b (minibatch b+L+1+ahead)
    take the buffers of minibatch b-2, whose gathers' metadata has finished by
    then (the host has seen gather b-1's unique counts, and the metadata
    stream is in order)."""

    def __init__(self, torch, lsmgnn, first, cfg, L, max_len, dev, stream=None, ahead=0, typed=False):
        import numpy as np
        self.torch, self.lsmgnn, self.np = torch, lsmgnn, np
        g = first["graph"]
        self.off = torch.as_tensor(g.offsets).to(dev)
        self.adj = torch.as_tensor(g.adj.view("int32")).to(dev)
        self.sampler = lsmgnn.GpuSampler(self.off, self.adj, cfg.fanout, seed=cfg.seed)
        self.seeds = torch.as_tensor(first["seeds"]).to(dev)
        self.B = cfg.batch_size
        self.stream = stream
        K = L + 3 + ahead
        self.T = cfg.num_types if typed else 0
        gmax = first.get("global_max", max_len)
        self.glob = [torch.empty(gmax, dtype=torch.int64, device=dev) for _ in range(K)]
        self.res = lsmgnn.PinnedBuffer(16 * K)  # sampler: (length, status) per buffer
        self.res_np = self.res.numpy(np.uint64, (K, 2))
        if self.T:
            self.node_type = torch.as_tensor(first["node_type"]).to(dev)
            self.local = torch.as_tensor(first["node_local"].astype(np.int32)).to(dev)
            self.outs = [[torch.empty(max_len, dtype=torch.int64, device=dev) for _ in range(self.T)]
                         for _ in range(K)]
            self.work = torch.empty(lsmgnn.split_work_bytes(gmax, self.T), dtype=torch.uint8, device=dev)
            self.tres = lsmgnn.PinnedBuffer(8 * (self.T + 1) * K)  # split: lengths + status per buffer
            self.tres_np = self.tres.numpy(np.uint64, (K, self.T + 1))
        self.events = [torch.cuda.Event() for _ in range(K)]
        self.issued = [None] * K  # minibatch queued into each buffer
        self.ready = [None] * K   # its lists, once waited for

    def _record(self, k):
        self.events[k].record(self.stream if self.stream is not None else self.torch.cuda.current_stream())

    def prefetch(self, b):
        k = b % len(self.glob)
        if self.issued[k] == b:
            return
        self.sampler.sample_async(self.seeds[b * self.B:(b + 1) * self.B], b, self.glob[k], self.res.ptr + 16 * k,
                                  stream=self.stream)
        self._record(k)
        if self.T:
            # the split needs the list's length on the host: wait for this sampling only
            self.events[k].synchronize()
            n, status = int(self.res_np[k, 0]), int(self.res_np[k, 1])
            if status != 0:
                raise RuntimeError(f"lsmgnn_sample_async of minibatch {b}: status {status}")
            self.lsmgnn.split_by_type_async(self.glob[k][:n], self.node_type, self.local, self.outs[k], self.work,
                                            self.tres.ptr + 8 * (self.T + 1) * k, stream=self.stream)
            self._record(k)
        self.issued[k], self.ready[k] = b, None

    def get(self, b, t):
        k = b % len(self.glob)
        self.prefetch(b)
        if self.ready[k] is None:
            self.events[k].synchronize()
            if self.T:
                status = int(self.tres_np[k, self.T])
                if status != 0:
                    raise RuntimeError(f"lsmgnn_split_by_type_async of minibatch {b}: status {status}")
                self.ready[k] = [self.outs[k][u][: int(self.tres_np[k, u])] for u in range(self.T)]
            else:
                n, status = int(self.res_np[k, 0]), int(self.res_np[k, 1])
                if status != 0:
                    raise RuntimeError(f"lsmgnn_sample_async of minibatch {b}: status {status}")
                self.ready[k] = [self.glob[k][:n]]
        return self.ready[k][t]

    def part_view(self, t):
        return _PartLists(self, t)

    def close(self):
        self.sampler.close()


class _PartLists:
    """One part's lists of a GpuLists producer (the type's, or the only one)."""

    def __init__(self, prod, t):
        self.prod, self.t = prod, t

    def prefetch(self, b):
        self.prod.prefetch(b)

    def __getitem__(self, b):
        return self.prod.get(b, self.t)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=180)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="rmat-100M-e1.6B-f16x1024",
                    choices=["rmat-s14-e18-f32x128", "rmat-s20-deg16-f32x256", "rmat-10M-e120M-f32x1024",
                             "rmat-20M-e250M-4types", "rmat-100M-e1.6B-f16x1024"],
                    help="workload shape by name")
    ap.add_argument("--first-timed", type=int, default=None,
                    help="first timed minibatch (default: the steady state, max(L+1, 10%% of the configured "
                         "minibatches); the minibatches before the warmup ones fill the cold cache, untimed)")
    ap.add_argument("--cpu-budget", type=float, default=15.0, help="seconds of oracle time for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--host-threads", type=int, default=16,
                    help="host threads copying rows for a store kept in pageable memory")
    ap.add_argument("--policy", default="hybrid", choices=["hybrid", "static", "dynamic", "round_robin"],
                    help="eviction policy: the method's hybrid order or one of the evaluation's alternatives")
    ap.add_argument("--no-ring", action="store_true", help="no victim buffer (and so no PVP level swap)")
    ap.add_argument("--refresh-period", type=int, default=1,
                    help="update period of the dynamic information (1: exact at every gather)")
    ap.add_argument("--victim-mode", default="fifo", choices=["fifo", "queues"],
                    help="victim buffer: one FIFO ring, or per-reuse-iteration queues prefetched into HBM")
    ap.add_argument("--train-us", type=float, default=0.0,
                    help="simulated training step per minibatch: a GPU wait of this length on the caller's "
                         "stream after each minibatch's rows arrive (no memory or link traffic)")
    ap.add_argument("--static", default="indegree", choices=["indegree", "pagerank"],
                    help="static score: the in-degree, or the reverse PageRank computed on the GPU")
    ap.add_argument("--sync", action="store_true",
                    help="blocking lsmgnn_gather per minibatch instead of the pipelined lsmgnn_gather_async")
    ap.add_argument("--gpu-sampler", action="store_true",
                    help="sample each minibatch's request list on the GPU inside the timed region (lsmgnn_sample; "
                         "homogeneous workloads) instead of taking the resident host-generated lists")
    ap.add_argument("--duplex-probe", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--hbm-probe", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--no-duplex-probe", action="store_true",
                    help="skip the link probe with both directions at once (a child process)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU: the library has no multi-GPU path (asked for --gpus "
              f"{args.gpus}). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    if args.duplex_probe:
        duplex_probe()
        return
    if args.hbm_probe:
        hbm_probe()
        return
    if args.gpu_sampler:
        # the sampler's stream is a fifth stream beside the caller's and the
        # library's three: give each its own hardware queue (HIP's default is 4)
        os.environ["GPU_MAX_HW_QUEUES"] = "8"
    # The child process starts before this one touches the GPU.  Not under a
    # profiler: its preloaded library would trace the child too, into the same
    # output files.
    profiled_run = any(k.startswith("ROCPROF") for k in os.environ)
    duplex = None if args.no_duplex_probe or profiled_run else child_probe("--duplex-probe")
    log(f"[bench] duplex link probe: {duplex}")
    hbm = None if profiled_run else child_probe("--hbm-probe")
    log(f"[bench] HBM copy probe: {hbm}")

    import numpy as np
    import torch
    from paper_2407_15264_amd import lsmgnn
    from paper_2407_15264_amd import workload as W

    lsmgnn.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    cfg = W.WORKLOADS[args.workload]
    L = cfg.lookahead if isinstance(cfg, W.HeteroConfig) else cfg.cache.lookahead
    # The timed minibatches start at the steady state: every pass gathers
    # minibatches 0 .. first-1 untimed from fresh caches (the cold-start fill,
    # then the W warmup steps), then times K steps.
    first = steady_start(cfg, L) if args.first_timed is None else args.first_timed
    first = max(first, args.warmup)
    if first + args.steps > cfg.batches:
        print(f"bench.py: minibatches {first}..{first + args.steps - 1} needed, the workload has {cfg.batches}",
              file=sys.stderr)
        sys.exit(2)
    # the minibatches the timed stream gathers or announces (a prefix of the
    # configured run); near the run's end the last gathers announce nothing
    nb = min(cfg.batches, first + args.steps + L + 1)
    if args.static == "pagerank" and isinstance(cfg, W.HeteroConfig):
        print("bench.py: --static pagerank is for the homogeneous workloads", file=sys.stderr)
        sys.exit(2)
    t0 = time.perf_counter()
    parts, requests = make_parts(W, cfg, nb)
    log(f"[bench] workload {cfg.name}: {nb} minibatches generated in {time.perf_counter() - t0:.1f}s "
        f"(mean {requests:.0f} requests)")
    pinned = W.pin_plan([p["num_nodes"] * p["R"] for p in parts],
                        sum(p["shape"].victim_rows * p["R"] for p in parts))
    for p, pin in zip(parts, pinned):
        p["pinned"] = pin
        if pin:
            p["store"] = lsmgnn.PinnedBuffer(p["num_nodes"] * p["R"])
            p["store_np"] = p["store"].numpy(np.uint8, (p["num_nodes"], p["R"]))
        else:  # beyond the pinned-memory budget: ordinary memory, rows copied by the library's host threads
            p["store_np"] = np.empty((p["num_nodes"], p["R"]), np.uint8)
            p["store"] = p["store_np"]
        # in slices of about 8 GiB, with a progress line for each of a large store
        step = max(1, (8 << 30) // p["R"])
        for v0 in range(0, p["num_nodes"], step):
            v1 = min(p["num_nodes"], v0 + step)
            W.fill_features(p["store_np"][v0:].ctypes.data, p["dim"], p["elt"], v0, v1, p["seed"])
            if p["num_nodes"] > step:
                log(f"[bench]   {p['label']}: store rows {v1} of {p['num_nodes']} filled")
    log(f"[bench] stores filled: {sum(p['num_nodes'] * p['R'] for p in parts) / 2**30:.2f} GiB "
        f"({'pinned' if all(pinned) else 'pinned per part: ' + str(pinned)})")

    pinned_parts = [p for p in parts if p["pinned"]]
    if pinned_parts:
        big = max(pinned_parts, key=lambda p: p["num_nodes"] * p["R"])
        cbuf, cbytes = big["store"], big["num_nodes"] * big["R"]
    else:
        cbytes = 1 << 30
        cbuf = lsmgnn.PinnedBuffer(cbytes)
    ceil = measure_ceilings(torch, lsmgnn, cbuf.ptr, cbytes, duplex, hbm)
    log(f"[bench] ceilings: {json.dumps({k: round(v, 1) if isinstance(v, float) else v for k, v in ceil.items()})}")

    dev = torch.device("cuda", 0)
    static_info = {"kind": "in-degree"}
    if args.static == "pagerank":
        g = parts[0]["graph"]
        off_t = torch.as_tensor(g.offsets).to(dev)
        adj_t = torch.as_tensor(g.adj.view(np.int32)).to(dev)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        sc = lsmgnn.pagerank_scores(off_t, adj_t, 0.85, 20)
        torch.cuda.synchronize()
        static_info = {"kind": "reverse PageRank (d = 0.85, 20 iterations) on the GPU",
                       "ms": 1e3 * (time.perf_counter() - t0)}
        parts[0]["static"] = sc.cpu().numpy().view(np.uint32).copy()
        del off_t, adj_t, sc
        log(f"[bench] reverse-PageRank static scores in {static_info['ms']:.1f} ms")
    sampler_info = None
    if args.gpu_sampler:
        sampler_info = gpu_sampler_check(torch, lsmgnn, W, parts, cfg, L, nb, first, args.steps, dev)
        log(f"[bench] GPU sampler: {sampler_info}")
        producer = GpuLists(torch, lsmgnn, parts[0], cfg, L, max(1, max(b.size for p in parts for b in p["batches"])),
                            dev, side_stream(torch), ahead=SAMPLE_AHEAD, typed=len(parts) > 1)
    for t, p in enumerate(parts):
        if args.gpu_sampler:
            p["dev_batches"] = producer.part_view(t)
        else:
            p["dev_batches"] = [torch.as_tensor(np.asarray(b, np.int64)).to(dev) for b in p["batches"]]
        p.pop("graph", None)
        mb = max(1, max(b.size for b in p["batches"]))
        # three output sets rotate: at most two gathers are in flight
        p["bufs"] = [(torch.empty(mb * p["R"], dtype=torch.uint8, device=dev),
                      torch.empty(mb, dtype=torch.int64, device=dev),
                      torch.empty(mb, dtype=torch.int64, device=dev)) for _ in range(3)]

    def fresh_caches():
        """A new cache per part (the previous one closed first), its window
        holding the first L+1 minibatches."""
        for p in parts:
            if "cache" in p:
                p["cache"].close()
            sh = p["shape"]
            mb = p["bufs"][0][1].numel()
            p["cache"] = lsmgnn.FeatureCache(p["num_nodes"], p["R"], p["store"], p["static"], sh.num_sets,
                                             0 if args.no_ring else sh.victim_rows, sh.lookahead, mb,
                                             near_threshold=sh.near_threshold, pageable=not p["pinned"],
                                             host_threads=args.host_threads, policy=args.policy,
                                             victim_mode=args.victim_mode, refresh_period=args.refresh_period)
            for j in range(L + 1):
                p["cache"].advance(p["dev_batches"][j])
            p["tickets"] = {}

    sleep_cycles = 0
    if args.train_us > 0:
        # calibrate the device wait: cycles per microsecond of torch's spin kernel
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(1000000)
        e0.record()
        torch.cuda._sleep(10000000)
        e1.record()
        torch.cuda.synchronize()
        sleep_cycles = int(args.train_us * 10000000 / (1e3 * e0.elapsed_time(e1)))
        log(f"[bench] simulated training step: {args.train_us:.0f} us = {sleep_cycles} spin cycles")

    def step(b):
        nbytes = 0
        for p in parts:
            c, db = p["cache"], p["dev_batches"]
            if args.gpu_sampler and b + L + 1 + SAMPLE_AHEAD < nb:
                db.prefetch(b + L + 1 + SAMPLE_AHEAD)  # sampled ahead on its own stream
            out, uniq, inv = p["bufs"][b % 3]
            if args.sync:
                r = c.gather(db[b], out=out, unique=uniq, inverse=inv)
                if b + L + 1 < nb:
                    c.advance(db[b + L + 1])
            else:  # gather minibatch b and announce minibatch b+L+1 in one call
                p["tickets"][b], r = c.gather_async(db[b], out, uniq, inverse=inv,
                                                    announce=db[b + L + 1] if b + L + 1 < nb else None)
            nbytes += r.n_unique * p["R"]
        if not args.sync:
            for p in parts:
                if b - 1 in p["tickets"]:
                    p["cache"].wait(p["tickets"].pop(b - 1))  # a consumer of minibatch b-1 would run after this
        if sleep_cycles:  # the training step that consumes minibatch b-1 (or b, with blocking calls)
            torch.cuda._sleep(sleep_cycles)
        return nbytes

    def drain():
        for p in parts:
            for b in list(p["tickets"]):
                p["cache"].wait(p["tickets"].pop(b))

    def run_pass(profiled, per_gather=False):
        """Fresh caches, the cold-start fill and the W warmup minibatches, then
        K timed ones; with `profiled` the library records HIP events around
        every row copy.  With `per_gather` the counts of the latest counted
        gather are read after every step (a call that waits for the queued
        work: not for timing)."""
        fresh_caches()
        for b in range(first):
            step(b)
        drain()
        tot0 = [p["cache"].stats()[1] for p in parts]
        for p in parts:
            p["cache"].set_profiling(profiled)
        per = [dict() for _ in parts]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        nbytes = 0
        for b in range(first, first + args.steps):
            nbytes += step(b)
            if per_gather:
                for p, pp in zip(parts, per):
                    last = p["cache"].stats()[0]
                    pp[last["batch"]] = last
        drain()
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        profs = [p["cache"].profile() for p in parts] if profiled else None
        for p, pp in zip(parts, per):
            p["cache"].set_profiling(False)
            if per_gather:
                last = p["cache"].stats()[0]
                pp[last["batch"]] = last
        tot1 = [p["cache"].stats()[1] for p in parts]
        d = {k: sum(t1[k] - t0_[k] for t0_, t1 in zip(tot0, tot1)) for k in tot1[0]}
        return dt, nbytes, d, profs, per

    # The headline pass runs as a user would, without the library's timing
    # events (each is a marker on a stream of the pipeline and costs a few
    # percent).  A second pass over the same minibatches, from fresh caches,
    # records the events for the per-kernel figures.
    dt, nbytes, d, _, _ = run_pass(False)
    log(f"[bench] timed pass: {args.steps} minibatches in {1e3 * dt:.1f} ms")
    dt_p, nbytes_p, d_p, profs, _ = run_pass(True)
    log(f"[bench] profiled pass: {1e3 * dt_p:.1f} ms")
    # a third, untimed pass reads every gather's counts
    _, nbytes_c, d_c, _, per = run_pass(False, per_gather=True)
    assert nbytes_p == nbytes == nbytes_c and d_p == d == d_c, "the passes over one stream must do identical work"
    alone = hit_path_alone(parts, first + args.steps - 1)
    # per-minibatch rates over the timed gathers (all parts of a minibatch summed)
    timed = [b for b in range(first, first + args.steps) if all(b in pp for pp in per)]

    def spread(key):
        v = sorted(sum(pp[b][key] for pp in per) / max(sum(pp[b]["unique"] for pp in per), 1) for b in timed)
        if not v:
            return None
        q = lambda f: v[min(len(v) - 1, int(f * len(v)))]  # noqa: E731
        return {"min": v[0], "p10": q(0.1), "median": q(0.5), "p90": q(0.9), "max": v[-1]}
    per_minibatch = {"gathers": len(timed), "hit_rate": spread("hits"), "victim_hit_rate": spread("victim_hits"),
                     "miss_rate": spread("misses")}
    gbps = nbytes / dt / 1e9
    rows = d["unique"]

    # per-kernel rates from HIP events on the gather streams, summed over the parts
    kern = {}
    for name, key, per_row, bound in (
            ("hbm_copy", "hbm_copy", 2, "hbm"),
            ("host_fetch", "host_fetch", 1, "host_link"),
            ("ring_write_dma", "enqueue", 1, "host_link"),
            ("fill", "fill", 2, "hbm"),
            ("prefetch", "prefetch", 1, "host_link")):
        ms = sum(pr[key + "_ms"] for pr in profs)
        rows_k = sum(pr[key + "_rows"] for pr in profs)
        kbytes = sum(pr[key + "_rows"] * per_row * p["R"] for pr, p in zip(profs, parts))
        launches = max(sum(pr[key + "_launches"] for pr in profs), 1)
        kern[name] = dict(ms_total=ms, launches=launches, rows=rows_k, avg_us=1e3 * ms / launches,
                          bytes_per_launch=kbytes / launches,
                          GBps=(kbytes / (ms / 1e3) / 1e9) if ms > 0 else 0.0, bound=bound,
                          launches_per_minibatch=launches / args.steps,
                          us_per_minibatch=1e3 * ms / args.steps,
                          # busy time per minibatch over the profiled pass's own step time
                          share_of_step=ms / (1e3 * dt_p))
    kern["ring_write_dma"]["engine"] = "runtime copy (hipMemcpyAsync of the staged rows), not one of our kernels"
    hc_ms = sum(pr["host_copy_ms"] for pr in profs)
    if hc_ms > 0:
        hc_bytes = sum(pr["host_copy_rows"] * p["R"] for pr, p in zip(profs, parts))
        kern["host_copy"] = dict(ms_total=hc_ms, rows=sum(pr["host_copy_rows"] for pr in profs),
                                 GBps=hc_bytes / (hc_ms / 1e3) / 1e9, bound="host_memory",
                                 engine=f"{args.host_threads} host threads (pageable store -> pinned bounce), "
                                        "wall time")
    dom = max((k for k in kern if "engine" not in kern[k]), key=lambda k: kern[k]["ms_total"])
    kd = kern[dom]
    link_peak = max(ceil["dma_h2d_GBps"], ceil["zero_copy_read_GBps"])
    if kd["bound"] == "hbm":
        roof = {"bound": "hbm", "achieved": kd["GBps"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": kd["GBps"] / HBM_PEAK_GBPS, "traffic": None}
    else:
        peak = link_peak if dom == "host_fetch" else max(ceil["dma_d2h_GBps"], ceil["zero_copy_write_GBps"])
        roof = {"bound": "host_link", "achieved": kd["GBps"], "peak": peak, "unit": "GB/s",
                "frac": kd["GBps"] / peak, "traffic": None,
                "peak_source": "measured in this run (best of pinned DMA and zero-copy kernel)",
                "frac_of_published_pcie5_x16": kd["GBps"] / PCIE5_X16_PEAK_GBPS}
    roof.update(kernel=dom, avg_launch_us=kd["avg_us"], bytes_per_launch=kd["bytes_per_launch"],
                launches_per_minibatch=kd["launches_per_minibatch"], us_per_minibatch=kd["us_per_minibatch"],
                share_of_step=kd["share_of_step"])
    if kd["bound"] == "host_link":
        # both link directions over the headline pass: rows in (host fetch,
        # prefetch) and rows out (ring writes), against the duplex ceiling
        b_in = sum((pr["host_fetch_rows"] + pr["prefetch_rows"]) * p["R"] for pr, p in zip(profs, parts))
        b_out = sum(pr["enqueue_rows"] * p["R"] for pr, p in zip(profs, parts))
        roof["link_both_directions"] = {
            "in_GBps": b_in / dt / 1e9, "out_GBps": b_out / dt / 1e9, "total_GBps": (b_in + b_out) / dt / 1e9,
            "frac_of_duplex_total": None if ceil["duplex"] is None else
            (b_in + b_out) / dt / 1e9 / ceil["duplex"]["total_GBps"]}
    tr = recorded_traffic(cfg.name, dom)
    if tr is not None:
        # algorithmic bytes of the launch on both sides of the copy (read + write)
        alg = kd["bytes_per_launch"] * (1 if kd["bound"] == "hbm" else 2)
        roof["traffic"] = tr["bytes"]
        roof["traffic_detail"] = dict(tr, algorithmic_read_plus_write=alg, ratio=tr["bytes"] / alg)
    hb = kern["hbm_copy"]
    trh = recorded_traffic(cfg.name, "hbm_copy")
    roof_hbm = {"bound": "hbm", "kernel": "hbm_copy (hit rows cache->out)", "achieved": hb["GBps"],
                "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": hb["GBps"] / HBM_PEAK_GBPS,
                "frac_of_measured_d2d": hb["GBps"] / ceil["hbm_copy_GBps"] if ceil["hbm_copy_GBps"] else None,
                "avg_launch_us": hb["avg_us"],
                "bytes_per_launch": hb["bytes_per_launch"],
                "traffic": None if trh is None else trh["bytes"],
                "target_frac": HIT_PATH_TARGET_FRAC,
                "gap_to_target": HIT_PATH_TARGET_FRAC - hb["GBps"] / HBM_PEAK_GBPS,
                "alone": dict(alone, frac_of_measured_d2d=alone["achieved"] / ceil["hbm_copy_GBps"]
                              if ceil["hbm_copy_GBps"] else None)}

    res = {
        "metric": METRIC, "value": gbps, "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": 1e3 * dt / args.steps, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int64", "data": "synthetic",
        "config": dict(cfg.describe(), feature_dtype="fp32" if cfg.elt_bytes == 4 else "fp16",
                       minibatches_timed=args.steps, policy=args.policy, static_score=static_info,
                       victim_ring="off" if args.no_ring else "on", victim_mode=args.victim_mode,
                       refresh_period=args.refresh_period,
                       simulated_training_us=args.train_us,
                       requests=(f"sampled on the GPU inside the timed region (lsmgnn_sample_async on a stream "
                                 f"of its own, {SAMPLE_AHEAD} minibatches before their announcement)"
                                 if args.gpu_sampler
                                 else "host-generated, resident in HBM before the timed region"),
                       first_timed_minibatch=first,
                       cold_start_fill_minibatches=first - args.warmup,
                       api=("lsmgnn_gather + lsmgnn_advance" if args.sync
                            else "lsmgnn_gather_async with announcement (two minibatches in flight)")),
        "rows_per_s": rows / dt,
        "parts": len(parts),
        "hit_rate": d["hits"] / max(d["unique"], 1),
        "victim_hit_rate": d["victim_hits"] / max(d["unique"], 1),
        "miss_rate": d["misses"] / max(d["unique"], 1),
        # the same outcomes per raw request (a repeated ID counts each time)
        "request_hit_rate": d["request_hits"] / max(d["requests"], 1),
        "request_victim_hit_rate": d["request_victim_hits"] / max(d["requests"], 1),
        "request_miss_rate": 1.0 - (d["request_hits"] + d["request_victim_hits"]) / max(d["requests"], 1),
        # where the victim hits' rows were read (all from the victim buffer):
        # the pinned ring over the link, the previous gather's staged rows in
        # HBM, the cache row of a line evicted earlier in the same gather, or
        # (queues) the HBM prefetch buffer
        "victim_hit_rows": {k[len("victim_rows_"):]: d[k] for k in ("victim_rows_ring", "victim_rows_staged",
                                                                  "victim_rows_cache", "victim_rows_prefetched")},
        "per_minibatch": per_minibatch,
        "unique_per_minibatch": d["unique"] / args.steps,
        "requests_per_minibatch": d["requests"] / args.steps,
        "roofline": roof,
        "roofline_hbm": roof_hbm,
        "kernels": {k: {kk: (round(vv, 4) if isinstance(vv, float) else vv) for kk, vv in v.items()}
                    for k, v in kern.items()},
        "gather_ms_events": sum(pr["gather_ms"] for pr in profs) / max(sum(pr["gathers"] for pr in profs), 1),
        "ceilings": ceil,
        "gpu_sampler": sampler_info,
        "profiled_pass": {"value": nbytes_p / dt_p / 1e9, "ms_per_step": 1e3 * dt_p / args.steps,
                          "how": "the same minibatches from fresh caches with the library's HIP timing "
                                 "events on; `kernels` and the rooflines come from this pass, `value` "
                                 "from the pass without them"},
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(parts, args.cpu_budget, first, args.policy,
                                           0 if args.no_ring else None, args.victim_mode, args.refresh_period)
        res["cpu_baseline"]["gpu_over_cpu"] = gbps / res["cpu_baseline"]["value"]
    for p in parts:
        p["cache"].close()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
