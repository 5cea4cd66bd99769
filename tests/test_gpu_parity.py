"""GPU <-> oracle parity through the C ABI (needs an MI355X).

Every case drives the GPU library and the CPU oracle with the same seeded
stream and requires identical unique IDs, inverse, per-ID outcomes, counters,
rows (bit-exact) and final cache/ring state.  Cases: the two smaller workload
shapes end to end, randomized small caches, adversarial streams (one set,
duplicates, single IDs, ragged ID ranges, empty batches, batches larger than
the cache, L = 0, V = 0 and 1, n = max_batch), error paths that must leave the
state unchanged, determinism, and provenance (hits come from HBM, misses from
the backing store).
"""
import time

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from paper_2407_15264_amd import lsmgnn  # noqa: E402
from paper_2407_15264_amd import workload as W  # noqa: E402
from tests.parity_driver import (Store, compare_state, config_stream, device_store, log,  # noqa: E402
                                 run_async_parity, run_mixed_parity, run_parity, run_typed_async_parity)
from oracle.oracle import Oracle  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lsmgnn.lib()


def test_workload_rmat14_full_parity():
    cfg = W.CONFIGS[W.RMAT14]
    log(f"case: {cfg.name}, all {cfg.batches} gathers, all rows")
    wl, batches = config_stream(cfg)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    res = run_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead, batches,
                     rows="all", state_every=5, label=cfg.name)
    tot = res["total"]
    assert tot["victim_hits"] > 0 and tot["enqueued"] > 0


@pytest.mark.timeout(600)
def test_workload_rmat20_parity():
    cfg = W.CONFIGS[W.RMAT20]
    log(f"case: {cfg.name}, all {cfg.batches} gathers; rows vs oracle every 20th gather, "
        f"vs the backing store on the GPU for every gather")
    wl, batches = config_stream(cfg)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    store_gpu = torch.from_numpy(store.np).to("cuda")
    res = run_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead, batches,
                     rows=20, state_every=50, label=cfg.name, store_gpu=store_gpu)
    tot = res["total"]
    log(f"  {cfg.name}: {tot}")
    assert tot["victim_hits"] > 0 and tot["hits"] > 0


@pytest.mark.timeout(1500)
def test_workload_rmat10m_full_size_pipelined_parity():
    """The 10M-node workload at full size (41 GB pinned store, 8 GiB cache,
    4 GiB ring, 500 minibatches of 4096 seeds) in the bench's launch
    configuration.  Every gather: unique IDs, inverse and outcomes against the
    oracle, rows against the backing store (a device copy); every 50th gather:
    rows against the oracle's; every 100th and at the end: cache and ring
    state; at the end: all counters."""
    cfg = W.CONFIGS[W.RMAT10M]
    log(f"case: {cfg.name}, all {cfg.batches} gathers, pipelined, full size")
    t0 = time.time()
    wl, batches = config_stream(cfg)
    log(f"  workload generated in {time.time() - t0:.1f} s (max batch {wl.max_batch})")
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    sg = device_store(store)
    log(f"  store filled and copied to the device ({time.time() - t0:.1f} s)")
    res = run_async_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead,
                           batches, rows=50, store_gpu=sg, state_every=100, label=cfg.name)
    tot = res["total"]
    log(f"  {cfg.name}: {tot} in {res['seconds']:.1f} s")
    assert tot["hits"] > 0 and tot["victim_hits"] > 0 and tot["misses"] > 0
    del sg
    torch.cuda.empty_cache()
    # the GPU sampler on the full-size graph gives the same request lists
    off = torch.as_tensor(wl.graph.offsets).cuda()
    adj = torch.as_tensor(wl.graph.adj.view(np.int32)).cuda()
    smp = lsmgnn.GpuSampler(off, adj, cfg.fanout, seed=cfg.seed)
    seeds = torch.as_tensor(wl.seeds).cuda()
    out = torch.empty(wl.max_batch, dtype=torch.int64, device="cuda")
    B = cfg.batch_size
    for b in list(range(8)) + [cfg.batches - 1]:
        got = smp.sample(seeds[b * B:(b + 1) * B], b, out).cpu().numpy()
        assert np.array_equal(got, batches[b]), f"GPU sampler, minibatch {b}"
    log(f"  GPU sampler: minibatches 0-7 and {cfg.batches - 1} identical to the generated lists")
    smp.close()
    del off, adj, seeds, out
    torch.cuda.empty_cache()


@pytest.mark.timeout(2400)
def test_workload_typed_20m_full_size_pipelined_parity():
    """The typed 20M-node workload at full size: four node types with their own
    feature widths, caches and rings (56 GB of pinned stores, 32 GiB of caches,
    16 GiB of rings, 500 minibatches of 8192 seeds), one cache per type, all in
    the bench's launch configuration.  Checks as for the 10M-node workload,
    per type."""
    cfg = W.HETERO[W.TYPED20M]
    log(f"case: {cfg.name}, all {cfg.batches} gathers per type, pipelined, full size")
    t0 = time.time()
    wl = W.HeteroWorkload(cfg)
    type_batches = [wl.type_batches(t) for t in range(cfg.num_types)]
    log(f"  workload generated in {time.time() - t0:.1f} s")
    shapes = [cfg.cache_shape(t) for t in range(cfg.num_types)]
    pinned = W.pin_plan([cfg.store_bytes(t) for t in range(cfg.num_types)],
                        sum(sh.victim_rows * cfg.row_bytes(t) for t, sh in enumerate(shapes)))
    log(f"  pinned stores: {pinned} (the others pageable)")
    stores = [Store(n, d, cfg.elt_bytes, cfg.seed + 1 + t, pinned=pinned[t])
              for t, (n, d) in enumerate(zip(cfg.type_counts(), cfg.dims))]
    sg = [device_store(st) for st in stores]
    log(f"  stores filled and copied to the device ({time.time() - t0:.1f} s)")
    res = run_typed_async_parity(stores, wl.static, shapes, type_batches, rows=50, stores_gpu=sg, state_every=100,
                                 label=cfg.name)
    for t, tot in enumerate(res["totals"]):
        log(f"  {cfg.name} type {t}: {tot}")
        assert tot["hits"] > 0 and tot["misses"] > 0
    log(f"  {res['seconds']:.1f} s")
    del sg
    torch.cuda.empty_cache()
    # the GPU sampler and the split by type give the per-type lists
    off = torch.as_tensor(wl.graph.offsets).cuda()
    adj = torch.as_tensor(wl.graph.adj.view(np.int32)).cuda()
    smp = lsmgnn.GpuSampler(off, adj, cfg.fanout, seed=cfg.seed)
    seeds = torch.as_tensor(wl.seeds).cuda()
    node_type = torch.as_tensor(wl.node_type).cuda()
    local = torch.as_tensor(wl.node_local.astype(np.int32)).cuda()
    mb = int(np.diff(wl.offsets).max())
    glob = torch.empty(mb, dtype=torch.int64, device="cuda")
    outs = [torch.empty(mb, dtype=torch.int64, device="cuda") for _ in range(cfg.num_types)]
    work = torch.empty(lsmgnn.split_work_bytes(mb, cfg.num_types), dtype=torch.uint8, device="cuda")
    res_h = lsmgnn.PinnedBuffer(8 * (cfg.num_types + 1))
    r = res_h.numpy(np.uint64, (cfg.num_types + 1,))
    B = cfg.batch_size
    for b in list(range(4)) + [cfg.batches - 1]:
        lst = smp.sample(seeds[b * B:(b + 1) * B], b, glob)
        lsmgnn.split_by_type_async(lst, node_type, local, outs, work, res_h.ptr)
        torch.cuda.current_stream().synchronize()
        assert int(r[cfg.num_types]) == 0, b
        for t in range(cfg.num_types):
            got = outs[t][: int(r[t])].cpu().numpy()
            assert np.array_equal(got, type_batches[t][b]), f"minibatch {b}, type {t}"
    log(f"  GPU sampler + split by type: minibatches 0-3 and {cfg.batches - 1} identical per type")
    smp.close()
    res_h.close()


def _random_case(seed):
    rng = np.random.default_rng(5000 + seed)
    n = int(rng.choice([1, 7, 33, 100, 1000, 5000, 70001]))
    S = int(rng.choice([1, 2, 3, 5, 16, 61, 400]))
    V = int(rng.choice([0, 1, 2, 7, 64, 1000]))
    L = int(rng.choice([0, 1, 2, 4, 8, 16, 31]))
    T = int(rng.choice([0, 0, 1, 2, 3]))
    rb = int(rng.choice([16, 48, 64, 512]))
    nb = int(rng.integers(1, 12))
    bmax = int(rng.choice([1, 5, 40, 300, 3000]))
    stat = rng.integers(0, rng.choice([1, 3, 1000]), n).astype(np.uint32)
    batches = [rng.integers(0, n, rng.integers(0, bmax + 1)) for _ in range(nb)]
    if rng.random() < 0.5:
        announce = [rng.integers(0, n, rng.integers(0, bmax + 1)) for _ in range(nb + L)]
    else:
        announce = batches
    return n, S, V, L, T, rb, stat, batches, announce


@pytest.mark.parametrize("seed", range(40))
def test_random_small_caches(seed):
    n, S, V, L, T, rb, stat, batches, announce = _random_case(seed)
    log(f"case: random seed {seed}: N={n} S={S} V={V} L={L} T={T} R={rb} batches={len(batches)}")
    store = Store.random_bytes(n, rb, seed)
    run_parity(store, stat, S, V, L, batches, announce, near_threshold=T, rows="all", label=f"random{seed}")


def _adversarial():
    rng = np.random.default_rng(7)
    cases = {}
    # every request maps to one set
    cases["one_set"] = dict(n=64, S=1, V=8, L=3, batches=[rng.integers(0, 64, 30) for _ in range(10)])
    # heavy duplication
    cases["duplicates"] = dict(n=1000, S=4, V=4, L=2,
                               batches=[np.repeat(rng.integers(0, 1000, 3), 1000) for _ in range(6)])
    cases["single_ids"] = dict(n=50, S=2, V=2, L=2, batches=[np.array([i % 7]) for i in range(20)])
    # top of the ID range and a ragged bitmap tail
    top = (1 << 20) + 37
    cases["id_top"] = dict(n=top, S=64, V=16, L=2,
                           batches=[np.array([top - 1, top - 2, 0, top - 33, top - 1] * 3)
                                    for _ in range(4)] + [rng.integers(top - 3000, top, 2000)])
    cases["no_window"] = dict(n=3000, S=16, V=64, L=0, batches=[rng.integers(0, 3000, 500) for _ in range(8)])
    cases["no_ring"] = dict(n=3000, S=16, V=0, L=4, batches=[rng.integers(0, 3000, 500) for _ in range(8)])
    cases["ring_of_one"] = dict(n=300, S=4, V=1, L=4, batches=[rng.integers(0, 300, 80) for _ in range(12)])
    cases["batch_exceeds_cache"] = dict(n=100000, S=4, V=100, L=3,
                                        batches=[rng.integers(0, 100000, 5000) for _ in range(6)])
    cases["empty_batches"] = dict(n=500, S=8, V=8, L=2,
                                  batches=[np.array([], np.int64), rng.integers(0, 500, 100), np.array([], np.int64),
                                           rng.integers(0, 500, 100), rng.integers(0, 500, 100)])
    cases["single_node"] = dict(n=1, S=1, V=1, L=1, batches=[np.zeros(5, np.int64), np.zeros(1, np.int64)] * 3)
    cases["big_batch"] = dict(n=1 << 22, S=4096, V=20000, L=4,
                              batches=[rng.integers(0, 1 << 22, 1 << 20) for _ in range(3)])
    # one set receiving about 10^5 unique IDs per gather (its segment is
    # ordered by a block's radix sort, linear in the set's size)
    cases["one_set_large"] = dict(n=300000, S=1, V=5000, L=2,
                                  batches=[rng.integers(0, 300000, 150000) for _ in range(3)])
    # sets on both sides of the size at which a set's segment is sorted by a block
    cases["sets_near_sort_threshold"] = dict(n=50000, S=200, V=2000, L=3,
                                             batches=[rng.integers(0, 50000, 13000) for _ in range(4)])
    return cases


@pytest.mark.parametrize("name", sorted(_adversarial().keys()))
def test_adversarial_streams(name):
    c = _adversarial()[name]
    log(f"case: adversarial {name}: N={c['n']} S={c['S']} V={c['V']} L={c['L']}")
    rb = 64 if c["n"] < (1 << 21) else 16
    store = Store.random_bytes(c["n"], rb, 1)
    stat = np.random.default_rng(3).integers(0, 5, c["n"]).astype(np.uint32)
    mb = max(1, max(len(b) for b in c["batches"]))
    run_parity(store, stat, c["S"], c["V"], c["L"], c["batches"], rows="all", max_batch=mb, label=name)


def test_errors_leave_state_unchanged():
    log("case: error paths")
    n, S, V, L = 200, 4, 8, 1
    store = Store.random_bytes(n, 32, 2)
    stat = np.arange(n, dtype=np.uint32) % 5
    cache = lsmgnn.FeatureCache(n, 32, store.buf, stat, S, V, L, 64)
    orc = Oracle(n, 32, stat, S, V, L, store=store.np)
    dev = lambda a: torch.as_tensor(np.asarray(a, np.int64)).cuda()  # noqa: E731
    a0, a1 = np.arange(0, 40), np.arange(20, 60)
    for a in (a0, a1):
        cache.advance(dev(a))
        orc.advance(a)
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        cache.advance(dev([1]))
    assert e.value.status == "E_WINDOW"
    r = cache.gather(dev(a0), outcome=True)
    orc.gather(a0)
    before = cache.export_state()
    for bad in ([0, 200], [-1, 3], [199, 1 << 40]):
        with pytest.raises(lsmgnn.LsmgnnError) as e:
            cache.gather(dev(bad))
        assert e.value.status == "E_RANGE"
        with pytest.raises(lsmgnn.LsmgnnError) as e:
            cache.advance(dev(bad))
        assert e.value.status == "E_RANGE"
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        cache.gather(dev(np.zeros(65)))
    assert e.value.status == "E_INVAL"
    after = cache.export_state()
    assert after["t"] == before["t"] and np.array_equal(after["tags"], before["tags"])
    assert np.array_equal(after["ring_tags"], before["ring_tags"])
    # the stream continues exactly like the oracle's after the rejected calls
    cache.advance(dev(a1))
    orc.advance(a1)
    r = cache.gather(dev(a1), outcome=True)
    o = orc.gather(a1)
    assert np.array_equal(r.outcome.cpu().numpy(), o["outcome"])
    assert np.array_equal(r.out.cpu().numpy(), o["out"])
    compare_state(cache, orc, "after errors")
    r = cache.gather(dev([]))
    assert r.n_unique == 0 and cache.stats()[0]["unique"] == 0
    cache.close()


def test_bad_configs_rejected():
    store = Store.random_bytes(16, 16, 0)
    stat = np.ones(16, np.uint32)
    base = dict(num_nodes=16, row_bytes=16, host_store=store.buf, static_score=stat, num_sets=2, victim_rows=2,
                lookahead=1, max_batch=8)
    for bad in (dict(num_sets=0), dict(row_bytes=24), dict(lookahead=32), dict(max_batch=0), dict(num_nodes=0)):
        kw = dict(base, **bad)
        with pytest.raises(lsmgnn.LsmgnnError) as e:
            lsmgnn.FeatureCache(**kw)
        assert e.value.status == "E_INVAL", bad
    pageable = np.zeros(16 * 16, np.uint8)
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        lsmgnn.FeatureCache(**dict(base, host_store=pageable.ctypes.data))
    assert e.value.status == "E_INVAL"
    # cache rows beyond the device memory: 2^31 lines of 4 KiB (8 TiB)
    big = Store.random_bytes(16, 4096, 0)
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        lsmgnn.FeatureCache(**dict(base, host_store=big.buf, row_bytes=4096, num_sets=1 << 28))
    assert e.value.status == "E_NOMEM"


def test_deterministic_state():
    cfg = W.CONFIGS[W.RMAT14]
    wl, batches = config_stream(cfg)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes)
    states = []
    for rep in range(2):
        log(f"case: determinism run {rep}")
        c = lsmgnn.FeatureCache(cfg.num_nodes, cfg.row_bytes, store.buf, wl.static, cfg.cache.num_sets,
                                cfg.cache.victim_rows, cfg.cache.lookahead, wl.max_batch)
        dev = [torch.as_tensor(b).cuda() for b in batches]
        for j in range(cfg.cache.lookahead + 1):
            c.advance(dev[j])
        for b in range(len(batches)):
            c.gather(dev[b])
            if b + cfg.cache.lookahead + 1 < len(batches):
                c.advance(dev[b + cfg.cache.lookahead + 1])
        states.append(c.export_state())
        c.close()
    assert np.array_equal(states[0]["tags"], states[1]["tags"])
    assert np.array_equal(states[0]["ring_tags"], states[1]["ring_tags"])


def test_provenance_hits_from_hbm_misses_from_store():
    """After warm-up, overwrite the backing-store rows of every resident line
    with a sentinel: hits must still return the original bytes (served from
    HBM), while misses of non-resident nodes return the sentinel (served from
    the store)."""
    log("case: provenance")
    n, S, rb = 4096, 64, 64
    store = Store.random_bytes(n, rb, 11)
    orig = store.np.copy()
    stat = np.ones(n, np.uint32)
    cache = lsmgnn.FeatureCache(n, rb, store.buf, stat, S, 0, 0, 1024)
    warm = np.arange(0, 4096, 9)
    cache.gather(torch.as_tensor(warm).cuda())
    tags = cache.export_state()["tags"]
    resident = tags[tags != lsmgnn.EMPTY].astype(np.int64)
    absent = np.setdiff1d(np.arange(n), resident)[:200]
    store.np[resident] = 0xAB
    store.np[absent] = 0xCD
    # hits alone (a hit changes nothing, so every probed line stays resident)
    r = cache.gather(torch.as_tensor(resident[:300]).cuda(), outcome=True)
    uq = r.unique.cpu().numpy()
    assert (r.outcome.cpu().numpy() == lsmgnn.HIT).all()
    assert np.array_equal(r.out.cpu().numpy(), orig[uq])
    # then misses alone
    r = cache.gather(torch.as_tensor(absent).cuda(), outcome=True)
    assert (r.outcome.cpu().numpy() == lsmgnn.MISS).all()
    assert (r.out.cpu().numpy() == 0xCD).all()
    cache.close()


def _victim_stream(seed, n, nb, size):
    """Minibatches drawn from a skewed popularity (hot nodes reappear within
    the window, so lines evicted with an announced reuse return as victim
    hits)."""
    rng = np.random.default_rng(seed)
    p = 1.0 / np.arange(1, n + 1) ** 0.6
    p /= p.sum()
    perm = rng.permutation(n)
    return [perm[rng.choice(n, size=size, p=p)].astype(np.int64) for _ in range(nb)]


@pytest.mark.parametrize("policy", ["hybrid", "round_robin"])
@pytest.mark.parametrize("pageable", [False, True])
@pytest.mark.parametrize("pipelined", [False, True])
def test_victim_rows_come_from_the_victim_buffer(pipelined, pageable, policy):
    """Row provenance of the victim buffer (Sec. 4.3, 4.3.1).  After a warm-up,
    the backing-store row of every node that is not resident in the cache is
    overwritten with a sentinel.  From then on a row's bytes travel with its
    line: a hit or a victim hit must return the bytes the line was loaded with
    (the original ones, unless the node missed since the overwrite and so was
    loaded with the sentinel), and only a miss may read the store.  A victim
    hit served from the backing store would return the sentinel for a line
    loaded before the overwrite.  Victim rows must come from the pinned ring,
    and with the round-robin policy (which evicts lines whose next use is the
    very next minibatch, the hybrid order keeps those) also from the previous
    gather's staged rows."""
    log(f"case: victim-row provenance, pipelined={pipelined}, pageable={pageable}, policy={policy}")
    n, rb, S, V, L = 6000, 64, 32, 300, 4  # the ring wraps every few gathers
    batches = _victim_stream(7, n, 44, 1200)
    store = Store.random_bytes(n, rb, 21, pinned=not pageable)
    expect = store.np.copy()  # the bytes each node's line carries
    stat = np.random.default_rng(3).integers(0, 50, n).astype(np.uint32)
    mb = max(b.size for b in batches)
    cache = lsmgnn.FeatureCache(n, rb, store.buf, stat, S, V, L, mb, pageable=pageable, policy=policy)
    dev = [torch.as_tensor(b).cuda() for b in batches]
    for j in range(L + 1):
        cache.advance(dev[j])
    bufs = [(torch.empty(mb * rb, dtype=torch.uint8, device="cuda"), torch.empty(mb, dtype=torch.int64, device="cuda"),
             torch.empty(mb, dtype=torch.int64, device="cuda"), torch.empty(mb, dtype=torch.uint8, device="cuda"))
            for _ in range(3)]
    POISON, warm = 0xEE, 14
    checked = {"vhit_loaded_before": 0, "gathers": 0}

    def check(r, b):
        uq = r.unique.cpu().numpy()
        oc = r.outcome.cpu().numpy()
        rows = r.out.cpu().numpy()
        if b < warm:
            return
        served = oc != lsmgnn.MISS
        want = np.where(served[:, None], expect[uq], store.np[uq])
        bad = np.flatnonzero((rows != want).any(axis=1))
        assert bad.size == 0, (f"gather {b}: rows of unique idx {bad[:5].tolist()} (outcomes "
                               f"{oc[bad[:5]].tolist()}) are not the bytes their lines carry")
        vh = oc == lsmgnn.VICTIM_HIT
        checked["vhit_loaded_before"] += int((vh & (expect[uq] != POISON).any(axis=1)
                                              & (store.np[uq] == POISON).all(axis=1)).sum())
        checked["gathers"] += 1
        miss = uq[oc == lsmgnn.MISS]
        expect[miss] = store.np[miss]

    pending = []
    for b in range(len(batches)):
        if b == warm:
            # drain, then overwrite the store rows of every non-resident node
            for tk, r, bb in pending:
                cache.wait(tk)
                torch.cuda.current_stream().synchronize()
                check(r, bb)
            pending = []
            cache.sync()
            tags = cache.export_state()["tags"]
            resident = np.unique(tags[tags != lsmgnn.EMPTY]).astype(np.int64)
            poison = np.setdiff1d(np.arange(n), resident)
            store.np[poison] = POISON
        out, uq, inv, oc = bufs[b % 3]
        nxt = dev[b + L + 1] if b + L + 1 < len(batches) else None
        if pipelined:
            tk, r = cache.gather_async(dev[b], out, uq, inverse=inv, outcome=oc, announce=nxt)
            pending.append((tk, r, b))
            if len(pending) == 2:
                tk0, r0, b0 = pending.pop(0)
                cache.wait(tk0)
                torch.cuda.current_stream().synchronize()
                check(r0, b0)
        else:
            r = cache.gather(dev[b], out=out, unique=uq, inverse=inv, outcome=oc)
            if nxt is not None:
                cache.advance(nxt)
            check(r, b)
    for tk, r, bb in pending:
        cache.wait(tk)
        torch.cuda.current_stream().synchronize()
        check(r, bb)
    tot = cache.stats()[1]
    cache.close()
    log(f"  totals {tot}; victim hits on lines loaded before the overwrite: {checked['vhit_loaded_before']}")
    assert checked["gathers"] == len(batches) - warm
    assert checked["vhit_loaded_before"] > 0
    assert tot["victim_rows_ring"] > 0
    if policy == "round_robin":
        assert tot["victim_rows_staged"] > 0
    assert (tot["victim_rows_ring"] + tot["victim_rows_staged"] + tot["victim_rows_cache"]
            + tot["victim_rows_prefetched"] == tot["victim_hits"])


def _run_async_parity(store, static, S, V, L, batches, label, combined=True):
    run_async_parity(store, static, S, V, L, batches, rows="all", label=label, combined=combined)


def test_async_pipeline_rmat14():
    cfg = W.CONFIGS[W.RMAT14]
    log(f"case: pipelined gathers, {cfg.name}")
    wl, batches = config_stream(cfg)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    _run_async_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead, batches,
                      cfg.name)


@pytest.mark.timeout(600)
def test_async_pipeline_rmat20_first_60():
    cfg = W.CONFIGS[W.RMAT20]
    log(f"case: pipelined gathers, {cfg.name}, first 60 minibatches")
    wl, batches = config_stream(cfg, 60)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    _run_async_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead, batches,
                      cfg.name)


@pytest.mark.parametrize("seed", range(6))
def test_async_pipeline_random(seed):
    n, S, V, L, T, rb, stat, batches, announce = _random_case(100 + seed)
    combined = seed % 2 == 0
    log(f"case: pipelined random seed {seed}: N={n} S={S} V={V} L={L} combined={combined}")
    store = Store.random_bytes(n, rb, seed)
    _run_async_parity(store, stat, S, V, L, batches, f"async-random{seed}", combined=combined)


def _long_case(seed):
    rng = np.random.default_rng(77 + seed)
    n = int(rng.integers(50, 400))
    S = int(rng.integers(2, 12))
    V = int(rng.choice([0, 5, 40]))
    L = int(rng.choice([4, 8, 9, 16, 31]))
    T = int(rng.choice([0, 1, 2]))
    stat = rng.integers(0, 50, n).astype(np.uint32)
    batches = [rng.integers(0, n, rng.integers(10, 60)) for _ in range(90)]
    return n, S, V, L, T, stat, batches


@pytest.mark.parametrize("pipelined", [False, True])
@pytest.mark.parametrize("seed", range(12))
def test_long_streams_window_wrap(seed, pipelined):
    """90 minibatches, so the announced-minibatch bit positions wrap around
    their 32-bit word several times, with lookaheads up to 31."""
    n, S, V, L, T, stat, batches = _long_case(seed)
    log(f"case: long stream seed {seed} pipelined={pipelined}: N={n} S={S} V={V} L={L} T={T}")
    store = Store.random_bytes(n, 32, seed)
    if pipelined:
        run_async_parity(store, stat, S, V, L, batches, rows="all", near_threshold=T, label=f"long{seed}",
                         state_every=10)
    else:
        run_parity(store, stat, S, V, L, batches, near_threshold=T, rows="all", state_every=10,
                   label=f"long{seed}")


@pytest.mark.parametrize("seed", range(8))
def test_blocking_gathers_back_to_back(seed):
    """Blocking gathers with no call in between that waits for the library's
    internal streams (counters are compared as totals at the end): each
    gather's fills, the ring writes and the next gather's staging are ordered
    by the library's events alone.  Rows, unique IDs, inverse and outcomes
    after every gather; the final cache and ring state.  Odd seeds use a
    pageable store, every fourth the victim queues."""
    n, S, V, L, T, stat, batches = _long_case(200 + seed)
    mode = "queues" if seed % 4 == 3 else "fifo"
    if mode == "queues":
        V = max(V, 1) * (L + 1)
    log(f"case: blocking back to back seed {seed} {mode}: N={n} S={S} V={V} L={L} T={T}")
    store = Store.random_bytes(n, 32, seed, pinned=seed % 2 == 0)
    run_parity(store, stat, S, V, L, batches, near_threshold=T, rows="all", label=f"blocking{seed}",
               victim_mode=mode, per_gather_stats=False)


@pytest.mark.parametrize("seed", range(8))
def test_blocking_and_pipelined_gathers_interleaved(seed):
    """The two entry points alternate by a seeded coin on one cache: a blocking
    gather's fills run on the host-link stream, a pipelined gather's on the
    dma stream, and each gather's ring write must still follow its own host
    fetch.  Odd seeds use a pageable store, every fourth the victim queues,
    every third an update period of 2."""
    n, S, V, L, T, stat, batches = _long_case(300 + seed)
    mode = "queues" if seed % 4 == 3 else "fifo"
    if mode == "queues":
        V = max(V, 1) * (L + 1)
    U = 2 if seed % 3 == 2 else 1
    log(f"case: interleaved seed {seed} {mode} U={U}: N={n} S={S} V={V} L={L} T={T}")
    store = Store.random_bytes(n, 32, seed, pinned=seed % 2 == 0)
    run_mixed_parity(store, stat, S, V, L, batches, seed, state_every=15, label=f"interleaved{seed}",
                     near_threshold=T, victim_mode=mode, refresh_period=U)


def test_blocking_and_pipelined_gathers_interleaved_rmat14():
    cfg = W.CONFIGS[W.RMAT14]
    log(f"case: {cfg.name}, blocking and pipelined gathers interleaved")
    wl, batches = config_stream(cfg)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    res = run_mixed_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead,
                           batches, 14, state_every=5, label=f"{cfg.name}-interleaved")
    assert res["total"]["victim_hits"] > 0


def test_blocking_gathers_back_to_back_rmat14():
    cfg = W.CONFIGS[W.RMAT14]
    log(f"case: {cfg.name}, blocking gathers back to back")
    wl, batches = config_stream(cfg)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    res = run_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead, batches,
                     rows="all", label=f"{cfg.name}-blocking", per_gather_stats=False)
    assert res["total"]["victim_hits"] > 0


@pytest.mark.parametrize("seed", range(12))
def test_pageable_store_random(seed):
    """The same policy with the backing store in ordinary pageable memory:
    misses and victim hits are copied by host threads into the pinned bounce
    buffer.  Odd seeds go through the pipelined entry point."""
    n, S, V, L, T, rb, stat, batches, announce = _random_case(300 + seed)
    log(f"case: pageable store, random seed {seed}: N={n} S={S} V={V} L={L} T={T}")
    store = Store.random_bytes(n, rb, seed, pinned=False)
    if seed % 2:
        run_async_parity(store, stat, S, V, L, batches, rows="all", near_threshold=T, label=f"pageable{seed}")
    else:
        mb = max(1, max(len(b) for b in list(batches) + list(announce)))
        run_parity(store, stat, S, V, L, batches, announce=announce, near_threshold=T, rows="all", max_batch=mb,
                   label=f"pageable{seed}")


def test_pageable_store_rmat14_pipelined():
    cfg = W.CONFIGS[W.RMAT14]
    log(f"case: pageable store, {cfg.name}, pipelined")
    wl, batches = config_stream(cfg)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed, pinned=False)
    res = run_async_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead,
                           batches, rows="all", state_every=5, label=f"{cfg.name} pageable")
    assert res["total"]["victim_hits"] > 0


@pytest.mark.parametrize("seed", range(4))
def test_pageable_store_long_streams(seed):
    n, S, V, L, T, stat, batches = _long_case(40 + seed)
    log(f"case: pageable store, long stream seed {seed}: N={n} S={S} V={V} L={L} T={T}")
    store = Store.random_bytes(n, 64, seed, pinned=False)
    run_async_parity(store, stat, S, V, L, batches, rows="all", near_threshold=T, label=f"pageable-long{seed}",
                     state_every=10)


def test_async_announce_errors_leave_state_unchanged():
    """A pipelined gather whose own list or announced list holds an
    out-of-range ID is rejected as a whole: neither the gather nor the
    announcement happens, and the stream then continues exactly like the
    oracle's."""
    log("case: pipelined gather + announcement error paths")
    n, S, V, L, mb = 300, 4, 8, 2, 64
    store = Store.random_bytes(n, 32, 3)
    stat = (np.arange(n, dtype=np.uint32) * 7) % 11
    cache = lsmgnn.FeatureCache(n, 32, store.buf, stat, S, V, L, mb)
    orc = Oracle(n, 32, stat, S, V, L, store=store.np)
    dev = lambda a: torch.as_tensor(np.asarray(a, np.int64)).cuda()  # noqa: E731
    rng = np.random.default_rng(9)
    batches = [rng.integers(0, n, size=int(rng.integers(1, mb + 1))) for _ in range(12)]
    db = [dev(b) for b in batches]
    out, uq, inv, oc = (torch.empty(mb * 32, dtype=torch.uint8, device="cuda"),
                        torch.empty(mb, dtype=torch.int64, device="cuda"),
                        torch.empty(mb, dtype=torch.int64, device="cuda"),
                        torch.empty(mb, dtype=torch.uint8, device="cuda"))
    for j in range(L + 1):
        cache.advance(db[j])
        orc.advance(batches[j])

    def good(b):
        tk, r = cache.gather_async(db[b], out, uq, inverse=inv, outcome=oc, announce=db[b + L + 1])
        cache.wait(tk)
        torch.cuda.current_stream().synchronize()
        o = orc.gather(batches[b])
        orc.advance(batches[b + L + 1])
        assert np.array_equal(r.unique.cpu().numpy(), o["uniq"]), b
        assert np.array_equal(r.inverse.cpu().numpy(), o["inv"]), b
        assert np.array_equal(r.outcome.cpu().numpy(), o["outcome"]), b
        assert np.array_equal(r.out.cpu().numpy(), o["out"]), b

    good(0)
    good(1)
    cache.sync()
    before = cache.export_state()
    for bad in ([0, n], [-5, 1], [n - 1, 1 << 40]):
        with pytest.raises(lsmgnn.LsmgnnError) as e:
            cache.gather_async(db[2], out, uq, inverse=inv, outcome=oc, announce=dev(bad))
        assert e.value.status == "E_RANGE"
        with pytest.raises(lsmgnn.LsmgnnError) as e:  # a bad gather list with a good announcement
            cache.gather_async(dev(bad), out, uq, inverse=inv, outcome=oc, announce=db[2 + L + 1])
        assert e.value.status == "E_RANGE"
    # the combined calls keep the window full: a separate announcement is refused
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        cache.advance(db[2 + L + 1])
    assert e.value.status == "E_WINDOW"
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        cache.gather_async(db[2], out, uq, inverse=inv, outcome=oc, announce=dev(np.zeros(mb + 1)))
    assert e.value.status == "E_INVAL"
    cache.sync()
    after = cache.export_state()
    assert after["t"] == before["t"] and np.array_equal(after["tags"], before["tags"])
    assert np.array_equal(after["ring_tags"], before["ring_tags"]) and after["ring_tail"] == before["ring_tail"]
    # the stream continues exactly like the oracle's
    last = len(batches) - L - 1
    for b in range(2, last):
        good(b)
    compare_state(cache, orc, "after pipelined errors")
    # an empty announcement is an announcement: the window is full after it
    tk, r = cache.gather_async(db[last], out, uq, inverse=inv, outcome=oc, announce=dev([]))
    cache.wait(tk)
    torch.cuda.current_stream().synchronize()
    o = orc.gather(batches[last])
    orc.advance(np.zeros(0, np.int64))
    assert np.array_equal(r.out.cpu().numpy(), o["out"])
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        cache.advance(db[0])
    assert e.value.status == "E_WINDOW"
    compare_state(cache, orc, "after empty announcement")
    cache.close()


# ---------------------------------------------- the evaluation's ablations
POLICIES = ["static", "dynamic", "round_robin"]


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("seed", range(10))
def test_policies_random_small_caches(seed, policy):
    """The alternative eviction policies (static score only, next announced use
    only, round-robin) on randomized small caches, blocking entry point."""
    n, S, V, L, T, rb, stat, batches, announce = _random_case(700 + seed)
    log(f"case: policy {policy} random seed {seed}: N={n} S={S} V={V} L={L} T={T} R={rb}")
    store = Store.random_bytes(n, rb, seed)
    run_parity(store, stat, S, V, L, batches, announce, near_threshold=T, rows="all", label=f"{policy}{seed}",
               policy=policy)


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("seed", range(3))
def test_policies_long_streams_pipelined(seed, policy):
    """90 minibatches through the pipelined entry point, so the announced-use
    bits wrap their 32-bit word (the dynamic policy's distances come from
    them) and the round-robin pointers go round many times."""
    n, S, V, L, T, stat, batches = _long_case(40 + seed)
    log(f"case: policy {policy} long stream seed {seed}: N={n} S={S} V={V} L={L} T={T}")
    store = Store.random_bytes(n, 32, seed)
    run_async_parity(store, stat, S, V, L, batches, rows="all", near_threshold=T, label=f"{policy}-long{seed}",
                     state_every=10, policy=policy)


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("name", ["one_set", "batch_exceeds_cache", "no_window", "big_batch"])
def test_policies_adversarial(name, policy):
    c = _adversarial()[name]
    log(f"case: policy {policy} adversarial {name}: N={c['n']} S={c['S']} V={c['V']} L={c['L']}")
    rb = 64 if c["n"] < (1 << 21) else 16
    store = Store.random_bytes(c["n"], rb, 1)
    stat = np.random.default_rng(3).integers(0, 5, c["n"]).astype(np.uint32)
    mb = max(1, max(len(b) for b in c["batches"]))
    run_parity(store, stat, c["S"], c["V"], c["L"], c["batches"], rows="all", max_batch=mb,
               label=f"{policy}-{name}", policy=policy)


@pytest.mark.parametrize("policy", POLICIES)
def test_policies_workload_rmat14_pipelined(policy):
    cfg = W.CONFIGS[W.RMAT14]
    log(f"case: policy {policy} {cfg.name} pipelined")
    wl, batches = config_stream(cfg)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    res = run_async_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead,
                           batches, rows="all", state_every=25, label=f"{policy}-{cfg.name}", policy=policy)
    log(f"  {policy}: {res['total']}")


# ------------------------------------------- per-iteration victim queues
QPOL = ["hybrid", "static", "dynamic", "round_robin"]


@pytest.mark.parametrize("seed", range(20))
def test_queues_random_small_caches(seed):
    """The paper's victim-queue form (a queue per reuse iteration, prefetched
    into HBM before its iteration) on randomized small caches, blocking calls;
    the policy rotates with the seed."""
    n, S, V, L, T, rb, stat, batches, announce = _random_case(900 + seed)
    V = V * (L + 1)  # C = V / (L + 1) rows per queue
    pol = QPOL[seed % 4]
    log(f"case: queues random seed {seed} policy {pol}: N={n} S={S} V={V} L={L} T={T} R={rb}")
    store = Store.random_bytes(n, rb, seed)
    run_parity(store, stat, S, V, L, batches, announce, near_threshold=T, rows="all", label=f"queues{seed}",
               policy=pol, victim_mode="queues")


@pytest.mark.parametrize("seed", range(6))
def test_queues_long_streams_pipelined(seed):
    """90 minibatches through the pipelined entry point: every queue slot is
    reused many times, and each gather's prefetch overlaps the next gather's
    metadata."""
    n, S, V, L, T, stat, batches = _long_case(60 + seed)
    V = max(V, 1) * (L + 1)
    if seed % 3 == 2:
        V = L + 1  # one row per queue: most candidates are dropped
    log(f"case: queues long stream seed {seed}: N={n} S={S} V={V} L={L} T={T}")
    store = Store.random_bytes(n, 32, seed)
    run_async_parity(store, stat, S, V, L, batches, rows="all", near_threshold=T, label=f"queues-long{seed}",
                     state_every=10, victim_mode="queues")


def test_queues_worked_example():
    """Eight lines evicted at gather 1 with next use at minibatch 4 fill queue
    4 in eviction order; with C = 5 the last three are dropped, and gather 4
    serves five victim hits from the prefetched queue."""
    log("case: queues worked example")
    n, L = 16, 4
    stat = np.zeros(n, np.uint32)
    stat[:8] = [5, 3, 4, 0, 2, 1, 7, 6]
    batches = [np.arange(8), np.arange(8, 16), np.array([], np.int64), np.array([], np.int64), np.arange(8)]
    for C in (8, 5):
        store = Store.random_bytes(n, 64, C)
        run_parity(store, stat, 1, 5 * C, L, batches, rows="all", state_every=1, label=f"queue-example-C{C}",
                   victim_mode="queues")


def test_queues_workload_rmat14_pipelined():
    cfg = W.CONFIGS[W.RMAT14]
    log(f"case: queues {cfg.name} pipelined")
    wl, batches = config_stream(cfg)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    run_async_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead, batches,
                     rows="all", state_every=5, label=f"queues-{cfg.name}", victim_mode="queues")


@pytest.mark.timeout(600)
def test_queues_workload_rmat20_first_60_pipelined():
    cfg = W.CONFIGS[W.RMAT20]
    log(f"case: queues {cfg.name} first 60 pipelined")
    wl, batches = config_stream(cfg, 60)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    res = run_async_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead,
                           batches, rows=4, store_gpu=device_store(store), state_every=20,
                           label=f"queues-{cfg.name}", victim_mode="queues")
    assert res["total"]["victim_hits"] > 0


@pytest.mark.parametrize("seed", range(4))
def test_queues_pageable_store(seed):
    n, S, V, L, T, rb, stat, batches, announce = _random_case(950 + seed)
    V = max(V, 1) * (L + 1)
    log(f"case: queues pageable seed {seed}: N={n} S={S} V={V} L={L}")
    store = Store.random_bytes(n, rb, seed, pinned=False)
    if seed % 2:
        run_async_parity(store, stat, S, V, L, batches, rows="all", near_threshold=T, label=f"queues-pg{seed}",
                         state_every=3, victim_mode="queues")
    else:
        run_parity(store, stat, S, V, L, batches, announce, near_threshold=T, rows="all", label=f"queues-pg{seed}",
                   victim_mode="queues")


@pytest.mark.parametrize("pageable", [False, True])
def test_async_rejected_calls_while_gathers_in_flight(pageable):
    """Rejected calls between pipelined gathers, with no wait in between: the
    rejected call's queued kernels (no-ops) reuse a flight whose previous
    gather's fills and ring write may still be running, and the next good call
    reuses it again.  Every gather's rows, outcomes and the final state match
    the oracle's."""
    log(f"case: pipelined gathers with rejected calls in flight, pageable={pageable}")
    rng = np.random.default_rng(4242)
    n, R, S, V, L, mb, nb = 20000, 1024, 150, 2500, 3, 6000, 36
    store = Store.random_bytes(n, R, 11, pinned=not pageable)
    stat = rng.integers(0, 50, n).astype(np.uint32)
    hot = rng.permutation(n)[:3000]
    batches = [np.concatenate([rng.choice(hot, int(rng.integers(1000, 3000))),
                               rng.integers(0, n, int(rng.integers(500, 3000)))]) for _ in range(nb)]
    cache = lsmgnn.FeatureCache(n, R, store.buf, stat, S, V, L, mb, pageable=pageable)
    orc = Oracle(n, R, stat, S, V, L, store=store.np)
    dev = lambda a: torch.as_tensor(np.asarray(a, np.int64)).cuda()  # noqa: E731
    db = [dev(b) for b in batches]
    bufs = [(torch.empty(mb * R, dtype=torch.uint8, device="cuda"), torch.empty(mb, dtype=torch.int64, device="cuda"),
             torch.empty(mb, dtype=torch.int64, device="cuda"), torch.empty(mb, dtype=torch.uint8, device="cuda"))
            for _ in range(3)]
    for j in range(L + 1):
        cache.advance(db[j])
    pending, rejected, checked = {}, 0, 0

    def check(b):
        tk, r = pending.pop(b)
        cache.wait(tk)
        torch.cuda.current_stream().synchronize()
        o = orc.gather(batches[b])
        if b + L + 1 < nb:
            orc.advance(batches[b + L + 1])
        assert np.array_equal(r.unique.cpu().numpy(), o["uniq"]), b
        assert np.array_equal(r.outcome.cpu().numpy(), o["outcome"]), b
        assert np.array_equal(r.out.cpu().numpy(), o["out"]), b

    for j in range(L + 1):
        orc.advance(batches[j])
    for b in range(nb):
        out, uq, inv, oc = bufs[b % 3]
        ann = db[b + L + 1] if b + L + 1 < nb else None
        if b % 3 == 2:  # rejected calls right before the good one, gathers b-1 and b-2 still in flight
            bad = dev([int(batches[b][0]), n + b])
            with pytest.raises(lsmgnn.LsmgnnError) as e:
                cache.gather_async(bad, out, uq, inverse=inv, outcome=oc, announce=ann)
            assert e.value.status == "E_RANGE"
            if ann is not None:
                with pytest.raises(lsmgnn.LsmgnnError) as e:
                    cache.gather_async(db[b], out, uq, inverse=inv, outcome=oc, announce=bad)
                assert e.value.status == "E_RANGE"
            rejected += 1
        pending[b] = cache.gather_async(db[b], out, uq, inverse=inv, outcome=oc, announce=ann)
        if b - 1 in pending:
            check(b - 1)
            checked += 1
    check(nb - 1)
    checked += 1
    compare_state(cache, orc, "after the stream with rejected calls")
    tot = cache.stats()[1]
    log(f"  {checked} gathers checked, {rejected} rounds of rejected calls; totals {tot}")
    assert tot["victim_hits"] > 0 and tot["evictions"] > 0
    cache.close()


@pytest.mark.parametrize("pipelined", [False, True])
def test_queues_rejected_gathers_in_between(pipelined):
    """A rejected gather between good ones changes nothing, also the queue
    that the previous good gather prefetched for the next one."""
    log(f"case: queues with rejected gathers, pipelined={pipelined}")
    rng = np.random.default_rng(77)
    n, S, V, L, mb = 400, 3, 3 * 5, 4, 64
    store = Store.random_bytes(n, 32, 5)
    stat = rng.integers(0, 9, n).astype(np.uint32)
    batches = [rng.integers(0, n, int(rng.integers(20, mb + 1))) for _ in range(30)]
    cache = lsmgnn.FeatureCache(n, 32, store.buf, stat, S, V, L, mb, victim_mode="queues")
    orc = Oracle(n, 32, stat, S, V, L, store=store.np, victim_mode="queues")
    dev = lambda a: torch.as_tensor(np.asarray(a, np.int64)).cuda()  # noqa: E731
    db = [dev(b) for b in batches]
    out, uq, inv, oc = (torch.empty(mb * 32, dtype=torch.uint8, device="cuda"),
                        torch.empty(mb, dtype=torch.int64, device="cuda"),
                        torch.empty(mb, dtype=torch.int64, device="cuda"),
                        torch.empty(mb, dtype=torch.uint8, device="cuda"))
    for j in range(L + 1):
        cache.advance(db[j])
        orc.advance(batches[j])
    vh = 0
    for b in range(len(batches) - L - 1):
        if b % 3 == 1:  # a bad list first
            with pytest.raises(lsmgnn.LsmgnnError) as e:
                if pipelined:
                    cache.gather_async(dev([0, n + b]), out, uq, inverse=inv, outcome=oc, announce=db[b + L + 1])
                else:
                    cache.gather(dev([0, n + b]), out=out, unique=uq, inverse=inv, outcome=oc)
            assert e.value.status == "E_RANGE"
        if pipelined:
            tk, r = cache.gather_async(db[b], out, uq, inverse=inv, outcome=oc, announce=db[b + L + 1])
            cache.wait(tk)
            torch.cuda.current_stream().synchronize()
        else:
            r = cache.gather(db[b], out=out, unique=uq, inverse=inv, outcome=oc)
            cache.advance(db[b + L + 1])
        o = orc.gather(batches[b])
        orc.advance(batches[b + L + 1])
        assert np.array_equal(r.outcome.cpu().numpy(), o["outcome"]), b
        assert np.array_equal(r.out.cpu().numpy(), o["out"]), b
        vh += int((o["outcome"] == 1).sum())
    compare_state(cache, orc, "queues after rejected gathers")
    assert vh > 0
    cache.close()
    orc.close()


# ------------------------------- update period of the dynamic information
@pytest.mark.parametrize("seed", range(16))
def test_update_period_random_small_caches(seed):
    """Dynamic information updated every U-th gather (U > 1): lines inserted
    since the update rank as recently inserted, passed reuses as recent.
    Policy and victim-buffer form rotate with the seed."""
    n, S, V, L, T, rb, stat, batches, announce = _random_case(1100 + seed)
    U = [2, 3, 4, 7][seed % 4]
    pol = QPOL[(seed // 4) % 4]
    mode = "queues" if seed % 2 else "fifo"
    if mode == "queues":
        V = V * (L + 1)
    log(f"case: update period {U} seed {seed} policy {pol} {mode}: N={n} S={S} V={V} L={L} T={T} R={rb}")
    store = Store.random_bytes(n, rb, seed)
    run_parity(store, stat, S, V, L, batches, announce, near_threshold=T, rows="all", label=f"upd{seed}",
               policy=pol, victim_mode=mode, refresh_period=U)


@pytest.mark.parametrize("seed", range(6))
def test_update_period_long_streams_pipelined(seed):
    n, S, V, L, T, stat, batches = _long_case(80 + seed)
    U = [2, 4, 5][seed % 3]
    mode = "queues" if seed >= 3 else "fifo"
    if mode == "queues":
        V = max(V, 1) * (L + 1)
    log(f"case: update period {U} long stream seed {seed} {mode}: N={n} S={S} V={V} L={L} T={T}")
    store = Store.random_bytes(n, 32, seed)
    run_async_parity(store, stat, S, V, L, batches, rows="all", near_threshold=T, label=f"upd-long{seed}",
                     state_every=10, victim_mode=mode, refresh_period=U)


@pytest.mark.parametrize("U", [2, 4])
def test_update_period_workload_rmat14_pipelined(U):
    cfg = W.CONFIGS[W.RMAT14]
    log(f"case: update period {U}, {cfg.name} pipelined")
    wl, batches = config_stream(cfg)
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    run_async_parity(store, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead, batches,
                     rows="all", state_every=5, label=f"upd{U}-{cfg.name}", refresh_period=U)


# ------------------------------------------------- rows in request order
@pytest.mark.parametrize("rb", [16, 48, 64, 1024])
def test_expand_gives_every_request_its_row(rb):
    """lsmgnn_expand after a gather: row i of the result is the stored row of
    request i (closed form), duplicates included."""
    log(f"case: expand R={rb}")
    rng = np.random.default_rng(rb)
    n_nodes, S, V, L = 5000, 16, 64, 2
    store = Store.random_bytes(n_nodes, rb, rb)
    stat = rng.integers(0, 9, n_nodes).astype(np.uint32)
    batches = [rng.integers(0, n_nodes, int(rng.integers(1, 3000))) for _ in range(8)]
    mb = max(b.size for b in batches)
    cache = lsmgnn.FeatureCache(n_nodes, rb, store.buf, stat, S, V, L, mb)
    for j in range(L + 1):
        cache.advance(torch.as_tensor(batches[j]).cuda())
    for b, ids in enumerate(batches):
        ids_t = torch.as_tensor(ids).cuda()
        r = cache.gather(ids_t, inverse=True)
        rows = lsmgnn.expand(r.out, r.inverse, rb)
        torch.cuda.synchronize()
        got = rows.cpu().numpy().reshape(ids.size, rb)
        assert np.array_equal(got, store.np[ids]), b
        if b + L + 1 < len(batches):
            cache.advance(torch.as_tensor(batches[b + L + 1]).cuda())
    cache.close()


def test_expand_arguments():
    log("case: expand arguments")
    L = lsmgnn.lib()
    rows = torch.zeros(64, dtype=torch.uint8, device="cuda")
    inv = torch.zeros(2, dtype=torch.int64, device="cuda")
    out = torch.zeros(64, dtype=torch.uint8, device="cuda")
    assert L.lsmgnn_expand(None, None, 0, 16, None, None) == lsmgnn.OK  # nothing to do
    assert L.lsmgnn_expand(rows.data_ptr(), inv.data_ptr(), 2, 24, out.data_ptr(), None) == lsmgnn.E_INVAL
    assert L.lsmgnn_expand(rows.data_ptr() + 8, inv.data_ptr(), 2, 16, out.data_ptr(), None) == lsmgnn.E_INVAL
    assert L.lsmgnn_expand(rows.data_ptr(), None, 2, 16, out.data_ptr(), None) == lsmgnn.E_INVAL
