"""Pins for the CPU oracle (no GPU).

The oracle is the definition the GPU library is held to, so it is pinned here to
things other than itself: published SplitMix64 outputs, hand-derived scenarios
(tests/golden/scenarios.yaml), closed-form special cases, library routines
(numpy unique), invariants that follow from the rules, an optimal-policy upper
bound (Belady MIN with bypass), and a naive brute-force model on tiny inputs.
"""
import itertools
import os

import numpy as np
import pytest
import yaml

from oracle.oracle import HIT, MISS, VICTIM_HIT, Oracle, OracleError, set_of
from paper_2407_15264_amd import workload as W
from tests.naive_model import NaiveCache

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
GAMMA = 0x9E3779B97F4A7C15
EMPTY = 0xFFFFFFFF
CODE = {HIT: "H", VICTIM_HIT: "V", MISS: "M"}


def _published_splitmix():
    vals = []
    with open(os.path.join(GOLDEN, "splitmix64_seed1234567.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                vals.append(int(line))
    return vals


def test_set_index_matches_published_splitmix64_outputs():
    # set(x) is fastrange(hi32(first SplitMix64 output of state x)).  The k-th
    # output of the stream seeded with s is the first output of state s + k*gamma.
    vals = _published_splitmix()
    assert len(vals) == 5
    for k, v in enumerate(vals):
        x = (1234567 + k * GAMMA) % (1 << 64)
        for S in (1, 2, 13107, 262144, 6291456, (1 << 32) - 1):
            assert set_of(x, S) == ((v >> 32) * S) >> 32
    assert W.splitmix_at(1234567, 0) == vals[0]  # the generators use the same stream


def test_set_index_is_uniform_enough():
    S = 2048
    counts = np.bincount([set_of(x, S) for x in range(1 << 15)], minlength=S)
    assert counts.min() >= 3 and counts.max() <= 40  # mean 16


# --------------------------------------------------------------- scenarios
def _load_scenarios():
    with open(os.path.join(GOLDEN, "scenarios.yaml")) as f:
        return yaml.safe_load(f)


def _static_array(spec, n):
    a = np.full(n, spec.get("default", 0), np.uint32)
    for k, v in spec.items():
        if k != "default":
            a[int(k)] = v
    return a


@pytest.mark.parametrize("name", sorted(_load_scenarios().keys()))
def test_golden_scenario(name):
    sc = _load_scenarios()[name]
    n = sc["num_nodes"]
    o = Oracle(n, 16, _static_array(sc["static"], n), sc["num_sets"], sc["victim_rows"],
               sc["lookahead"], ways=sc["ways"])
    for op in sc["ops"]:
        if op[0] == "advance":
            o.advance(np.array(op[1], np.int64))
            continue
        r = o.gather(np.array(op[1], np.int64), rows=False)
        exp = op[2]
        if "outcome" in exp:
            assert "".join(CODE[c] for c in r["outcome"]) == exp["outcome"]
        for key in ("hits", "victim_hits", "misses", "evictions", "enqueued", "dropped"):
            if key in exp:
                assert r["stats"][key] == exp[key], key
        st = o.export_state()
        if "tags" in exp:
            tags = [[-1 if t == EMPTY else int(t) for t in row] for row in st["tags"]]
            assert tags == exp["tags"]
        if "ring" in exp:
            assert [-1 if t == EMPTY else int(t) for t in st["ring_tags"]] == exp["ring"]
        if "tail" in exp:
            assert st["ring_tail"] == exp["tail"]


# ----------------------------------------------------------- special cases
def test_single_set_small_universe_misses_are_first_touches():
    rng = np.random.default_rng(1)
    n = 8
    o = Oracle(n, 16, rng.integers(0, 5, n), 1, 4, 2)
    seen = set()
    for b in range(12):
        ids = rng.integers(0, n, rng.integers(0, 10))
        r = o.gather(ids, rows=False)
        first = set(np.unique(ids).tolist()) - seen
        assert r["stats"]["misses"] == len(first)
        assert r["stats"]["hits"] == np.unique(ids).size - len(first)
        assert r["stats"]["evictions"] == 0 and r["stats"]["victim_hits"] == 0
        seen |= first


@pytest.mark.parametrize("k", [1, 3, 8])
def test_no_window_reduces_to_static_order(k):
    # L = 0: no line has reuse information, so within a batch the policy evicts
    # the lowest-static line that was not inserted in this batch (Sec. 4.2).
    rng = np.random.default_rng(k)
    stat = rng.permutation(np.arange(100, 116)).astype(np.uint32)
    stat[16 - 8:] = 1  # new IDs 8..15
    o = Oracle(16, 16, stat, 1, 0, 0)
    o.gather(np.arange(8))
    o.gather(np.arange(8, 8 + k))
    tags = set(o.export_state()["tags"][0].tolist())
    survivors = sorted(range(8), key=lambda x: stat[x])[k:]
    assert tags == set(survivors) | set(range(8, 8 + k))


# --------------------------------------------------------------- invariants
def _check_invariants(o, ids, r, store=None):
    st = r["stats"]
    uniq, inv = np.unique(ids, return_inverse=True)
    assert np.array_equal(r["uniq"], uniq)
    assert np.array_equal(r["inv"], inv.reshape(-1))
    assert st["hits"] + st["victim_hits"] + st["misses"] == st["unique"] == uniq.size
    assert st["evictions"] == st["enqueued"] + st["dropped"]
    assert np.count_nonzero(r["outcome"] == HIT) == st["hits"]
    assert np.count_nonzero(r["outcome"] == VICTIM_HIT) == st["victim_hits"]
    per_request = r["outcome"][inv.reshape(-1)]  # each request takes its unique ID's outcome
    assert st["request_hits"] == np.count_nonzero(per_request == HIT)
    assert st["request_victim_hits"] == np.count_nonzero(per_request == VICTIM_HIT)
    s = o.export_state()
    tags = s["tags"]
    live = tags[tags != EMPTY]
    assert np.unique(live).size == live.size, "duplicate resident tag"
    for si in range(tags.shape[0]):
        for t in tags[si]:
            if t != EMPTY:
                assert set_of(int(t), o.num_sets) == si
    ring = s["ring_tags"][s["ring_tags"] != EMPTY]
    assert np.unique(ring).size == ring.size
    assert not (set(ring.tolist()) & set(live.tolist())), "a line is in the cache and the ring"
    _, tot = o.stats()
    assert s["ring_tail"] == tot["enqueued"]
    assert live.size == tot["victim_hits"] + tot["misses"] - tot["evictions"]
    if store is not None:
        assert np.array_equal(r["out"], store.view(np.uint8).reshape(store.shape[0], -1)[uniq])


def _drive(o, batches, L, announce=None, check=None):
    announce = batches if announce is None else announce
    for j in range(min(L + 1, len(announce))):
        o.advance(announce[j])
    res = []
    for b, ids in enumerate(batches):
        r = o.gather(ids, rows=check is not None and check.get("rows", False))
        if check is not None:
            _check_invariants(o, ids, r, check.get("store"))
        res.append(r)
        if b + L + 1 < len(announce):
            o.advance(announce[b + L + 1])
    return res


def test_invariants_on_small_rmat_stream():
    cfg = W.CONFIGS[W.RMAT14]
    wl = W.Workload(cfg)
    store = W.features(cfg.num_nodes, cfg.dim)
    o = Oracle(cfg.num_nodes, cfg.row_bytes, wl.static, cfg.cache.num_sets, cfg.cache.victim_rows,
               cfg.cache.lookahead, store=store)
    res = _drive(o, [wl.batch(b) for b in range(wl.num_batches)], cfg.cache.lookahead,
                 check=dict(rows=True, store=store))
    _, tot = o.stats()
    assert tot["victim_hits"] > 0 and tot["enqueued"] > 0 and tot["hits"] > 0
    assert len(res) == cfg.batches


def test_features_are_standard_normal():
    x = W.features(4096, 128).astype(np.float64)
    assert abs(x.mean()) < 0.01 and abs(x.std() - 1) < 0.01
    assert np.array_equal(x, W.features(4096, 128).astype(np.float64))


# ------------------------------------------------------------- Belady bound
def _belady_hits(seq, ways):
    """Optimal hits for one fully associative set of `ways` lines with bypass
    allowed (Belady's MIN): on a miss with a full set, drop whichever of the
    residents and the newcomer is next used farthest in the future."""
    hits, cache = 0, set()
    for i, x in enumerate(seq):
        if x in cache:
            hits += 1
            continue
        if len(cache) < ways:
            cache.add(x)
            continue

        def nxt(y):
            for j in range(i + 1, len(seq)):
                if seq[j] == y:
                    return j
            return len(seq) + 1
        far = max(list(cache) + [x], key=nxt)
        if far != x:
            cache.remove(far)
            cache.add(x)
    return hits


@pytest.mark.parametrize("seed", range(6))
def test_hits_never_exceed_belady(seed):
    rng = np.random.default_rng(seed)
    n, S, ways_ = 40, 3, 8
    batches = [rng.integers(0, n, rng.integers(5, 30)) for _ in range(15)]
    o = Oracle(n, 16, rng.integers(0, 4, n), S, int(rng.integers(0, 6)), 3)
    res = _drive(o, batches, 3)
    per_set = {s: [] for s in range(S)}
    for ids in batches:
        for x in np.unique(ids):
            per_set[set_of(int(x), S)].append(int(x))
    bound = sum(_belady_hits(seq, ways_) for seq in per_set.values())
    assert sum(r["stats"]["hits"] for r in res) <= bound


# ---------------------------------------------------- eviction policies
# The evaluation's ablation (Sec. 5, impact of the cache eviction policy) swaps
# only the choice of victim in a full set; these pins hold each alternative to
# a closed form or to an exhaustive optimum.
POLICY_NAMES = ["hybrid", "static", "dynamic", "round_robin"]


@pytest.mark.parametrize("ways", [1, 2, 4, 8])
@pytest.mark.parametrize("V", [0, 3])
@pytest.mark.parametrize("one_batch", [False, True])
def test_round_robin_closed_form(ways, V, one_batch):
    # Round-robin ignores scores and reuse: the k-th distinct ID into a set
    # goes to way k mod W, so way w ends up holding the largest such k.  With
    # no window nothing has reuse information and every eviction is dropped.
    n = 11
    rng = np.random.default_rng(ways * 10 + V)
    o = Oracle(n, 16, rng.integers(0, 9, n), 1, V, 0, ways=ways, policy="round_robin")
    if one_batch:
        res = [o.gather(rng.permutation(n), rows=False)]  # uniques are served in ascending order
    else:
        res = [o.gather(np.array([k]), rows=False) for k in range(n)]
    st = o.export_state()
    assert [int(t) for t in st["tags"][0]] == [max(k for k in range(n) if k % ways == w) for w in range(ways)]
    assert sum(r["stats"]["evictions"] for r in res) == n - ways
    assert sum(r["stats"]["dropped"] for r in res) == n - ways


def test_round_robin_pointer_example():
    # four ways, IDs 0..9 one per gather: ways hold 8, 9, 6, 7 and the next
    # eviction (ID 10) replaces way 2
    o = Oracle(16, 16, np.ones(16, np.uint32), 1, 0, 0, ways=4, policy="round_robin")
    for k in range(10):
        o.gather(np.array([k]), rows=False)
    assert o.export_state()["tags"][0].tolist() == [8, 9, 6, 7]
    o.gather(np.array([10]), rows=False)
    assert o.export_state()["tags"][0].tolist() == [8, 9, 10, 7]


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("ways", [1, 2, 3, 5])
def test_static_only_keeps_newest_and_best_scores(seed, ways):
    # Static-only evicts the lowest score in the full set whatever the window
    # says, so after distinct IDs x_1..x_m arrive one per gather the set holds
    # x_m and the W - 1 highest-scored of x_1..x_{m-1}.
    rng = np.random.default_rng(seed)
    n, m, L = 30, 17, 4
    stat = rng.permutation(n).astype(np.uint32)
    seq = rng.permutation(n)[:m]
    announce = [rng.integers(0, n, 5) for _ in range(m + L)]
    o = Oracle(n, 16, stat, 1, 2, L, ways=ways, policy="static")
    _drive(o, [np.array([x]) for x in seq], L, announce)
    keep = {int(seq[-1])} | set(sorted(seq[:-1].tolist(), key=lambda x: -int(stat[x]))[:ways - 1])
    assert set(o.export_state()["tags"][0].tolist()) == keep


def _min_demand_misses(seq, ways):
    """Fewest misses any policy that must insert every missed ID can reach on
    one fully associative set, by exhaustive search over the evictions."""
    import functools

    @functools.lru_cache(maxsize=None)
    def best(i, cache):
        if i == len(seq):
            return 0
        x = seq[i]
        if x in cache:
            return best(i + 1, cache)
        if len(cache) < ways:
            return 1 + best(i + 1, cache | {x})
        return 1 + min(best(i + 1, (cache - {y}) | {x}) for y in cache)

    return best(0, frozenset())


@pytest.mark.parametrize("seed", range(40))
def test_dynamic_only_with_full_window_is_optimal(seed):
    # With one ID per gather and a window covering the whole stream, evicting
    # the line whose next use is furthest (unused lines first) is Belady's
    # rule, optimal among policies that insert every miss.
    rng = np.random.default_rng(500 + seed)
    n, ways = int(rng.integers(3, 7)), int(rng.integers(1, 4))
    seq = rng.integers(0, n, int(rng.integers(4, 13))).tolist()
    L = len(seq)
    o = Oracle(n, 16, rng.integers(0, 4, n), 1, 0, L, ways=ways, policy="dynamic")
    res = _drive(o, [np.array([x]) for x in seq], L)
    assert sum(r["stats"]["misses"] for r in res) == _min_demand_misses(tuple(seq), ways)


@pytest.mark.parametrize("policy", POLICY_NAMES)
@pytest.mark.parametrize("seed", range(3))
def test_policies_never_exceed_belady(policy, seed):
    rng = np.random.default_rng(seed)
    n, S, ways_ = 40, 3, 8
    batches = [rng.integers(0, n, rng.integers(5, 30)) for _ in range(15)]
    o = Oracle(n, 16, rng.integers(0, 4, n), S, 0, 3, policy=policy)
    res = _drive(o, batches, 3)
    per_set = {s: [] for s in range(S)}
    for ids in batches:
        for x in np.unique(ids):
            per_set[set_of(int(x), S)].append(int(x))
    assert sum(r["stats"]["hits"] for r in res) <= sum(_belady_hits(q, ways_) for q in per_set.values())


def test_policy_rejected_when_unknown():
    with pytest.raises(OracleError) as e:
        Oracle(10, 16, np.ones(10, np.uint32), 2, 2, 1, policy=4)
    assert e.value.status == "E_INVAL"


# ------------------------------------------------------- naive brute force
def _naive_run(n, S, ways, V, L, T, stat, batches, announce, policy="hybrid", victim_mode="fifo", U=1):
    m = NaiveCache(n, S, ways, V, L, stat, lambda x: set_of(x, S), T, policy=policy, victim_mode=victim_mode,
                   refresh_period=U)
    out = []
    for j in range(min(L + 1, len(announce))):
        assert m.advance(announce[j]) == "OK"
    for b, ids in enumerate(batches):
        _, r = m.gather(ids)
        out.append(r)
        if b + L + 1 < len(announce):
            assert m.advance(announce[b + L + 1]) == "OK"
    return m, out


def _compare(n, S, ways, V, L, T, stat, batches, announce, policy="hybrid", victim_mode="fifo", U=1):
    m, exp = _naive_run(n, S, ways, V, L, T, stat, batches, announce, policy, victim_mode, U)
    o = Oracle(n, 16, stat, S, V, L, near_threshold=T, ways=ways, policy=policy, victim_mode=victim_mode,
               refresh_period=U)
    got = _drive(o, batches, L, announce)
    for e, g in zip(exp, got):
        assert "".join(CODE[c] for c in g["outcome"]) == e["outcome"]
        for k in ("hits", "victim_hits", "misses", "evictions", "enqueued", "dropped"):
            assert g["stats"][k] == e[k], k
    st = o.export_state()
    assert [[-1 if t == EMPTY else int(t) for t in row] for row in st["tags"]] == m.tags()
    assert [-1 if t == EMPTY else int(t) for t in st["ring_tags"]] == m.ring_tags()
    assert st["ring_tail"] == m.tail


@pytest.mark.parametrize("policy", POLICY_NAMES)
def test_exhaustive_tiny_universe_against_naive_model(policy):
    n = 3
    subsets = [np.array(c, np.int64) for r in range(n + 1) for c in itertools.combinations(range(n), r)]
    stat = np.array([2, 1, 2], np.uint32)
    count = 0
    for V in (0, 1):
        for L in (1, 2):
            for seq in itertools.product(range(len(subsets)), repeat=4):
                batches = [subsets[i] for i in seq]
                _compare(n, 1, 2, V, L, 0, stat, batches, batches, policy)
                count += 1
    assert count == 4 * len(subsets) ** 4


@pytest.mark.parametrize("policy", POLICY_NAMES)
@pytest.mark.parametrize("seed", range(150))
def test_random_small_against_naive_model(seed, policy):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(2, 14))
    S = int(rng.integers(1, 4))
    ways = int(rng.integers(1, 4))
    V = int(rng.choice([0, 1, 2, 3, 5]))
    L = int(rng.choice([0, 1, 2, 3, 5, 9]))
    T = int(rng.choice([0, 0, 1, 2]))
    stat = rng.integers(0, 4, n).astype(np.uint32)
    nb = int(rng.integers(1, 8))
    batches = [rng.integers(0, n, rng.integers(0, 8)) for _ in range(nb)]
    # announced lists differ from the served ones half of the time
    if rng.random() < 0.5:
        announce = [rng.integers(0, n, rng.integers(0, 8)) for _ in range(nb + L)]
    else:
        announce = batches
    _compare(n, S, ways, V, L, T, stat, batches, announce, policy)


# ------------------------------------------------------------------- errors
def test_errors_leave_state_unchanged():
    o = Oracle(10, 16, np.ones(10, np.uint32), 2, 2, 1)
    o.advance(np.array([1, 2]))
    o.advance(np.array([3]))
    with pytest.raises(OracleError) as e:
        o.advance(np.array([4]))
    assert e.value.status == "E_WINDOW"
    o.gather(np.array([1, 2, 5]))
    before = o.export_state()
    with pytest.raises(OracleError) as e:
        o.gather(np.array([1, 10]))
    assert e.value.status == "E_RANGE"
    with pytest.raises(OracleError) as e:
        o.gather(np.array([-1]))
    assert e.value.status == "E_RANGE"
    with pytest.raises(OracleError) as e:
        o.advance(np.array([11]))
    assert e.value.status == "E_RANGE"
    after = o.export_state()
    assert after["t"] == before["t"]
    assert np.array_equal(after["tags"], before["tags"])
    r = o.gather(np.array([], np.int64))
    assert r["stats"]["unique"] == 0 and r["stats"]["requests"] == 0
    assert o.export_state()["t"] == before["t"] + 1


@pytest.mark.parametrize("kw", [dict(num_nodes=0), dict(row_bytes=8), dict(num_sets=0),
                                dict(lookahead=32), dict(num_nodes=1 << 33)])
def test_bad_config_rejected(kw):
    args = dict(num_nodes=10, row_bytes=16, num_sets=2, victim_rows=2, lookahead=1)
    args.update(kw)
    with pytest.raises(OracleError) as e:
        Oracle(args["num_nodes"], args["row_bytes"], np.ones(max(1, min(args["num_nodes"], 64)), np.uint32),
               args["num_sets"], args["victim_rows"], args["lookahead"])
    assert e.value.status == "E_INVAL"


# ------------------------------------------------ per-iteration victim queues
# Sec. 4.3.1's form of the victim buffer: one queue per reuse iteration, a
# counter giving each evicted line its position, drop when full.
def _queue_scenario(C):
    """Worked case in the spirit of the paper's example (a line whose next reuse
    iteration is 4 goes to the queue of iteration 4 at the position its
    counter names).  One 8-way set, L = 4 (so T = 1), V = 5 * C.  Gather 0
    fills nodes 0..7; gather 1 brings 8..15 and evicts all of 0..7, whose next
    announced use is minibatch 4 (distance 3: the far level), in ascending
    static score (all lines are far, so the score decides)."""
    n, L = 16, 4
    stat = np.zeros(n, np.uint32)
    stat[:8] = [5, 3, 4, 0, 2, 1, 7, 6]
    batches = [np.arange(8), np.arange(8, 16), np.array([], np.int64), np.array([], np.int64), np.arange(8)]
    o = Oracle(n, 16, stat, 1, 5 * C, L, victim_mode="queues")
    return o, stat, batches, L


def test_queue_positions_follow_the_counter():
    o, stat, batches, L = _queue_scenario(C=8)
    res = _drive(o, batches[:2], L, batches)
    assert res[1]["stats"]["evictions"] == 8 and res[1]["stats"]["enqueued"] == 8
    order = sorted(range(8), key=lambda x: stat[x])  # eviction order: 3, 5, 4, 1, 2, 0, 7, 6
    ring = o.export_state()["ring_tags"].reshape(5, 8)
    assert ring[4].tolist() == order  # queue of iteration 4, slot 4 mod 5; the 6th eviction (counter 5) at position 5
    assert ring[4][5] == 0
    assert (np.delete(ring, 4, axis=0) == EMPTY).all()


def test_queue_full_drops_and_queue_serves_only_its_iteration():
    o, stat, batches, L = _queue_scenario(C=5)
    res = _drive(o, batches, L)
    assert res[1]["stats"]["enqueued"] == 5 and res[1]["stats"]["dropped"] == 3  # counters 5, 6, 7 find it full
    kept = sorted(range(8), key=lambda x: stat[x])[:5]
    st4 = res[4]
    assert st4["stats"]["victim_hits"] == 5 and st4["stats"]["misses"] == 3
    assert sorted(int(x) for x in st4["uniq"][st4["outcome"] == VICTIM_HIT]) == sorted(kept)
    assert (o.export_state()["ring_tags"] == EMPTY).all()  # the served queue is emptied


def test_queue_entry_is_not_served_before_its_iteration():
    # node 3 sits in the queue of iteration 4; requested (unannounced) at
    # gather 2 it is a miss.  At gather 4 its queue entry is still there, so
    # it is served from the cache or, if an earlier fill of that gather evicted
    # it again, from the queue: never from storage.
    o, stat, batches, L = _queue_scenario(C=8)
    served = list(batches)
    served[2] = np.array([3])
    res = _drive(o, served, L, batches)
    assert res[2]["stats"]["misses"] == 1 and res[2]["stats"]["victim_hits"] == 0
    r4 = res[4]
    assert r4["outcome"][list(r4["uniq"]).index(3)] != MISS
    assert r4["stats"]["misses"] == 0


@pytest.mark.parametrize("policy", POLICY_NAMES)
def test_queues_exhaustive_tiny_universe_against_naive_model(policy):
    n = 3
    subsets = [np.array(c, np.int64) for r in range(n + 1) for c in itertools.combinations(range(n), r)]
    stat = np.array([2, 1, 2], np.uint32)
    for L in (1, 2):
        for V in (0, L + 1, 2 * (L + 1)):
            for seq in itertools.product(range(len(subsets)), repeat=4):
                batches = [subsets[i] for i in seq]
                _compare(n, 1, 2, V, L, 0, stat, batches, batches, policy, "queues")


@pytest.mark.parametrize("policy", POLICY_NAMES)
@pytest.mark.parametrize("seed", range(100))
def test_queues_random_small_against_naive_model(seed, policy):
    rng = np.random.default_rng(5000 + seed)
    n = int(rng.integers(2, 14))
    S = int(rng.integers(1, 4))
    ways = int(rng.integers(1, 4))
    L = int(rng.choice([0, 1, 2, 3, 5, 9]))
    V = int(rng.choice([0, 1, 2, 3])) * (L + 1)
    T = int(rng.choice([0, 0, 1, 2]))
    stat = rng.integers(0, 4, n).astype(np.uint32)
    nb = int(rng.integers(1, 10))
    batches = [rng.integers(0, n, rng.integers(0, 8)) for _ in range(nb)]
    if rng.random() < 0.5:
        announce = [rng.integers(0, n, rng.integers(0, 8)) for _ in range(nb + L)]
    else:
        announce = batches
    _compare(n, S, ways, V, L, T, stat, batches, announce, policy, "queues")


def test_queue_mode_needs_a_row_per_queue():
    with pytest.raises(OracleError) as e:
        Oracle(10, 16, np.ones(10, np.uint32), 2, 3, 3, victim_mode="queues")  # V = 3 < L + 1 = 4
    assert e.value.status == "E_INVAL"


# ------------------------------------------ update period of the dynamic information
# Sec. 4.2 updates the lines' next reuse iterations every few iterations; lines
# inserted since the last update lack dynamic information (recently inserted).
def test_lines_inserted_since_the_update_are_recent():
    # A = 0 (static 5), B = 1 (static 1), C = 2; L = 2 (T = 1).  At gather 1, B's
    # next use is gather 2 (near) and A has none.  Updating every gather, A (no
    # reuse) is evicted for C; updating every third gather, both still count as
    # recently inserted at gather 1 and the lower static score, B, goes.
    stat = np.array([5, 1, 9], np.uint32)
    batches = [np.array([0, 1]), np.array([2]), np.array([1])]
    for U, gone in ((1, 0), (3, 1)):
        o = Oracle(3, 16, stat, 1, 0, 2, ways=2, refresh_period=U)
        _drive(o, batches[:2], 2, batches)
        assert gone not in o.export_state()["tags"][0].tolist(), U


def test_a_passed_reuse_counts_as_recent():
    # C = 0 (static 9), X = 2 (static 1), Y = 3 (static 5); L = 2.  Updated at
    # gather 2, X's next use is gather 3.  At gather 3 (no update with U = 2)
    # that recorded use has come, so X ranks as recent and Y (no reuse) makes
    # room for C: X is then a hit.  Updated at gather 3 (U = 1), X has no further
    # use, loses on its static score, and is a miss.
    stat = np.array([9, 0, 1, 5], np.uint32)
    batches = [np.array([2, 3]), np.array([], np.int64), np.array([], np.int64), np.array([0, 2])]
    for U, outcome_x in ((2, HIT), (1, MISS)):
        o = Oracle(4, 16, stat, 1, 0, 2, ways=2, refresh_period=U)
        r = _drive(o, batches, 2)[3]
        assert r["outcome"][list(r["uniq"]).index(2)] == outcome_x, U


@pytest.mark.parametrize("seed", range(20))
def test_no_update_reduces_hybrid_to_static_order(seed):
    # With no update after the first (empty) one, no line ever has dynamic
    # information: the hybrid order is the static order over all lines.
    rng = np.random.default_rng(seed)
    n, S, L = 40, 2, 3
    stat = rng.integers(0, 6, n).astype(np.uint32)
    batches = [rng.integers(0, n, int(rng.integers(1, 12))) for _ in range(12)]
    a = Oracle(n, 16, stat, S, 0, L, ways=3, refresh_period=1000)
    b = Oracle(n, 16, stat, S, 0, L, ways=3, policy="static")
    ra, rb = _drive(a, batches, L), _drive(b, batches, L)
    for x, y in zip(ra, rb):
        assert np.array_equal(x["outcome"], y["outcome"])
    assert np.array_equal(a.export_state()["tags"], b.export_state()["tags"])


@pytest.mark.parametrize("mode", ["fifo", "queues"])
@pytest.mark.parametrize("policy", POLICY_NAMES)
@pytest.mark.parametrize("seed", range(40))
def test_update_period_random_small_against_naive_model(seed, policy, mode):
    rng = np.random.default_rng(7000 + seed)
    n = int(rng.integers(2, 14))
    S = int(rng.integers(1, 4))
    ways = int(rng.integers(1, 4))
    L = int(rng.choice([0, 1, 2, 3, 5, 9]))
    V = int(rng.choice([0, 1, 2, 3])) * (L + 1)
    T = int(rng.choice([0, 0, 1, 2]))
    U = int(rng.choice([2, 3, 4, 7]))
    stat = rng.integers(0, 4, n).astype(np.uint32)
    nb = int(rng.integers(1, 12))
    batches = [rng.integers(0, n, rng.integers(0, 8)) for _ in range(nb)]
    if rng.random() < 0.5:
        announce = [rng.integers(0, n, rng.integers(0, 8)) for _ in range(nb + L)]
    else:
        announce = batches
    _compare(n, S, ways, V, L, T, stat, batches, announce, policy, mode, U)


def test_request_counts_repeat_with_the_request():
    # a node requested k times counts k times per request and once per unique ID
    o = Oracle(10, 16, np.ones(10, np.uint32), 1, 0, 0)
    o.gather(np.array([3, 4]))
    r = o.gather(np.array([3, 3, 3, 4, 5, 5]))
    st = r["stats"]
    assert (st["hits"], st["misses"]) == (2, 1)
    assert (st["request_hits"], st["request_victim_hits"]) == (4, 0)
    assert st["requests"] - st["request_hits"] - st["request_victim_hits"] == 2
