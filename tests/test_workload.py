"""The seeded input generators (no GPU), checked against their definitions:
R-MAT quadrant probabilities and CSR form, seed permutations (and the prefix
property the benchmark relies on), the GraphSAGE request-list structure
(seeds, then per hop distinct CSR entries of each frontier node in ascending
position order, the next frontier being the sorted unique samples), the
features against a float64 Box-Muller evaluation of the same draws and fp16
features as the round-to-nearest-even of the fp32 ones (numpy's conversion,
also over wide sweeps of float bit patterns), node typing, and the
pinned-memory plan.
"""
import numpy as np
import pytest

from paper_2407_15264_amd import workload as W


def test_rmat_csr_form_and_in_degree():
    g = W.rmat_graph(3000, 40000, seed=5)  # not a power of two: endpoints >= N are rejected
    assert g.offsets[0] == 0 and g.offsets[-1] == 40000
    assert np.all(np.diff(g.offsets) >= 0)
    assert g.adj.max() < 3000
    assert np.array_equal(g.indeg, np.bincount(g.adj, minlength=3000).astype(np.uint32))


def test_rmat_quadrant_probabilities():
    # At the top recursion level an edge lands in quadrant (src half, dst half)
    # with probability a, b, c, d = 0.57, 0.19, 0.19, 0.05.
    n, e = 1 << 14, 1 << 18
    g = W.rmat_graph(n, e, (0.57, 0.19, 0.19), seed=0)
    src = np.repeat(np.arange(n), np.diff(g.offsets))
    hi_s, hi_d = src >= n // 2, g.adj >= n // 2
    frac = [np.mean(~hi_s & ~hi_d), np.mean(~hi_s & hi_d), np.mean(hi_s & ~hi_d), np.mean(hi_s & hi_d)]
    for got, want in zip(frac, (0.57, 0.19, 0.19, 0.05)):
        assert abs(got - want) < 0.005, frac


def test_seed_permutation_prefixes():
    full = W.seed_permutation(1000, 1000, seed=3)
    assert np.array_equal(np.sort(full), np.arange(1000))
    assert np.array_equal(W.seed_permutation(1000, 137, seed=3), full[:137])
    assert not np.array_equal(W.seed_permutation(1000, 1000, seed=4), full)


def _check_request_structure(g, seeds, fanout, ids):
    B = seeds.size
    assert np.array_equal(ids[:B], seeds)
    frontier = np.unique(seeds)
    p = B
    for f in fanout:
        hop = []
        for v in frontier:
            row = g.adj[g.offsets[v]: g.offsets[v + 1]]
            k = min(f, row.size)
            got = ids[p: p + k]
            p += k
            if k == row.size:
                assert np.array_equal(got, row)
            else:
                # k distinct positions of the row, ascending: a subsequence
                j = 0
                for x in got:
                    while j < row.size and row[j] != x:
                        j += 1
                    assert j < row.size, (v, got, row)
                    j += 1
            hop.append(got)
        frontier = np.unique(np.concatenate(hop)) if hop else np.zeros(0, np.int64)
    assert p == ids.size


def test_sampler_request_structure():
    g = W.rmat_graph(2000, 16000, seed=1)
    seeds = W.seed_permutation(2000, 6 * 32, seed=1)
    ids, offs = W.sample_batches(g, seeds, 32, (5, 3, 2), 0, 6, seed=1)
    for b in range(6):
        _check_request_structure(g, seeds[b * 32:(b + 1) * 32], (5, 3, 2), ids[offs[b]: offs[b + 1]])
    # a later window of minibatches gives the same lists (counter-based draws)
    ids2, offs2 = W.sample_batches(g, seeds, 32, (5, 3, 2), 3, 6, seed=1)
    assert np.array_equal(ids2, ids[offs[3]: offs[6]])


def test_fp16_features_round_the_fp32_ones_to_nearest_even():
    f32 = W.features(300, 64, 4, seed=9)
    f16 = W.features(300, 64, 2, seed=9)
    assert np.array_equal(f16.view(np.uint16), f32.astype(np.float16).view(np.uint16))
    part = np.empty((100, 64), np.float32)
    W.fill_features(part.ctypes.data, 64, 4, 100, 200, seed=9)  # any row range gives the same rows
    assert np.array_equal(part, f32[100:200])


def _np_mix(z):
    z = (z ^ (z >> np.uint64(30))) * np.uint64(0xbf58476d1ce4e5b9)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94d049bb133111eb)
    return z ^ (z >> np.uint64(31))


def _np_at(key, k):
    with np.errstate(over="ignore"):
        return _np_mix(np.uint64(key) + (np.asarray(k, np.uint64) + np.uint64(1)) * np.uint64(0x9e3779b97f4a7c15))


def test_features_are_box_muller_pairs_of_the_documented_draws():
    """Pair j of row v is (rho cos theta, rho sin theta) from draw v*dim/2 + j:
    u1 = (top 24 bits + 1) / 2^24, theta = 2 pi (next 24 bits) / 2^24.  The
    generator's binary32 polynomials must agree with float64 numpy to a few
    float roundings."""
    dim, n, seed = 96, 2000, 5
    with np.errstate(over="ignore"):
        key = int(_np_at(int(_np_mix(np.uint64(seed) ^ np.uint64(0x5851f42d4c957f2d))), 4))  # LABEL_FEAT = 4
    r = _np_at(key, np.arange(n * dim // 2, dtype=np.uint64))
    u1 = ((r >> np.uint64(40)).astype(np.float64) + 1) / 2 ** 24
    th = 2 * np.pi * ((r >> np.uint64(16)) & np.uint64(0xffffff)).astype(np.float64) / 2 ** 24
    rho = np.sqrt(-2 * np.log(u1))
    want = np.stack([rho * np.cos(th), rho * np.sin(th)], axis=1).reshape(n, dim)
    got = W.features(n, dim, 4, seed=seed).astype(np.float64)
    err = np.abs(got - want)
    assert err.max() < 4e-6 * max(1.0, np.abs(want).max()), err.max()
    # the bulk is within two float ulps of the value
    assert np.mean(err <= 2 * np.spacing(np.abs(want).astype(np.float32)).astype(np.float64) + 1e-12) > 0.99


def test_fp16_rounding_matches_numpy_over_float_bit_sweeps():
    import ctypes
    lib = W.lib()
    lib.wl_f32_to_f16.restype = None
    lib.wl_f32_to_f16.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint64]
    # every 61st pattern of the finite fp16 range (|x| <= 65504 = 0x477fe000 in
    # binary32), every 7th across the subnormal boundary, all around the
    # rounding ties of the smallest normals, with both signs
    bits = np.concatenate([np.arange(0, 0x477fe001, 61, dtype=np.uint64),
                           np.arange(0x33000000, 0x38800000 + 4096, 7, dtype=np.uint64),
                           np.arange(0x387fe000, 0x38802000, dtype=np.uint64)]).astype(np.uint32)
    bits = np.concatenate([bits, bits | np.uint32(0x80000000)])
    f = bits.view(np.float32)
    out = np.empty(f.size, np.uint16)
    lib.wl_f32_to_f16(f.ctypes.data, out.ctypes.data, f.size)
    want = f.astype(np.float16).view(np.uint16)
    bad = np.flatnonzero(out != want)
    assert bad.size == 0, (hex(int(bits[bad[0]])), hex(int(out[bad[0]])), hex(int(want[bad[0]])))


def test_typed_workload_split():
    cfg = W.HeteroConfig("typed-test", 20000, 200000, (0.4, 0.3, 0.2, 0.1), (64, 32, 16, 16), 4, 4, 64, (5, 3),
                         1 << 20, 1 << 19, 2)
    wl = W.HeteroWorkload(cfg)
    counts = cfg.type_counts()
    assert sum(counts) == 20000 and counts[0] == 8000 and counts[3] == 2000
    for t in range(4):
        local = wl.node_local[wl.node_type == t]
        assert np.array_equal(np.sort(local), np.arange(counts[t]))
        assert np.array_equal(wl.static[t][local], wl.graph.indeg[wl.node_type == t])
    for b in range(4):
        g = wl.ids[wl.offsets[b]: wl.offsets[b + 1]]
        for t in range(4):
            exp = wl.node_local[g[wl.node_type[g] == t]]
            assert np.array_equal(wl.type_batches(t)[b], exp)
            assert np.array_equal(wl.batch(b, t), exp)


@pytest.mark.parametrize("stores, ring, budget, want", [
    ([10, 30, 20], 5, 65, [True, True, True]),
    ([10, 30, 20], 5, 60, [False, True, True]),   # the largest first, then whatever still fits
    ([10, 30, 20], 5, 50, [True, True, False]),
    ([10, 30, 20], 25, 50, [False, False, True]),
    ([40], 30, 50, [False]),
])
def test_pin_plan(stores, ring, budget, want):
    assert W.pin_plan(stores, ring, budget) == want
