"""Pins for the oracle's static score (no GPU): the reverse-PageRank power
iteration and its 32-bit quantization (oracle/pagerank.c).

Pinned against a hand-derived iteration (tests/golden/pagerank_small.yaml),
closed forms (directed cycle, complete graph, two-way star), the fixed point
of the same Markov chain solved as a dense linear system (numpy), the
contraction bound of the power iteration, mass conservation, and the
quantization formula on hand-picked vectors.
"""
import os

import numpy as np
import pytest
import yaml

from oracle.oracle import OracleError, pagerank, rank_scores

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _csr(n, edges):
    edges = sorted(edges, key=lambda e: e[0])  # CSR order: by source, stable
    offsets = np.zeros(n + 1, np.int64)
    for u, _ in edges:
        offsets[u + 1] += 1
    return np.cumsum(offsets), np.array([v for _, v in edges], np.uint32)


def test_hand_derived_iteration():
    g = yaml.safe_load(open(os.path.join(GOLDEN, "pagerank_small.yaml")))
    r = pagerank(g["offsets"], g["adj"], g["damping"], g["iterations"])
    exp = np.array([0.05 + 0.85 * k / 18 for k in g["rank_k_over_18"]])
    assert np.allclose(r, exp, rtol=1e-14, atol=0)
    s = rank_scores(r)
    assert s[2] == 2**32 - 1
    assert s[0] == int(np.floor(exp[0] / exp[2] * 4294967295.0))


@pytest.mark.parametrize("n", [1, 2, 7, 100])
def test_directed_cycle_is_uniform(n):
    off, adj = _csr(n, [(u, (u + 1) % n) for u in range(n)])
    r = pagerank(off, adj, 0.85, 30)
    assert np.allclose(r, 1.0 / n, rtol=1e-13, atol=0)


def test_complete_graph_is_uniform():
    n = 9
    off, adj = _csr(n, [(u, v) for u in range(n) for v in range(n) if u != v])
    assert np.allclose(pagerank(off, adj, 0.85, 25), 1.0 / n, rtol=1e-13, atol=0)


@pytest.mark.parametrize("m", [1, 3, 10])
def test_two_way_star_closed_form(m):
    # centre 0 <-> leaves 1..m.  Fixed point: r0 = (1-d)/N + d*m*rl and
    # rl = (1-d)/N + d*r0/m, so r0 = (1 + d*m) / (N*(1 + d)).
    n, d = m + 1, 0.85
    off, adj = _csr(n, [(0, v) for v in range(1, n)] + [(v, 0) for v in range(1, n)])
    r = pagerank(off, adj, d, 300)
    r0 = (1 + d * m) / (n * (1 + d))
    assert abs(r[0] - r0) < 1e-13
    assert np.allclose(r[1:], (1 - r0) / m, rtol=1e-12, atol=0)


def _fixed_point(n, off, adj, d):
    M = np.zeros((n, n))
    for u in range(n):
        deg = off[u + 1] - off[u]
        if deg == 0:
            M[:, u] = 1.0 / n
        for e in range(off[u], off[u + 1]):
            M[adj[e], u] += 1.0 / deg
    return np.linalg.solve(np.eye(n) - d * M, np.full(n, (1 - d) / n))


@pytest.mark.parametrize("seed", range(12))
def test_power_iteration_contracts_to_the_linear_fixed_point(seed):
    # Random graphs with multi-edges, self loops and nodes without entries.
    rng = np.random.default_rng(seed)
    n = int(rng.integers(2, 40))
    d = float(rng.choice([0.5, 0.85, 0.9]))
    edges = [(int(rng.integers(0, n)), int(rng.integers(0, n))) for _ in range(int(rng.integers(0, 4 * n)))]
    off, adj = _csr(n, edges)
    star = _fixed_point(n, off, adj, d)
    for K in (0, 1, 5, 40, 200):
        r = pagerank(off, adj, d, K)
        assert abs(r.sum() - 1.0) < 1e-12  # the chain conserves mass
        # the iteration is a d-contraction in the 1-norm, from a start at most 2 away
        assert np.abs(r - star).sum() <= 2 * d**K + 1e-12


def test_zero_iterations_and_no_damping_are_uniform():
    off, adj = _csr(5, [(0, 1), (0, 1), (2, 3)])
    assert np.array_equal(pagerank(off, adj, 0.85, 0), np.full(5, 0.2))
    assert np.allclose(pagerank(off, adj, 0.0, 7), 0.2, rtol=1e-15, atol=0)


def test_more_entries_more_rank():
    # a node sampled by more nodes ranks higher; repeated entries count
    off, adj = _csr(4, [(0, 3), (1, 3), (2, 3), (3, 0), (3, 1), (3, 1)])
    r = pagerank(off, adj, 0.85, 60)
    assert r[3] > r[1] > r[0] > r[2]


def test_quantization():
    s = rank_scores(np.array([1.0, 0.5, 0.25, 0.0, 1.0]))
    assert s.tolist() == [4294967295, 2147483647, 1073741823, 0, 4294967295]
    s = rank_scores(np.array([3e-9, 1e-9]))
    assert s[0] == 4294967295 and s[1] == int(np.floor(1e-9 / 3e-9 * 4294967295.0))


def test_errors():
    with pytest.raises(OracleError) as e:
        pagerank([0, 1], [1], 0.85, 3)  # entry names node 1 of a 1-node graph
    assert e.value.status == "E_RANGE"
    with pytest.raises(OracleError) as e:
        pagerank([0, 2, 1], [0, 1], 0.85, 3)  # offsets decrease
    assert e.value.status == "E_INVAL"
    with pytest.raises(OracleError) as e:
        pagerank([0, 0], [], 1.0, 3)
    assert e.value.status == "E_INVAL"
    with pytest.raises(OracleError) as e:
        rank_scores(np.zeros(3))
    assert e.value.status == "E_INVAL"
