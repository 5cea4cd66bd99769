"""GPU <-> oracle parity of the static score (lsmgnn_pagerank_scores), needs an
MI355X.

Ranks: the GPU accumulates each node's pushed sum with atomics in varying
order, so it matches the oracle's sequential sums to rounding.  A sum of m
terms carries at most (m - 1) eps of its magnitude in rounding error, the
update adds a few more, and the iteration is a d-contraction in the 1-norm,
so over any number of iterations each side stays within (D + 4) eps / (1 - d)
of the exact iterate in the 1-norm (D = the largest in-degree, eps = 2^-53):
the two sides differ by at most twice that.  Scores: the GPU's must equal the
quantization of its own ranks evaluated on the host in the same (float64)
precision; against the oracle's scores they may differ only where the ranks
do, which the test bounds and reports.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from oracle.oracle import Oracle, pagerank, rank_scores  # noqa: E402
from paper_2407_15264_amd import lsmgnn  # noqa: E402
from paper_2407_15264_amd import workload as W  # noqa: E402
from tests.parity_driver import Store, log, run_parity  # noqa: E402

EPS = 2.0 ** -53


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lsmgnn.lib()


def _gpu_pagerank(offsets, adj, d, K):
    off_t = torch.as_tensor(np.asarray(offsets, np.int64)).cuda()
    adj_t = torch.as_tensor(np.asarray(adj, np.uint32).view(np.int32)).cuda()
    s, r = lsmgnn.pagerank_scores(off_t, adj_t, d, K, rank=True)
    torch.cuda.synchronize()
    return s.cpu().numpy().view(np.uint32), r.cpu().numpy()


def _check(offsets, adj, d, K, label):
    offsets = np.asarray(offsets, np.int64)
    adj = np.asarray(adj, np.uint32)
    n = offsets.size - 1
    s_g, r_g = _gpu_pagerank(offsets, adj, d, K)
    r_o = pagerank(offsets, adj, d, K)
    s_o = rank_scores(r_o)
    D = int(np.bincount(adj, minlength=n).max()) if adj.size else 0
    bound = 2 * (D + 4) * EPS / (1 - d)
    l1 = float(np.abs(r_g - r_o).sum())
    rel = float(np.max(np.abs(r_g - r_o) / r_o))
    # the GPU's scores are the quantization of its own ranks, in float64
    q = np.floor(r_g / r_g.max() * 4294967295.0).astype(np.uint32)
    mism = int(np.count_nonzero(s_g != s_o))
    log(f"  {label}: N={n} E={adj.size} K={K} d={d}: |dr|_1 {l1:.3g} (bound {bound:.3g}), max rel {rel:.3g}, "
        f"scores differing from the oracle's: {mism}")
    assert l1 <= bound, (l1, bound)
    assert np.array_equal(s_g, q)
    if mism:
        assert np.abs(s_g.astype(np.int64) - s_o.astype(np.int64)).max() <= 1
    return s_g


@pytest.mark.parametrize("seed", range(10))
def test_random_small_graphs(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 300))
    deg = rng.integers(0, 12, n) * (rng.random(n) < 0.8)  # about one node in five has no entries
    offsets = np.concatenate([[0], np.cumsum(deg)]).astype(np.int64)
    adj = rng.integers(0, n, int(offsets[-1])).astype(np.uint32)
    d = float(rng.choice([0.5, 0.85, 0.95]))
    K = int(rng.choice([0, 1, 2, 20]))
    log(f"case: pagerank random seed {seed}")
    _check(offsets, adj, d, K, f"random{seed}")


def test_no_entries_at_all():
    s, r = _gpu_pagerank(np.zeros(6, np.int64), np.zeros(0, np.uint32), 0.85, 5)
    assert np.allclose(r, 0.2, rtol=1e-15, atol=0) and (s == 4294967295).all()


@pytest.mark.parametrize("name", ["rmat-s14-e18-f32x128", "rmat-s20-deg16-f32x256"])
def test_workload_graphs(name):
    cfg = W.CONFIGS[name]
    log(f"case: pagerank {cfg.name}")
    g = W.rmat_graph(cfg.num_nodes, cfg.num_edges, cfg.rmat, cfg.seed)
    _check(g.offsets, g.adj, 0.85, 20, cfg.name)


def test_errors_leave_scores_unwritten():
    log("case: pagerank errors")
    off = torch.tensor([0, 2, 3], dtype=torch.int64, device="cuda")
    bad_adj = torch.tensor([1, 2, 0], dtype=torch.int32, device="cuda")  # entry 2 >= N = 2
    scores = torch.full((2,), 7, dtype=torch.int32, device="cuda")
    rc = lsmgnn.lib().lsmgnn_pagerank_scores(off.data_ptr(), bad_adj.data_ptr(), 2, 0.85, 3, scores.data_ptr(), None,
                                             0, None)
    assert rc == lsmgnn.E_RANGE and scores.cpu().tolist() == [7, 7]
    dec = torch.tensor([0, 3, 2], dtype=torch.int64, device="cuda")
    rc = lsmgnn.lib().lsmgnn_pagerank_scores(dec.data_ptr(), bad_adj.data_ptr(), 2, 0.85, 3, scores.data_ptr(), None,
                                             0, None)
    assert rc == lsmgnn.E_RANGE
    for d in (1.0, -0.1, float("nan")):
        rc = lsmgnn.lib().lsmgnn_pagerank_scores(off.data_ptr(), bad_adj.data_ptr(), 2, d, 3, scores.data_ptr(),
                                                 None, 0, None)
        assert rc == lsmgnn.E_INVAL


def test_cache_parity_with_pagerank_scores():
    # the GPU's scores drive both the library's cache and the oracle's
    cfg = W.CONFIGS[W.RMAT14]
    log(f"case: cache parity with reverse-PageRank static scores, {cfg.name}")
    wl = W.Workload(cfg)
    off_t = torch.as_tensor(wl.graph.offsets).cuda()
    adj_t = torch.as_tensor(wl.graph.adj.view(np.int32)).cuda()
    static = lsmgnn.pagerank_scores(off_t, adj_t).cpu().numpy().view(np.uint32)
    batches = [wl.batch(b) for b in range(wl.num_batches)]
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed)
    for policy in ("hybrid", "static"):
        run_parity(store, static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead, batches,
                   rows="all", state_every=5, label=f"pagerank-{policy}", policy=policy)
