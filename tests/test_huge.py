"""Full-size parity of the 100M-node workload (needs an MI355X host with about
250 GiB of memory; run with `-m huge`, it is not part of `-m gpu`).

The store (10^8 fp16 x 1024 rows, 191 GiB) exceeds the pinned memory a process
may hold, so it lives in pageable memory and the library's host threads copy
miss rows; the 96 GiB cache and the 32 GiB ring are the configured ones.  The
first 300 minibatches of the stream (the cache fills after about 75) run in
the bench's launch configuration: every gather's unique IDs, inverse and
outcomes are compared with the oracle, a seeded sample of its rows with the
backing store, all rows with the oracle's every 8th gather, and the cache and
ring state every 16 gathers and at the end.
"""
import time

import pytest

pytestmark = pytest.mark.huge

torch = pytest.importorskip("torch")

from paper_2407_15264_amd import workload as W  # noqa: E402
from tests.parity_driver import Store, log, run_async_parity  # noqa: E402

PREFIX = 300  # minibatches checked: the cache fills after about 75 of them


@pytest.mark.timeout(3000)
def test_rmat100m_full_size_pipelined_prefix():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = W.CONFIGS[W.RMAT100M]
    log(f"case: {cfg.name}, first {PREFIX} minibatches, pipelined, full size, pageable store")
    t0 = time.time()
    wl = W.Workload(cfg, PREFIX)
    static = wl.static
    batches = [wl.batch(b) for b in range(PREFIX)]
    wl.graph = None  # only the in-degree is kept
    log(f"  workload generated in {time.time() - t0:.1f} s (max batch {max(b.size for b in batches)})")
    store = Store(cfg.num_nodes, cfg.dim, cfg.elt_bytes, cfg.seed, pinned=False)
    log(f"  store filled ({time.time() - t0:.1f} s)")
    res = run_async_parity(store, static, cfg.cache.num_sets, cfg.cache.victim_rows, cfg.cache.lookahead, batches,
                           rows=8, row_sample=4096, state_every=16, label=cfg.name)
    log(f"  {cfg.name}: {res['total']} in {res['seconds']:.1f} s")
    assert res["total"]["hits"] > 0 and res["total"]["misses"] > 0
