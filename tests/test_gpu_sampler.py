"""GPU neighbour sampler (lsmgnn_sampler_create / lsmgnn_sample) against the
seeded host sampler of the workload generator, needs an MI355X.

Both implement one definition (uniform sampling without replacement per hop,
Floyd's draws from counter-based SplitMix64 streams), so every request list
must be identical, element by element, including the seeds' order, the
frontier order and the order of each node's samples.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from paper_2407_15264_amd import lsmgnn  # noqa: E402
from paper_2407_15264_amd import workload as W  # noqa: E402
from tests.parity_driver import log  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lsmgnn.lib()


def _dev_graph(g):
    off = torch.as_tensor(np.asarray(g.offsets, np.int64)).cuda()
    adj = torch.as_tensor(np.asarray(g.adj, np.uint32).view(np.int32)).cuda()
    return off, adj


def _host_lists(g, seeds, batch_size, fanout, nb, seed):
    ids, offs = W.sample_batches(g, np.asarray(seeds, np.int64), batch_size, fanout, 0, nb, seed)
    return [ids[offs[b]:offs[b + 1]] for b in range(nb)]


def _check_stream(g, seeds, batch_size, fanout, nb, seed, label, cap=None):
    ref = _host_lists(g, seeds, batch_size, fanout, nb, seed)
    off, adj = _dev_graph(g)
    smp = lsmgnn.GpuSampler(off, adj, fanout, seed=seed)
    dseeds = torch.as_tensor(np.asarray(seeds, np.int64)).cuda()
    cap = cap or max(1, max(r.size for r in ref))
    out = torch.empty(cap, dtype=torch.int64, device="cuda")
    for b in range(nb):
        got = smp.sample(dseeds[b * batch_size:(b + 1) * batch_size], b, out).cpu().numpy()
        assert got.size == ref[b].size, (label, b, got.size, ref[b].size)
        assert np.array_equal(got, ref[b]), (label, b, int(np.argmax(got != ref[b])))
    log(f"  {label}: {nb} lists identical, {sum(r.size for r in ref)} requests")
    smp.close()
    return ref


@pytest.mark.parametrize("fanout", [(10, 5), (15, 10, 5), (64,), (3, 3, 3, 3), (1, 64, 1), (0, 5), (4, 0, 3)])
def test_rmat_lists_match_host_sampler(fanout):
    log(f"case: R-MAT 2^12 nodes, 2^15 edges, fanout {fanout}")
    g = W.rmat_graph(1 << 12, 1 << 15, seed=5)
    seeds = W.seed_permutation(1 << 12, 12 * 100, seed=5)
    _check_stream(g, seeds, 100, fanout, 12, seed=5, label=f"fanout {fanout}")


def test_duplicate_seeds_zero_degree_nodes_and_small_degrees():
    """Repeated seeds stay in the list as given (the frontier holds each once);
    nodes without neighbours draw nothing; nodes with fewer neighbours than
    the fanout list all of them."""
    log("case: duplicate seeds, zero-degree and low-degree nodes")
    rng = np.random.default_rng(3)
    n = 500
    deg = rng.choice([0, 0, 1, 2, 5, 30, 80], n)
    off = np.zeros(n + 1, np.int64)
    np.cumsum(deg, out=off[1:])
    adj = rng.integers(0, n, int(off[-1])).astype(np.uint32)
    g = W.Graph(off, adj, np.zeros(n, np.uint32))
    seeds = rng.integers(0, n, 40 * 30)
    seeds[::7] = seeds[0]
    _check_stream(g, seeds, 40, (6, 64, 2), 30, seed=11, label="mixed degrees")


def test_workload_stream_matches_generated_requests():
    """The first minibatches of the bench workload: the GPU sampler gives the
    request lists the bench's host-generated streams hold."""
    cfg = W.CONFIGS[W.RMAT20]
    log(f"case: {cfg.name}, first 6 minibatches")
    wl = W.Workload(cfg, 6)
    off, adj = _dev_graph(wl.graph)
    smp = lsmgnn.GpuSampler(off, adj, cfg.fanout, seed=cfg.seed)
    seeds = torch.as_tensor(wl.seeds).cuda()
    out = torch.empty(wl.max_batch, dtype=torch.int64, device="cuda")
    for b in range(6):
        got = smp.sample(seeds[b * cfg.batch_size:(b + 1) * cfg.batch_size], b, out).cpu().numpy()
        assert np.array_equal(got, wl.batch(b)), b
    log(f"  identical to the generated stream ({wl.ids.size} requests)")
    smp.close()


def test_capacity_empty_and_bad_seeds():
    g = W.rmat_graph(1 << 10, 1 << 13, seed=2)
    n = 1 << 10
    ref = _host_lists(g, np.arange(64), 64, (10, 5), 1, 9)[0]
    off, adj = _dev_graph(g)
    smp = lsmgnn.GpuSampler(off, adj, (10, 5), seed=9)
    seeds = torch.arange(64, dtype=torch.int64, device="cuda")
    # a list longer than the output: E_INVAL, the length needed, the prefix written
    small = torch.full((100,), -7, dtype=torch.int64, device="cuda")
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        smp.sample(seeds, 0, small)
    assert e.value.status == "E_INVAL"
    assert np.array_equal(small.cpu().numpy(), ref[:100])
    # no seeds: an empty list
    out = torch.empty(ref.size, dtype=torch.int64, device="cuda")
    assert smp.sample(torch.empty(0, dtype=torch.int64, device="cuda"), 0, out).numel() == 0
    # a seed outside [0, N) rejects the call; the next call is unaffected
    for bad in ([3, n], [-1, 5]):
        with pytest.raises(lsmgnn.LsmgnnError) as e:
            smp.sample(torch.as_tensor(bad, dtype=torch.int64).cuda(), 0, out)
        assert e.value.status == "E_RANGE"
        assert np.array_equal(smp.sample(seeds, 0, out).cpu().numpy(), ref)
    smp.close()


def test_bad_graphs_and_arguments_rejected():
    n = 64
    off = np.arange(n + 1, dtype=np.int64)
    adj = np.arange(n, dtype=np.uint32)
    good_off, good_adj = torch.as_tensor(off).cuda(), torch.as_tensor(adj.view(np.int32)).cuda()
    for fanout in ((), (65,), (1,) * 9):
        with pytest.raises(lsmgnn.LsmgnnError) as e:
            lsmgnn.GpuSampler(good_off, good_adj, fanout)
        assert e.value.status == "E_INVAL"
    bad_adj = adj.copy()
    bad_adj[10] = n  # an entry outside [0, N)
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        lsmgnn.GpuSampler(good_off, torch.as_tensor(bad_adj.view(np.int32)).cuda(), (4,))
    assert e.value.status == "E_RANGE"
    bad_off = off.copy()
    bad_off[5], bad_off[6] = 7, 6  # decreasing, same total
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        lsmgnn.GpuSampler(torch.as_tensor(bad_off).cuda(), good_adj, (4,))
    assert e.value.status == "E_RANGE"
    shifted = off + 1  # does not start at 0; adj still holds offsets[N] entries
    adj2 = np.zeros(n + 1, np.uint32)
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        lsmgnn.GpuSampler(torch.as_tensor(shifted).cuda(), torch.as_tensor(adj2.view(np.int32)).cuda(), (4,))
    assert e.value.status == "E_RANGE"


def test_async_calls_queue_several_minibatches():
    """lsmgnn_sample_async: several minibatches queued back to back on one
    stream, each into its own output, give the blocking call's lists; the
    status word reports a bad seed and a short output."""
    g = W.rmat_graph(1 << 11, 1 << 14, seed=8)
    fanout = (12, 6)
    nb, B = 6, 50
    seeds = W.seed_permutation(1 << 11, nb * B, seed=8)
    ref = _host_lists(g, seeds, B, fanout, nb, 8)
    off, adj = _dev_graph(g)
    smp = lsmgnn.GpuSampler(off, adj, fanout, seed=8)
    dseeds = torch.as_tensor(seeds).cuda()
    res = lsmgnn.PinnedBuffer(16 * (nb + 2))
    r = res.numpy(np.uint64, (nb + 2, 2))
    outs = [torch.full((max(x.size for x in ref),), -1, dtype=torch.int64, device="cuda") for _ in range(nb)]
    for b in range(nb):
        smp.sample_async(dseeds[b * B:(b + 1) * B], b, outs[b], res.ptr + 16 * b)
    short = torch.empty(10, dtype=torch.int64, device="cuda")
    smp.sample_async(dseeds[:B], 0, short, res.ptr + 16 * nb)
    bad_seeds = torch.as_tensor([1, 1 << 11], dtype=torch.int64).cuda()  # kept alive until the stream has run
    bad_out = torch.empty(5, dtype=torch.int64, device="cuda")
    smp.sample_async(bad_seeds, 0, bad_out, res.ptr + 16 * (nb + 1))
    torch.cuda.current_stream().synchronize()
    for b in range(nb):
        assert int(r[b, 1]) == 0 and int(r[b, 0]) == ref[b].size, b
        assert np.array_equal(outs[b][: ref[b].size].cpu().numpy(), ref[b]), b
    assert int(r[nb, 0]) == ref[0].size and int(r[nb, 1]) == 1  # LSMGNN_E_INVAL: longer than the output
    assert np.array_equal(short.cpu().numpy(), ref[0][:10])
    assert int(r[nb + 1, 1]) == 2  # LSMGNN_E_RANGE: a seed outside [0, N)
    smp.close()
    res.close()


def test_split_by_type_matches_a_stable_partition():
    """lsmgnn_split_by_type_async against numpy: per type, the requests of
    that type in request order, as within-type indices; status words for a
    bad ID, a bad type and a short output; an empty list."""
    rng = np.random.default_rng(21)
    N, T = 5000, 5
    node_type = rng.integers(0, T, N).astype(np.uint8)
    local = np.empty(N, np.uint32)
    for t in range(T):
        idx = np.flatnonzero(node_type == t)
        local[idx] = rng.permutation(idx.size)  # any index within the type
    d_type = torch.as_tensor(node_type).cuda()
    d_local = torch.as_tensor(local.view(np.int32)).cuda()
    cap = 30000
    outs = [torch.full((cap,), -1, dtype=torch.int64, device="cuda") for _ in range(T)]
    work = torch.empty(lsmgnn.split_work_bytes(cap, T), dtype=torch.uint8, device="cuda")
    res = lsmgnn.PinnedBuffer(8 * (T + 1))
    r = res.numpy(np.uint64, (T + 1,))
    for n in (0, 1, 255, 256, 257, 12345, 30000):
        ids = rng.integers(0, N, n)
        ids[::3] = ids[0] if n else 0
        d_ids = torch.as_tensor(ids.astype(np.int64)).cuda()
        lsmgnn.split_by_type_async(d_ids, d_type, d_local, outs, work, res.ptr)
        torch.cuda.current_stream().synchronize()
        assert int(r[T]) == 0, n
        for t in range(T):
            want = local[ids[node_type[ids] == t]].astype(np.int64)
            assert int(r[t]) == want.size and np.array_equal(outs[t][: want.size].cpu().numpy(), want), (n, t)
    # a short output: E_INVAL, the full lengths, the prefixes written
    ids = rng.integers(0, N, 4000)
    short = [torch.full((50,), -1, dtype=torch.int64, device="cuda") for _ in range(T)]
    d_ids = torch.as_tensor(ids.astype(np.int64)).cuda()
    lsmgnn.split_by_type_async(d_ids, d_type, d_local, short, work, res.ptr)
    torch.cuda.current_stream().synchronize()
    assert int(r[T]) == 1
    for t in range(T):
        want = local[ids[node_type[ids] == t]].astype(np.int64)
        assert int(r[t]) == want.size and np.array_equal(short[t].cpu().numpy(), want[:50]), t
    # an ID outside [0, N), or a node whose type is >= T: E_RANGE
    bad_ids = torch.as_tensor([1, 2, N], dtype=torch.int64).cuda()
    lsmgnn.split_by_type_async(bad_ids, d_type, d_local, outs, work, res.ptr)
    torch.cuda.current_stream().synchronize()
    assert int(r[T]) == 2
    bad_type = d_type.clone()
    bad_type[7] = T
    seven = torch.as_tensor([3, 7], dtype=torch.int64).cuda()
    lsmgnn.split_by_type_async(seven, bad_type, d_local, outs, work, res.ptr)
    torch.cuda.current_stream().synchronize()
    assert int(r[T]) == 2
    # work memory too small: rejected before anything is queued
    with pytest.raises(lsmgnn.LsmgnnError) as e:
        lsmgnn.split_by_type_async(d_ids, d_type, d_local, outs, work[:64], res.ptr)
    assert e.value.status == "E_INVAL"
    res.close()


def test_binding_checks_dtypes_and_takes_the_smallest_capacity():
    """The Python binding passes only contiguous device tensors of the right
    element type, and gives the split the smallest output length as its
    capacity (a longer list is then reported, not written past a short one)."""
    g = W.rmat_graph(2000, 20000, seed=4)
    off, adj = _dev_graph(g)
    with pytest.raises(TypeError):
        lsmgnn.GpuSampler(off.to(torch.int32), adj, (5, 3))
    smp = lsmgnn.GpuSampler(off, adj, (5, 3), seed=1)
    out = torch.empty(4096, dtype=torch.int64, device="cuda")
    with pytest.raises(TypeError):
        smp.sample(torch.arange(10, dtype=torch.int32, device="cuda"), 0, out)
    with pytest.raises(TypeError):
        smp.sample(torch.arange(10, dtype=torch.int64, device="cuda"), 0, out.to(torch.int32))
    with pytest.raises(TypeError):
        smp.sample(torch.arange(20, dtype=torch.int64, device="cuda")[::2], 0, out)
    smp.close()
    N, T = 300, 3
    node_type = torch.as_tensor(np.arange(N) % T, dtype=torch.uint8).cuda()
    local = torch.as_tensor(np.arange(N) // T, dtype=torch.int32).cuda()
    ids = torch.arange(N, dtype=torch.int64, device="cuda")
    work = torch.empty(lsmgnn.split_work_bytes(N, T), dtype=torch.uint8, device="cuda")
    res = lsmgnn.PinnedBuffer(8 * (T + 1))
    r = res.numpy(np.uint64, (T + 1,))
    with pytest.raises(TypeError):
        lsmgnn.split_by_type_async(ids.to(torch.int32), node_type, local, [out[:N]] * T, work, res.ptr)
    with pytest.raises(TypeError):
        lsmgnn.split_by_type_async(ids, node_type.to(torch.int32), local, [out[:N]] * T, work, res.ptr)
    with pytest.raises(TypeError):
        lsmgnn.split_by_type_async(ids, node_type, local.to(torch.int64), [out[:N]] * T, work, res.ptr)
    # unequal outputs: each type has 100 requests, the second output holds 40
    outs = [torch.full((128,), -1, dtype=torch.int64, device="cuda"),
            torch.full((40,), -1, dtype=torch.int64, device="cuda"),
            torch.full((128,), -1, dtype=torch.int64, device="cuda")]
    guard = torch.full((64,), -7, dtype=torch.int64, device="cuda")  # allocated after the short output
    lsmgnn.split_by_type_async(ids, node_type, local, outs, work, res.ptr)
    torch.cuda.current_stream().synchronize()
    assert int(r[T]) == lsmgnn.E_INVAL and [int(v) for v in r[:T]] == [100, 100, 100]
    for t in range(T):
        assert np.array_equal(outs[t][:40].cpu().numpy(), np.arange(40)), t
    assert (outs[0][40:].cpu().numpy() == -1).all() and (guard.cpu().numpy() == -7).all()
    res.close()
