"""The allocation-free split (lsmgnn_split_by_type_noalloc_async) against the
split that takes caller work memory (lsmgnn_split_by_type_async), through the
C ABI, on two calls in a row (the second with a smaller input, so that the
shared device array still holds the first call's contents), on the GPU.
Bit-exact: the per-type lists, their lengths and the status word; plus a
short output, a bad ID, and sizes beyond the array rejected on the host."""
import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

from paper_2407_15264_amd import lsmgnn  # noqa: E402


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    lsmgnn.lib()


def _typed_graph(N, T, seed):
    rng = np.random.default_rng(seed)
    node_type = rng.integers(0, T, N).astype(np.uint8)
    local = np.empty(N, np.uint32)
    for t in range(T):
        idx = np.flatnonzero(node_type == t)
        local[idx] = rng.permutation(idx.size)
    return node_type, local


def _both(ids, d_type, d_local, T, cap):
    """Run both entry points on `ids`; returns (lists, result words) of each."""
    res = []
    for noalloc in (False, True):
        outs = [torch.full((cap,), -1, dtype=torch.int64, device="cuda") for _ in range(T)]
        r = lsmgnn.PinnedBuffer(8 * (T + 1))
        rn = r.numpy(np.uint64, (T + 1,))
        if noalloc:
            lsmgnn.split_by_type_noalloc_async(ids, d_type, d_local, outs, r.ptr)
        else:
            work = torch.empty(lsmgnn.split_work_bytes(max(ids.numel(), 1), T), dtype=torch.uint8, device="cuda")
            lsmgnn.split_by_type_async(ids, d_type, d_local, outs, work, r.ptr)
        torch.cuda.current_stream().synchronize()
        res.append(([o.cpu().numpy() for o in outs], rn.copy()))
        r.close()
    return res


@pytest.mark.parametrize("T", [1, 4, 16])
def test_noalloc_split_matches_the_split_with_work_memory(T):
    N = 200_000
    node_type, local = _typed_graph(N, T, 5 + T)
    d_type = torch.as_tensor(node_type).cuda()
    d_local = torch.as_tensor(local.view(np.int32)).cuda()
    rng = np.random.default_rng(T)
    cap = 600_000
    for n in (500_000, 70_001):  # two calls in a row, the second smaller
        ids = torch.as_tensor(rng.integers(0, N, n)).cuda()
        (lw, rw), (ln, rn) = _both(ids, d_type, d_local, T, cap)
        assert int(rw[T]) == lsmgnn.OK and np.array_equal(rw, rn), (n, rw, rn)
        h = ids.cpu().numpy()
        for t in range(T):
            want = local[h[node_type[h] == t]].astype(np.int64)
            assert int(rn[t]) == want.size
            assert np.array_equal(ln[t], lw[t]), (n, t)
            assert np.array_equal(ln[t][: want.size], want), (n, t)


def test_noalloc_split_status_words_and_limits():
    T, N = 3, 5000
    node_type, local = _typed_graph(N, T, 1)
    d_type = torch.as_tensor(node_type).cuda()
    d_local = torch.as_tensor(local.view(np.int32)).cuda()
    # a short output: E_INVAL with the full lengths, the prefixes written
    ids = torch.as_tensor(np.random.default_rng(2).integers(0, N, 3000)).cuda()
    (lw, rw), (ln, rn) = _both(ids, d_type, d_local, T, 40)
    assert int(rn[T]) == lsmgnn.E_INVAL and np.array_equal(rw, rn)
    for t in range(T):
        assert np.array_equal(ln[t], lw[t])
    # an ID outside [0, N): E_RANGE in the status word, as the other entry point
    bad = torch.as_tensor([1, 2, N], dtype=torch.int64).cuda()
    (_, rw), (_, rn) = _both(bad, d_type, d_local, T, 16)
    assert int(rn[T]) == lsmgnn.E_RANGE and int(rw[T]) == lsmgnn.E_RANGE
    # sizes beyond the library's array are refused on the host, before any launch
    L = lsmgnn.lib()
    outs = (ctypes.c_void_p * 16)(*([ids.data_ptr()] * 16))
    r = lsmgnn.PinnedBuffer(8 * 17)
    too_many = (1 << 24) + 1  # with 16 types: one tile beyond the array
    assert lsmgnn.split_work_bytes(too_many, 16) > 256 + (1 << 24) // 256 * 16 * 4
    rc = L.lsmgnn_split_by_type_noalloc_async(ctypes.c_void_p(ids.data_ptr()), too_many, N,
                                              ctypes.c_void_p(d_type.data_ptr()), ctypes.c_void_p(d_local.data_ptr()),
                                              16, outs, 0, ctypes.c_void_p(r.ptr), None)
    assert rc == lsmgnn.E_INVAL
    r.close()
