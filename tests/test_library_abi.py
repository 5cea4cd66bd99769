"""CPU-side checks of the HIP library (no GPU needed): it loads, exports every
entry point its header declares, rejects bad configurations before touching a
device, and its host set-index helper agrees with the oracle's."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle.oracle import set_of as oracle_set_of
from paper_2407_15264_amd import lsmgnn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "lsmgnn.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(lsmgnn.LIB_PATH):
        from paper_2407_15264_amd import build
        build.build_hip()
    return lsmgnn.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(lsmgnn_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("lsmgnn_cache_create", "lsmgnn_cache_destroy", "lsmgnn_gather", "lsmgnn_advance",
                     "lsmgnn_stats", "lsmgnn_export_state"):
        assert required in names


def test_library_exports_every_declared_symbol(L):
    raw = ctypes.CDLL(lsmgnn.LIB_PATH)
    for name in declared_functions():
        assert hasattr(raw, name), name


def test_strerror(L):
    for code in range(7):
        assert L.lsmgnn_strerror(code)
    assert b"range" in L.lsmgnn_strerror(lsmgnn.E_RANGE)


def test_set_index_helper_matches_oracle(L):
    rng = np.random.default_rng(0)
    for x in rng.integers(0, 1 << 32, 200):
        for S in (1, 7, 2048, 13107, 6291456):
            assert lsmgnn.set_of(int(x), S) == oracle_set_of(int(x), S)


@pytest.mark.parametrize("bad", [dict(num_sets=0), dict(row_bytes=24), dict(lookahead=32), dict(max_batch=0),
                                 dict(num_nodes=0), dict(num_nodes=1 << 32), dict(flags=2), dict(flags=1 << 31),
                                 dict(flags=1, host_threads=257), dict(policy=4), dict(policy=1 << 31),
                                 dict(victim_mode=2), dict(victim_mode=1, victim_rows=1, lookahead=1)])
def test_bad_config_rejected_before_device(L, bad):
    stat = np.ones(16, np.uint32)
    store = np.zeros(16 * 16, np.uint8)
    kw = dict(num_nodes=16, row_bytes=16, num_sets=2, victim_rows=2, max_batch=8, lookahead=1, near_threshold=0,
              device=0, flags=0, host_threads=0, policy=0, victim_mode=0, refresh_period=0)
    kw.update(bad)
    cfg = lsmgnn.Config(kw["num_nodes"], kw["row_bytes"], kw["num_sets"], kw["victim_rows"], kw["max_batch"],
                        kw["lookahead"], kw["near_threshold"], kw["device"], kw["flags"], kw["host_threads"],
                        kw["policy"], kw["victim_mode"], kw["refresh_period"], ctypes.c_void_p(store.ctypes.data),
                        ctypes.c_void_p(stat.ctypes.data))
    h = ctypes.c_void_p()
    assert L.lsmgnn_cache_create(ctypes.byref(cfg), ctypes.byref(h)) == lsmgnn.E_INVAL
    assert not h.value


def test_null_arguments(L):
    h = ctypes.c_void_p()
    assert L.lsmgnn_cache_create(None, ctypes.byref(h)) == lsmgnn.E_INVAL
    assert L.lsmgnn_gather(None, None, 0, None, None, None, None, None, None) == lsmgnn.E_INVAL
    assert L.lsmgnn_advance(None, None, 0, None) == lsmgnn.E_INVAL
    assert L.lsmgnn_stats(None, None, None) == lsmgnn.E_INVAL


def test_struct_layouts_match_header(tmp_path):
    # The ctypes mirrors must place every field where a C compiler does.
    import subprocess
    structs = {"lsmgnn_config": lsmgnn.Config, "lsmgnn_counts": lsmgnn.Counts, "lsmgnn_profile": lsmgnn.Profile}
    lines = ["#include <stddef.h>", "#include <stdio.h>", '#include "lsmgnn.h"', "int main(void) {"]
    for name, cls in structs.items():
        lines.append(f'  printf("{name} %zu\\n", sizeof({name}));')
        for f, _ in cls._fields_:
            lines.append(f'  printf("{name}.{f} %zu\\n", offsetof({name}, {f}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    inc = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")
    subprocess.run(["gcc", "-std=c11", "-I", inc, str(src), "-o", str(exe)], check=True)
    got = dict(line.split() for line in subprocess.run([str(exe)], check=True, capture_output=True,
                                                       text=True).stdout.splitlines())
    for name, cls in structs.items():
        assert int(got[name]) == ctypes.sizeof(cls), name
        for f, _ in cls._fields_:
            assert int(got[f"{name}.{f}"]) == getattr(cls, f).offset, f"{name}.{f}"


def test_binding_rejects_host_tensors_before_calling_the_library(L):
    """Device pointers come only from device tensors: host tensors are refused
    in the binding, before anything reaches the library."""
    torch = pytest.importorskip("torch")
    off = torch.zeros(11, dtype=torch.int64)
    adj = torch.zeros(4, dtype=torch.int32)
    with pytest.raises(TypeError):
        lsmgnn.GpuSampler(off, adj, (3,))
    ids = torch.zeros(4, dtype=torch.int64)
    with pytest.raises(TypeError):
        lsmgnn.split_by_type_async(ids, torch.zeros(10, dtype=torch.uint8), torch.zeros(10, dtype=torch.int32),
                                   [torch.zeros(4, dtype=torch.int64)], torch.zeros(64, dtype=torch.uint8), 0)
    with pytest.raises(ValueError):
        lsmgnn.split_by_type_async(ids, torch.zeros(10, dtype=torch.uint8), torch.zeros(10, dtype=torch.int32),
                                   [], torch.zeros(64, dtype=torch.uint8), 0)
