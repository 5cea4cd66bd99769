"""bench.py's command-line contract on the CPU (no GPU): one GPU only, with a
message for more; the workload names and options it accepts."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = _bench("--gpus", "2", "--steps", "5", "--warmup", "1")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_options_and_workload_names():
    r = _bench("--help")
    assert r.returncode == 0
    for opt in ("--gpus", "--steps", "--warmup", "--workload", "--policy", "--victim-mode", "--refresh-period",
                "--static", "--train-us", "--sync", "--no-cpu-baseline"):
        assert opt in r.stdout, opt
    from paper_2407_15264_amd import workload as W
    for name in W.WORKLOADS:
        assert name in r.stdout, name
    bad = _bench("--workload", "no-such-workload")
    assert bad.returncode != 0


def test_steady_state_start():
    """The timed minibatches start after max(L+1, 10 %) of the configured run."""
    sys.path.insert(0, ROOT)
    import bench
    from paper_2407_15264_amd import workload as W
    want = {W.RMAT14: 3, W.RMAT20: 20, W.RMAT10M: 50, W.TYPED20M: 50, W.RMAT100M: 100}
    for name, first in want.items():
        cfg = W.WORKLOADS[name]
        L = cfg.lookahead if isinstance(cfg, W.HeteroConfig) else cfg.cache.lookahead
        assert bench.steady_start(cfg, L) == first, name
