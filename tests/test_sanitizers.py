"""Host code under sanitizers (no GPU): the C oracle driven through random
streams with AddressSanitizer + UndefinedBehaviorSanitizer, and the library's
host thread pool (the pageable-store row copies) with ThreadSanitizer and with
AddressSanitizer + UBSan."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)

pytestmark = pytest.mark.skipif(shutil.which("gcc") is None or shutil.which("g++") is None,
                                reason="needs gcc/g++")


def _run(cmd_build, exe, args=(), timeout=300):
    subprocess.run(cmd_build, check=True, capture_output=True, timeout=timeout)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=timeout, env=env)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    return r.stdout


def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_random")
    out = _run(["gcc", "-O1", "-g", "-std=c11", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
                "-I", os.path.join(ROOT, "oracle"), os.path.join(HERE, "sanitize", "oracle_random.c"),
                os.path.join(ROOT, "oracle", "oracle.c"), os.path.join(ROOT, "oracle", "pagerank.c"), "-lm",
                "-o", exe], exe, ["1500"])
    assert "ok" in out


@pytest.mark.parametrize("san", ["thread", "address,undefined"])
def test_host_pool_under_sanitizers(tmp_path, san):
    exe = str(tmp_path / "host_pool_check")
    out = _run(["g++", "-O1", "-g", "-std=c++17", f"-fsanitize={san}", "-I",
                os.path.join(ROOT, "paper_2407_15264_amd", "csrc"), os.path.join(HERE, "sanitize", "host_pool_check.cc"),
                "-o", exe, "-lpthread"], exe)
    assert "ok" in out
