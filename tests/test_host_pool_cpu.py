"""The host worker pool shared by the PBM channel, the dense runtime and the
fusion: concurrent and nested parallel_for calls (built from the library's
own header with g++, run under ThreadSanitizer when the toolchain has it)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "..", "paper_2608_07152_amd", "csrc")


def _build(tmp_path, extra):
    exe = tmp_path / "pool_stress"
    cmd = ["g++", "-O1", "-g", "-std=c++17", "-pthread", *extra, "-I", CSRC,
           os.path.join(HERE, "native", "pool_stress.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    return exe if r.returncode == 0 else None


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_pool_concurrent_and_nested_jobs(tmp_path):
    exe = _build(tmp_path, ["-fsanitize=thread"])
    reps = "40"
    if exe is None:   # no ThreadSanitizer runtime: a plain build still checks the counts
        exe = _build(tmp_path, [])
        reps = "200"
    assert exe is not None
    r = subprocess.run([str(exe), reps], capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("ok")
    assert "ThreadSanitizer" not in r.stderr, r.stderr
