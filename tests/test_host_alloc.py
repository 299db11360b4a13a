"""Host entry points under allocation failure (tests/host_alloc_check.cpp):
ICL-table creation fails cleanly with ILPC_ENOSPC, refinement allocates
nothing (so a call either is refused before it changes the table or
completes), and a prefix match that runs out of host memory at any of its
allocations returns ILPC_ENOSPC and leaves the cache as it was."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2507_08523_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_calls_under_allocation_failure(tmp_path):
    exe = tmp_path / "host_alloc_check"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "host_alloc_check.cpp"), os.path.join(CSRC, "prefix_cache.cpp"),
           os.path.join(CSRC, "pair_table.cpp"), "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600)
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-2000:]
    assert "host alloc ok" in res.stdout
