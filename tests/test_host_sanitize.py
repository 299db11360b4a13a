"""The host C++ of the library (prefix cache with and without block lifecycle,
ICL table) under AddressSanitizer + UndefinedBehaviorSanitizer: a random
stress of every host entry point (tests/host_stress.cpp) must run clean."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2507_08523_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_code_clean_under_sanitizers(tmp_path):
    exe = tmp_path / "host_stress"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-fno-omit-frame-pointer", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "host_stress.cpp"), os.path.join(CSRC, "prefix_cache.cpp"),
           os.path.join(CSRC, "pair_table.cpp"), "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600,
                         env={**os.environ, "ASAN_OPTIONS": "detect_leaks=1:halt_on_error=1"})
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-4000:]
    assert "host fuzz ok" in res.stdout
