"""Host-side page pool and sequence table (C++), built with g++ and run on the CPU.

Also built once with AddressSanitizer and UndefinedBehaviorSanitizer."""
import os
import shutil
import subprocess

import pytest


@pytest.mark.parametrize("sanitize", [False, True])
def test_kvpool_cpp(repo_root, tmp_path, sanitize):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "kvpool_test")
    flags = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer"] if sanitize else []
    cmd = [gxx, "-std=c++17", "-O1", "-g", *flags, os.path.join(repo_root, "tests", "kvpool_test.cpp"),
           os.path.join(repo_root, "paper_2411_03519_amd", "csrc", "kv_pool.cpp"), "-o", exe]
    subprocess.run(cmd, check=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "kvpool ok" in r.stdout
