"""Host-only test of the copy pool that fills the pinned bounce buffers of pageable-master staging.

The pool's source is plain C++; the check program (tests/native/copy_pool_check.cpp) is built with
g++ and asks freshly started pools for copies at once, the window in which a worker that sized its
share from a still-growing thread list left part of a copy to no thread.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "..", "paper_2606_21868_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_fresh_pools_copy_every_byte(tmp_path):
    exe = str(tmp_path / "copy_pool_check")
    subprocess.run(["g++", "-O2", "-std=c++17", "-pthread", "-I", CSRC, os.path.join(HERE, "native", "copy_pool_check.cpp"),
                    os.path.join(CSRC, "copy_pool.cpp"), "-o", exe], check=True, timeout=120)
    r = subprocess.run([exe, "400"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.startswith("ok"), r.stdout + r.stderr
