"""The library's host-only sources under the sanitizers (CPU only): the slot table, the predictor,
the allocator and its online controller, and the staging copy pool, driven by random sequences
(tests/native/host_sanitize_check.cpp) in a g++ build with AddressSanitizer and
UndefinedBehaviorSanitizer, and the copy pool again under ThreadSanitizer.  The HIP calls of the
KV pool are host-memory stand-ins in the driver, so the pool's growth, shrink and failure paths run
here too."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2606_21868_amd", "csrc")
INC = os.path.join(ROOT, "include")
HOST_SOURCES = ["slot_table.cpp", "predictor.cpp", "mvwsa.cpp", "copy_pool.cpp"]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")


def _build(tmp_path, name, sanitize, driver, sources):
    exe = str(tmp_path / name)
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", f"-fsanitize={sanitize}",
           "-fno-sanitize-recover=all", "-pthread", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", INC,
           "-I", CSRC, os.path.join(HERE, "native", driver), *[os.path.join(CSRC, s) for s in sources], "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout + r.stderr
    return exe


def _run(exe, *args):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([exe, *args], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0 and r.stdout.strip().startswith("ok"), r.stdout[-4000:] + r.stderr[-4000:]


@pytest.mark.skipif(not os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h"), reason="needs the HIP headers")
def test_host_sources_under_address_and_ub_sanitizers(tmp_path):
    _run(_build(tmp_path, "host_check_asan", "address,undefined", "host_sanitize_check.cpp", HOST_SOURCES))


def test_copy_pool_under_thread_sanitizer(tmp_path):
    _run(_build(tmp_path, "copy_pool_tsan", "thread", "copy_pool_check.cpp", ["copy_pool.cpp"]), "60")
