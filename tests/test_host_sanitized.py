"""The C ABI's host core built for the CPU under AddressSanitizer and
UndefinedBehaviorSanitizer, with the device launchers stubbed, and run
(CPU only; see tests/host_core/test_host_core.cpp for what it checks).

The host core (selection, cache, plan, schedule, block and stack
orchestration) is compiled by g++ from the same sources the library is
built from; no device code is involved.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_22283_amd", "csrc")
HERE = os.path.join(ROOT, "tests", "host_core")
SOURCES = [os.path.join(CSRC, f) for f in ("host.cpp", "schedule.cpp", "block.cpp")] + [
    os.path.join(HERE, f) for f in ("device_stubs.cpp", "test_host_core.cpp")]


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs g++ and the HIP headers")
def test_host_core_under_sanitizers(tmp_path):
    exe = str(tmp_path / "test_host_core")
    flags = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
             "-fno-sanitize-recover=undefined", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include"]
    build = subprocess.run(["g++"] + flags + SOURCES + ["-o", exe], capture_output=True, text=True)
    assert build.returncode == 0, build.stderr[-4000:]
    # verify_asan_link_order=0: the process may start with other libraries
    # preloaded, which ASan would otherwise refuse to run after
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    out = run.stdout + run.stderr
    assert run.returncode == 0, out[-4000:]
    assert "host core checks passed" in run.stdout
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
