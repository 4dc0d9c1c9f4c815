"""libzf's host code built with AddressSanitizer and UndefinedBehaviorSanitizer
(sanitizers on the host compilation only; no device code runs) and driven by
tests/native/host_asan_main.cpp: the multithreaded deferred update on
exact-size heap buffers, and the host-side argument validation."""
import importlib.util
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2505_12242_amd", "csrc")


def _library_sources():
    """The library's source list, as the build script compiles it."""
    spec = importlib.util.spec_from_file_location(
        "zf_build", os.path.join(ROOT, "paper_2505_12242_amd", "build.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return list(mod.SOURCES)


SOURCES = _library_sources()


@pytest.mark.timeout(600)
def test_host_code_under_address_and_ub_sanitizers(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "host_asan")
    cmd = [hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-pthread",
           "-ffp-contract=off", "-fno-omit-frame-pointer",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(ROOT, "tests", "native", "host_asan_main.cpp"),
           *[os.path.join(CSRC, s) for s in SOURCES], "-o", exe]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stdout + build.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stdout + run.stderr
    assert "clean under the sanitizers" in run.stdout
