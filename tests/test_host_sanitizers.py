"""The host side of the library (argument validation, format sizes, header parsing, tuning, launch-plan entry points)
under AddressSanitizer and UndefinedBehaviorSanitizer: libfluxbin_hostsan.so is the library with fluxbin_host.cpp
instrumented (host code only; the device objects are the ordinary build's), and the CPU host-ABI tests run against it
in a child process with the sanitizer runtime preloaded. Any sanitizer report aborts the child and fails this test."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_abi_tests_pass_under_asan_and_ubsan(tmp_path):
    sys.path.insert(0, ROOT)
    from paper_2608_15602_amd import build as b
    try:
        b.hipcc()
    except RuntimeError:
        pytest.skip("hipcc not available")
    lib = b.build_host_sanitized(verbose=False)
    rt = b.asan_runtime()
    assert os.path.exists(rt), rt
    log = tmp_path / "san"
    env = dict(os.environ)
    env.update(LD_PRELOAD=rt, FLUXBIN_LIBRARY=lib,
               ASAN_OPTIONS=f"detect_leaks=0:abort_on_error=1:log_path={log}",
               UBSAN_OPTIONS=f"halt_on_error=1:print_stacktrace=1:log_path={log}")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_host.py"), "-q", "-x",
                        "-p", "no:cacheprovider"], cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    reports = "".join(p.read_text() for p in tmp_path.glob("san*"))
    assert r.returncode == 0 and not reports, (r.stdout[-3000:], r.stderr[-3000:], reports[:5000])
