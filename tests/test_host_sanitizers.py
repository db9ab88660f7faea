"""The host code of libgnmr under AddressSanitizer and UndefinedBehaviorSanitizer:
the ABI tests (argument checks, work lists, overlap checks, error paths, all
before any device call) run in a child process against a build whose host
code is instrumented and aborts on any report.  CPU only."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_abi_tests_are_clean_under_host_sanitizers(tmp_path):
    from paper_2606_00539_amd import _build

    runtime = _build.sanitizer_runtime()
    if runtime is None:
        pytest.skip("no clang AddressSanitizer runtime in this toolchain")
    lib = _build.build_host_sanitized(str(tmp_path / "libgnmr_hostsan.so"))
    log = tmp_path / "san"
    env = dict(os.environ, GNMR_LIBRARY=lib, LD_PRELOAD=runtime,
               ASAN_OPTIONS=f"detect_leaks=0:alloc_dealloc_mismatch=0:log_path={log}",
               UBSAN_OPTIONS=f"print_stacktrace=1:log_path={log}")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", os.path.join(ROOT, "tests", "test_abi.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    reports = sorted(glob.glob(str(log) + "*"))
    text = "".join(open(f).read()[:4000] for f in reports)
    assert not reports, f"sanitizer reports:\n{text}"
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert " passed" in r.stdout
