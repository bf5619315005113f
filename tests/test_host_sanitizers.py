"""The C-ABI contract tests (tests/test_abi.py) rerun against a host
sanitizer build of the library: the argument validation, workspace sizing,
side-stream and rearrangement code compiled with clang's address and
undefined-behaviour sanitizers (the HIP kernels' device code is the ordinary
build).  CPU only."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_contract_under_host_sanitizers(tmp_path):
    from paper_2601_14327_amd import build

    try:
        runtime = build.sanitizer_runtime()
    except (RuntimeError, OSError, subprocess.CalledProcessError) as e:
        pytest.skip(f"no clang sanitizer runtime: {e}")
    lib = build.build_host_sanitized(str(tmp_path))
    env = dict(os.environ, LAEP_ABI_TEST_LIB=lib, LD_PRELOAD=runtime,
               ASAN_OPTIONS="detect_leaks=0:alloc_dealloc_mismatch=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", os.path.join(ROOT, "tests", "test_abi.py")],
                       cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                       text=True, timeout=900)
    out = r.stdout
    assert r.returncode == 0, out[-4000:]
    assert "passed" in out and "failed" not in out, out[-2000:]
    assert "AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
