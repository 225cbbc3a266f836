"""The host runtime under AddressSanitizer (CPU only).

libfe_asan.so is the same library with its host code (argument checks,
workspace layouts, chunking, the split arithmetic) built with
-fsanitize=address; build() makes it beside libfe.so.  This test reruns the
host-side ABI tests in a child process that loads that build (FE_LIBRARY) with
the sanitizer runtime preloaded: an out-of-bounds access or use after free in
the host code aborts the child with a report."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_runtime_under_asan():
    from paper_2509_20416_amd import build
    if not os.path.exists(build.LIB_ASAN):
        pytest.skip("libfe_asan.so not built (python -m paper_2509_20416_amd.build --asan)")
    env = dict(os.environ, LD_PRELOAD=build.asan_runtime(), FE_LIBRARY=build.LIB_ASAN,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        "tests/test_abi.py", "tests/test_attn_split.py"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
    assert "AddressSanitizer" not in r.stderr
