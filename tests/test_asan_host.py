"""The C ABI's host code under AddressSanitizer: argument validation,
workspace carving and size queries (api.hip, instrumented for the host only)
run the host-side tests with the sanitizer runtime preloaded.  No GPU is
touched: every call in those tests returns before any launch."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
def test_host_code_under_address_sanitizer():
    sys.path.insert(0, ROOT)
    from paper_2510_18830_amd import build as B
    lib = B.build_asan()
    env = dict(os.environ, MSPARSE_LIBRARY=lib, LD_PRELOAD=B.asan_runtime(),
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_lib_host.py"), os.path.join(ROOT, "tests", "test_zz_no_alloc.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-3000:]
    assert "AddressSanitizer" not in out, out[-3000:]
    assert " passed" in out
