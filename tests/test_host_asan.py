"""The CPU suite against a host AddressSanitizer build of the library
(tests/host_asan.py): argument checks, descriptors, the tile derivations and
the plan logic run with every host-side memory access checked."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SCRIPT = os.path.join(ROOT, "tests", "host_asan.py")


@pytest.mark.timeout(900)
def test_cpu_suite_is_clean_under_host_asan():
    if os.environ.get("ATTN_HOST_ASAN"):
        pytest.skip("this is the suite the sanitizer run itself started")
    if not os.path.exists(SCRIPT):
        pytest.skip("the sanitizer script is not part of this copy of the tree")
    r = subprocess.run([sys.executable, SCRIPT], capture_output=True, text=True, timeout=900)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "AddressSanitizer" not in out and " passed" in out
