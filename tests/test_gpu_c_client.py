"""The library driven from plain C: tests/c/abi_smoke.c (built by the package
build next to libquake.so) allocates with the HIP runtime, calls the C ABI of
include/quake.h and checks row sums, exact powers of two and argument
validation. No Python binding or torch code is involved in the calls."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLIENT = os.path.join(ROOT, "tests", "c", "abi_smoke")

pytestmark = pytest.mark.gpu


def test_c_client_runs_clean():
    assert os.path.exists(CLIENT), "build the package first (python -m paper_2412_00408_amd.build)"
    print("[gpu-case] C client", CLIENT, flush=True)
    r = subprocess.run([CLIENT], capture_output=True, text=True, timeout=60)
    print(r.stdout)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi smoke passed" in r.stdout
