"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer: a C driver
(tests/c/oracle_edges.c) runs every oracle function over special values,
strided and exhaustive bit patterns, masks, extreme temperatures and causal
limits. Any out-of-bounds access, signed overflow, or float-to-int conversion
outside the int range (what the clamp of l before convert_to_int rules out)
aborts the run. CPU only (gcc)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined,float-cast-overflow", "-fno-sanitize-recover=all"]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_edges_clean_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_edges")
    cmd = ["gcc", "-std=c11", "-O1", "-g", "-Wall", "-ffp-contract=off", "-fno-fast-math", *SAN,
           os.path.join(ROOT, "tests", "c", "oracle_edges.c"),
           os.path.join(ROOT, "oracle", "quake_oracle.c"), "-lm", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0 and "asan" in r.stderr.lower():
        pytest.skip("sanitizer runtime not available: " + r.stderr[-300:])
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert run.returncode == 0, run.stdout[-2000:] + run.stderr[-4000:]
    assert "oracle edges passed" in run.stdout
