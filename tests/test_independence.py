"""The product path and the oracle stay apart, and the product path has no
fallback: the binding refuses to import without the built library, nothing in
the package imports, links or reads the oracle, and the oracle uses nothing
of the package (only standard headers and numpy). Checked on the CPU."""
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2412_00408_amd")


def _sources(top, exts):
    for d, _, files in os.walk(top):
        for f in files:
            if f.endswith(exts):
                yield os.path.join(d, f)


def test_binding_raises_without_the_library(tmp_path):
    pkg = tmp_path / "pkg_without_lib"
    pkg.mkdir()
    (pkg / "__init__.py").write_text("")
    with open(os.path.join(PKG, "quake.py")) as f:
        (pkg / "quake.py").write_text(f.read())
    r = subprocess.run([sys.executable, "-c", "import pkg_without_lib.quake"], cwd=tmp_path,
                       capture_output=True, text=True, timeout=300,
                       env=dict(os.environ, PYTHONPATH=str(tmp_path)))
    assert r.returncode != 0
    assert "libquake.so is not built" in r.stderr


def test_product_code_does_not_use_the_oracle():
    pat = re.compile(r"^\s*(import\s+oracle|from\s+oracle\b)|oracle/|quake_oracle", re.M)
    for p in _sources(PKG, (".py", ".hip", ".hpp", ".cpp", ".h")):
        with open(p) as f:
            text = f.read()
        assert not pat.search(text), p


def test_oracle_uses_nothing_of_the_package():
    for p in _sources(os.path.join(ROOT, "oracle"), (".py", ".c", ".h")):
        with open(p) as f:
            text = f.read()
        assert "paper_2412_00408_amd" not in text and "csrc" not in text, p
        for inc in re.findall(r'#include\s*[<"]([^>"]+)[>"]', text):
            assert inc in ("math.h", "stdint.h", "string.h", "stdlib.h", "stdio.h"), (p, inc)
