"""The LDS-poisoning debug build (`python -m paper_2608_21343_amd.build
--poison`: every kernel fills its LDS with all bits set before use) decodes
like the product build, so no kernel reads an LDS word it has not written.

The checks (tests/poison_checks.py) run in a child process that imports the
package from a temporary copy whose library is the poison build."""

import os
import shutil
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2608_21343_amd")


def test_lds_poison_build_matches_the_oracle(tmp_path):
    lib = os.path.join(PKG, "libtbias_poison.so")
    if not os.path.exists(lib):
        pytest.skip("libtbias_poison.so is not built (python -m paper_2608_21343_amd.build --poison)")
    dst = tmp_path / "paper_2608_21343_amd"
    dst.mkdir()
    for f in os.listdir(PKG):
        if f.endswith(".py"):
            shutil.copy(os.path.join(PKG, f), dst / f)
    shutil.copy(lib, dst / "libtbias.so")
    r = subprocess.run([sys.executable, "-u", os.path.join(ROOT, "tests", "poison_checks.py"),
                        str(tmp_path)], capture_output=True, text=True, timeout=900)
    print(r.stdout[-3000:])
    assert r.returncode == 0, (r.stdout[-4000:], r.stderr[-4000:])
    assert "poison checks: ok" in r.stdout
