"""The C ABI from C: include/zq.h compiles as strict C99 / C11 (CPU), and a C
program (tests/c/abi_check.c) drives every entry point on the GPU and matches
the C oracle byte for byte."""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.join(HERE, "c"))
import build as cbuild  # noqa: E402


def test_header_is_strict_c():
    cbuild.syntax_check()


@pytest.mark.gpu
def test_c_program_matches_oracle(tmp_path):
    from paper_2501_04266_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("libzq.so is not built")
    exe = cbuild.build(out=str(tmp_path / "abi_check"))
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi_check ok" in r.stdout
