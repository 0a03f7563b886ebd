"""The C ABI from plain C: include/headguard.h compiles as C11 with every
warning an error, a C program links against libheadguard.so and, on a GPU,
quantizes, dequantizes and runs the one-pass form through the C entry points
alone (tests/c_abi/roundtrip.c states what it checks)."""
import os
import subprocess
import sys

import pytest

from conftest import ROOT

sys.path.insert(0, os.path.join(ROOT, "tests", "c_abi"))
import build as c_abi_build  # noqa: E402


def test_header_compiles_as_c_and_links(tmp_path):
    exe = c_abi_build.build(str(tmp_path / "hg_c_roundtrip"))
    assert os.path.exists(exe)


@pytest.mark.gpu
def test_c_client_round_trip():
    exe = c_abi_build.EXE
    if not os.path.exists(exe):
        c_abi_build.build()
    r = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == "ok", (r.returncode, r.stdout, r.stderr)
