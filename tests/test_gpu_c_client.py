"""The C ABI used from C++ alone (tests/c/abi_client.cpp: include/saef.h and
the HIP runtime, no Python in between), on an MI355X."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


def test_c_client_runs():
    from paper_2008_05823_amd import build as B
    exe = B.CLIENT
    if not os.path.exists(exe):
        B.build_client()
    print(f"[case] C ABI client {exe}", flush=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "abi client ok" in res.stdout
