"""The C ABI from a plain C program on the GPU (tests/c_client.c, built by
__graft_entry__.build()): device buffers from the HIP runtime, a stream of its own, and the
hand-worked ensemble's scores and leaf ids compared exactly."""
from __future__ import annotations

import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_client")


def test_c_client_on_the_gpu():
    assert os.path.exists(EXE), f"{EXE} is missing: run __graft_entry__.build()"
    r = subprocess.run([EXE, "gpu"], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c_client gpu: ok" in r.stdout
