"""The C-ABI from a plain C99 program on the GPU (no Python binding, no torch in its process):
snapshot, restore and verify results against the C oracle, and the model-state store."""
import os
import subprocess

import pytest

from gpu_util import need_gpu

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c", "build", "abi_gpu")


def test_c_client_on_gpu():
    need_gpu()
    if not os.path.exists(EXE):
        pytest.fail(f"{EXE} is not built: run __graft_entry__.build()")
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and "abi_gpu ok" in r.stdout, r.stdout + r.stderr
