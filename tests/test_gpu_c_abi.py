"""A torch-free restore on the GPU through the C ABI (GPU).

``tests/c_abi/gpu_restore`` (built by ``build()``) allocates with the HIP
runtime only, stores 43 chunks in bulk, binds, restores them window by
window (W = 8) through a reversed block table and commits; it checks the
pool image (plain concatenation, since a block holds one chunk here; both
planes of the planar group), the valid bytes, the exposure, the staging
peak and the untouched blocks itself, and prints "ok".
"""

import os
import subprocess

import pytest

from gpu_side import say

pytestmark = pytest.mark.gpu

EXE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi", "gpu_restore")


def test_torch_free_restore_through_the_c_abi():
    assert os.path.exists(EXE), f"{EXE} is not built: run __graft_entry__.build()"
    say("case: C ABI consumer, 43 chunks, W=8, reversed block table")
    r = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.startswith("ok 43 chunks"), r.stdout
