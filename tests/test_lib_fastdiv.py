"""The install kernel's division by invariant integers, checked on the CPU.

Every decode step of ``k_install`` (work item -> chunk, piece, tensor,
block; chunk -> ring slot and block index) divides by a per-layout divisor
with a multiply-high and two shifts whose constants the host builds
(Granlund & Montgomery 1994).  ``tests/c_abi/fastdiv_check.hip`` includes the
library's own header and compares that division with ``n / d`` for every
divisor up to 2^16 and a spread of larger ones, at and around multiples, at
the ends of the 32-bit range and at pseudo-random numerators.  Host code
only: it runs without a GPU.
"""

import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_abi", "fastdiv_check.hip")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_packed_division_matches_integer_division(tmp_path):
    exe = str(tmp_path / "fastdiv_check")
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-O2", "-std=c++17", "-x", "hip",
                    f"-I{ROOT}/include", f"-I{ROOT}/paper_2608_17826_amd/csrc",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", SRC, "-o", exe],
                   check=True, capture_output=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    lines = r.stdout.strip().splitlines()
    assert lines[-1] == "ok", r.stdout[-2000:]
    assert int(lines[-2].split()[1]) > 40_000_000  # 43.6 million comparisons
