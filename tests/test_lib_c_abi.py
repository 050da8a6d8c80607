"""The C ABI from plain C (CPU).

``tests/c_abi/host_abi.c`` includes only ``include/bsr.h`` and links
libbsr.so: no Python, no torch.  It drives a host-only context (keys,
single and bulk store insertion, probe, removal, the file tier, admission
configuration, error codes) and prints what it computed; the keys, tags and
probe result are compared here with the oracle on the same inputs.  The
same driver is then linked against the runtime's host code built with
AddressSanitizer and UndefinedBehaviorSanitizer (host code only; no device
code is instrumented) and must run clean, leaks included.
"""

import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle
from paper_2608_17826_amd import bsr
from workloads.configs import GroupSpec

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "c_abi", "host_abi.c")
CSRC = os.path.join(ROOT, "paper_2608_17826_amd", "csrc")
C, N_CHUNKS = 16, 6
N_TOKENS = C * N_CHUNKS + 5
SALT = 0x9E3779B97F4A7C15
GROUPS = (GroupSpec("c0", 8, 2, 40), GroupSpec("p1", 32, 1, 36, kind="planar", split_bytes=32))


def _fill(n, seed):
    """The driver's xorshift32 byte stream."""
    m = 0xFFFFFFFF
    x = (seed * 2654435761 + 1) & m
    out = np.empty(n, np.uint8)
    for i in range(n):
        x ^= (x << 13) & m
        x ^= x >> 17
        x ^= (x << 5) & m
        out[i] = x & 0xFF
    return out


def _check_output(text):
    out = text.strip().splitlines()
    assert out[-1] == "ok", text
    layout = oracle.OracleLayout.from_specs(C, GROUPS)
    assert int(out[0].split()[1]) == layout.slot_bytes
    tokens = np.array([(i * 7919 % 129280) - 3 for i in range(N_TOKENS)], dtype=np.int32)
    keys = oracle.chain_keys(tokens, C, SALT)
    got_keys = [int(l.split()[2], 16) for l in out if l.startswith("key ")]
    assert got_keys == keys[:N_CHUNKS]
    store = oracle.OracleStore(2)
    for i in range(N_CHUNKS - 1):
        store.put_chunk(keys[i], [_fill(2 * C * 40, 16 * i), _fill(C * 36, 16 * i + 1)])
    for l in out:
        if l.startswith("tag "):
            _, i, g, t = l.split()
            assert int(t, 16) == store.get(keys[int(i)], int(g))[1]
    store.remove(keys[2], 1)
    n, bm, _ = oracle.probe(store, tokens, C, SALT)
    probe = [l for l in out if l.startswith("probe ")][0].split()
    assert int(probe[1]) == n == 2
    assert int(probe[2], 16) == int(np.packbits(bm, bitorder="little")[0])


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_plain_c_consumer_matches_oracle(tmp_path):
    exe = tmp_path / "host_abi"
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", f"-I{ROOT}/include", SRC,
                    f"-L{os.path.dirname(bsr.LIB_PATH)}", "-lbsr",
                    f"-Wl,-rpath,{os.path.dirname(bsr.LIB_PATH)}", "-o", str(exe)], check=True)
    r = subprocess.run([str(exe), str(tmp_path / "tier")], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    _check_output(r.stdout)


HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# host code only: each sanitizer flag applies to the host pass
SANITIZE = "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -Xarch_host -fno-omit-frame-pointer".split()


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not available")
def test_host_code_clean_under_asan_and_ubsan(tmp_path):
    common = ["--offload-arch=gfx950", "-O1", "-g", "-std=c++17", "-fPIC", f"-I{ROOT}/include",
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
    objs = []
    for src, lang in (("bsr_runtime.cpp", []), ("bsr_file_tier.cpp", []), ("bsr_kernels.hip", ["-x", "hip"])):
        o = str(tmp_path / (src + ".o"))
        subprocess.run([HIPCC, *common, *SANITIZE, *lang, "-c", os.path.join(CSRC, src), "-o", o],
                       check=True, capture_output=True)
        objs.append(o)
    drv = str(tmp_path / "drv.o")
    subprocess.run([HIPCC, "-std=c11", "-x", "c", "-g", f"-I{ROOT}/include", *SANITIZE, "-c", SRC, "-o", drv],
                   check=True, capture_output=True)
    exe = str(tmp_path / "host_abi_asan")
    subprocess.run([HIPCC, "--offload-arch=gfx950", *SANITIZE, drv, *objs, "-o", exe, "-lpthread"],
                   check=True, capture_output=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe, str(tmp_path / "tier")], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr and "ERROR: AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    _check_output(r.stdout)
