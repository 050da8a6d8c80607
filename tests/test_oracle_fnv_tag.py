"""Pins of the oracle's hash primitive and entry tag (CPU)."""

import ast
import os

import numpy as np
import pytest

from oracle import fnv0_64, fnv1a64, FNV64_OFFSET_BASIS, FNV64_PRIME, entry_tag

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _vectors():
    out = []
    with open(os.path.join(GOLDEN, "fnv1a64_vectors.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            hx, lit = line.strip().split(" ", 1)
            out.append((int(hx, 16), ast.literal_eval(lit)))
    return out


@pytest.mark.parametrize("expected,data", _vectors())
def test_fnv1a64_published_vectors(expected, data):
    assert fnv1a64(data) == expected


def test_offset_basis_is_fnv0_of_spec_string():
    with open(os.path.join(GOLDEN, "fnv_basis_derivation.txt")) as f:
        lines = [ln.strip() for ln in f if not ln.startswith("#") and ln.strip()]
    s = ast.literal_eval(lines[0])
    assert len(s) == 32
    assert fnv0_64(s) == int(lines[1], 16) == FNV64_OFFSET_BASIS


def test_prime_structure():
    # the 64-bit FNV prime is 2**40 + 2**8 + 0xb3
    assert FNV64_PRIME == 2**40 + 2**8 + 0xB3


def test_fnv1a_streaming_equals_one_shot():
    rng = np.random.default_rng(5)
    a = rng.integers(0, 256, 37, dtype=np.uint8).tobytes()
    b = rng.integers(0, 256, 11, dtype=np.uint8).tobytes()
    assert fnv1a64(b, fnv1a64(a)) == fnv1a64(a + b)


def _tag_bruteforce(payload: bytes) -> int:
    s = x = 0
    for j in range(0, len(payload), 4):
        w = payload[j] | payload[j + 1] << 8 | payload[j + 2] << 16 | payload[j + 3] << 24
        s = (s + w) % 2**32
        x ^= w
    return x << 32 | s


def test_tag_matches_word_loop():
    rng = np.random.default_rng(1)
    for n in (0, 4, 8, 132, 4096 + 12):
        p = rng.integers(0, 256, n, dtype=np.uint8)
        assert entry_tag(p) == _tag_bruteforce(p.tobytes())


def test_tag_detects_any_single_byte_flip():
    rng = np.random.default_rng(2)
    p = rng.integers(0, 256, 1024, dtype=np.uint8)
    t0 = entry_tag(p)
    for _ in range(200):
        q = p.copy()
        j = int(rng.integers(0, p.size))
        q[j] ^= int(rng.integers(1, 256))
        assert entry_tag(q) & 0xFFFFFFFF != t0 & 0xFFFFFFFF


def test_tag_is_order_independent_over_words():
    rng = np.random.default_rng(3)
    p = rng.integers(0, 256, 400, dtype=np.uint8)
    w = p.view("<u4").copy()
    rng.shuffle(w)
    assert entry_tag(w.view(np.uint8)) == entry_tag(p)
