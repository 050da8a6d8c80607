"""Pins of the oracle's chunk keys and probe-only lookup (CPU)."""

import numpy as np
import pytest

import oracle
from oracle_side import build_case
from workloads import generate, get_config


def test_chain_prefix_sensitivity():
    """Changing one token of chunk i changes h_j for every j >= i and no j < i."""
    rng = np.random.default_rng(7)
    C, N = 16, 9
    toks = rng.integers(0, 129280, N * C + 5, dtype=np.int32)
    base = oracle.chain_keys(toks, C, salt=12345)
    assert len(base) == N                       # the 5-token tail is never keyed
    for i in range(N):
        t2 = toks.copy()
        t2[i * C + int(rng.integers(0, C))] ^= 1
        k2 = oracle.chain_keys(t2, C, salt=12345)
        for j in range(N):
            assert (k2[j] != base[j]) == (j >= i), (i, j)
    # the tail never influences any key
    t3 = toks.copy()
    t3[-1] ^= 7
    assert oracle.chain_keys(t3, C, 12345) == base


def test_chain_brute_force_tiny():
    """Keys of a 2-chunk sequence written out byte by byte from the FNV-1a steps."""
    toks = np.array([1, 2, 3, 4, -1, 0x01020304], dtype=np.int32)
    C = 3
    P, B0, M = 0x100000001B3, 0xCBF29CE484222325, 2**64

    def f(bs, h=B0):
        for x in bs:
            h = ((h ^ x) * P) % M
        return h

    le = lambda v, n: [(v >> (8 * j)) & 0xFF for j in range(n)]  # noqa: E731
    d0 = f(le(1, 4) + le(2, 4) + le(3, 4))
    d1 = f(le(4, 4) + [0xFF] * 4 + [4, 3, 2, 1])
    salt = 99
    h0 = f(le(salt, 8) + le(d0, 8))
    h1 = f(le(h0, 8) + le(d1, 8))
    assert oracle.chain_keys(toks, C, salt) == [h0, h1]


def test_new_salt_gives_fresh_keys_and_zero_hits():
    wi = generate(get_config(1))
    case = build_case(wi, tiny_payloads=True, with_pools=False)
    n, bm, keys = oracle.probe(case.store, wi.tokens, 64, wi.salt)
    assert n == 16 and bm.all()
    n2, bm2, keys2 = oracle.probe(case.store, wi.tokens, 64, wi.salt + 2)
    assert n2 == 0 and not bm2.any()
    assert not set(keys) & set(keys2)


def test_empty_store_and_force_local():
    wi = generate(get_config(1))
    empty = oracle.OracleStore(1)
    assert oracle.probe(empty, wi.tokens, 64, wi.salt)[0] == 0
    case = build_case(wi, tiny_payloads=True, with_pools=False)
    n, bm, _ = oracle.probe(case.store, wi.tokens, 64, wi.salt, force_local=True)
    assert n == 0 and not bm.any()


def test_hole_gives_prefix_but_bitmap_shows_later_hits():
    wi = generate(get_config(1))
    case = build_case(wi, tiny_payloads=True, with_pools=False)
    case.store.remove(case.keys[5], 0)
    n, bm, _ = oracle.probe(case.store, wi.tokens, 64, wi.salt)
    assert n == 5
    assert bm[:5].all() and bm[5] == 0 and bm[6:].all()


def test_probe_does_not_modify_store():
    wi = generate(get_config(1))
    case = build_case(wi, tiny_payloads=True, with_pools=False)
    before = dict(case.store._entries)
    oracle.probe(case.store, wi.tokens, 64, wi.salt)
    assert case.store._entries.keys() == before.keys()


def test_config3_prefix_is_exactly_75_percent():
    """Workload 3 holds the first 384 of 512 chunks: the probe must return 384."""
    wi = generate(get_config(3), values=False)
    case = build_case(wi, tiny_payloads=True, with_pools=False)
    n, bm, keys = oracle.probe(case.store, wi.tokens, 256, wi.salt)
    assert len(keys) == 512
    assert n == 384 and n * 256 == 98_304
    assert bm[:384].all() and not bm[384:].any()


def test_one_group_missing_before_probe_shortens_prefix():
    wi = generate(get_config(2), values=False)
    case = build_case(wi, tiny_payloads=True, with_pools=False)
    case.store.remove(case.keys[40], 1)
    assert oracle.probe(case.store, wi.tokens, 256, wi.salt)[0] == 40
