"""Pins of the oracle's tier choice (CPU): the §6.4 outcome table."""

import numpy as np

import oracle
from oracle_side import build_case
from workloads import generate, get_config


def _two_tiers(wi, in_remote, in_ssd):
    case = build_case(wi)
    remote, ssd = oracle.OracleStore(1), oracle.OracleStore(1)
    for i in in_remote:
        remote.put_chunk(case.keys[i], wi.payloads(i))
    for i in in_ssd:
        ssd.put_chunk(case.keys[i], wi.payloads(i))
    return case, [oracle.Tier(remote), oracle.Tier(ssd)]


def _restore(case, wi, tiers, force_local=False, after_probe=None):
    n, bm, keys, ct = oracle.probe_tiers(tiers, wi.tokens, 64, wi.salt, 1, force_local)
    if after_probe:
        after_probe(tiers, keys)
    store = oracle.PlannedStore(tiers, keys, ct)
    res = oracle.windowed_restore(case.layout, store, keys, n, 2, wi.block_tables, case.pools, case.valid)
    return n, ct, res


def test_outcome_table():
    wi = generate(get_config(1))
    allc = range(16)
    # remote healthy: full reuse, every chunk from the remote tier
    case, tiers = _two_tiers(wi, allc, allc)
    n, ct, res = _restore(case, wi, tiers)
    assert n == 16 and (ct == 0).all() and res.exposed_tokens == 1024
    # remote unavailable, SSD healthy: the complete prefix from SSD
    case2, tiers2 = _two_tiers(wi, allc, allc)
    tiers2[0].available = False
    n, ct, res2 = _restore(case2, wi, tiers2)
    assert n == 16 and (ct == 1).all() and res2.exposed_tokens == 1024
    for g in range(1):
        np.testing.assert_array_equal(case.pools[g], case2.pools[g])
    # remote + SSD absent: zero external reuse (found by the probe)
    case3, tiers3 = _two_tiers(wi, [], [])
    n, ct, res3 = _restore(case3, wi, tiers3)
    assert n == 0 and res3.exposed_tokens == 0 and (ct == oracle.NO_TIER).all()


def test_mixed_tiers_and_lower_tier_extends_prefix():
    wi = generate(get_config(1))
    case, tiers = _two_tiers(wi, range(8), range(4, 16))
    n, ct, res = _restore(case, wi, tiers)
    assert n == 16 and list(ct[:8]) == [0] * 8 and list(ct[8:]) == [1] * 8
    ref, rtiers = _two_tiers(wi, range(16), [])
    _restore(ref, wi, rtiers)
    np.testing.assert_array_equal(case.pools[0], ref.pools[0])


def test_tier_lost_after_probe_fails_closed():
    wi = generate(get_config(1))
    case, tiers = _two_tiers(wi, range(16), range(16))

    def drop(ts, keys):
        ts[0].available = False     # the remote store goes away mid-request

    n, ct, res = _restore(case, wi, tiers, after_probe=drop)
    assert n == 16 and res.exposed_tokens == 0 and res.fallback == 1
    assert res.fail_reason == oracle.FAIL_MISSING and res.first_failed_chunk == 0
