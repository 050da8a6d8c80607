"""Pins of the oracle's fail-closed commit (CPU).

§3 Eq. 6 and Prop. 2: exposure is the complete advertised prefix or zero.
The failure-outcome table of §6.4 gives the categorical outcomes: healthy
restore -> full prefix; both tiers absent -> zero (found by the probe); a
one-component fault after one window -> zero.
"""

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
from oracle_side import build_case
from workloads import generate, get_config
from workloads.gen import random_workload


def _probe(case, wi):
    return oracle.probe(case.store, wi.tokens, wi.workload.chunk_tokens, wi.salt)


def _check_invalidated(case, wi, n, res):
    assert res.exposed_tokens == 0 and res.fallback == 1
    for g, spec in enumerate(wi.workload.groups):
        nb = oracle.request_blocks(n, wi.workload.chunk_tokens, spec.block_tokens)
        req = wi.block_tables[g][:nb]
        assert (case.valid[g][req] == 0).all()
        others = np.setdiff1d(np.arange(wi.pool_blocks[g]), req)
        np.testing.assert_array_equal(case.valid[g][others], wi.valid_init[g][others])
        sent = wi.sentinel_pool(g)
        np.testing.assert_array_equal(case.pools[g][:, others], sent[:, others])


@pytest.mark.parametrize("mode", ["missing", "corrupt"])
@pytest.mark.parametrize("k", [0, 1, 5, 15])
def test_fault_after_probe_invalidates_whole_prefix(mode, k):
    wi = generate(get_config(1))
    case = build_case(wi)
    n, _, keys = _probe(case, wi)
    assert n == 16
    if mode == "missing":
        case.store.remove(keys[k], 0)
    else:
        case.store.corrupt(keys[k], 0, byte=1000, mask=0x5A)
    res = oracle.windowed_restore(case.layout, case.store, keys, n, 2, wi.block_tables,
                                  case.pools, case.valid)
    _check_invalidated(case, wi, n, res)
    assert res.first_failed_chunk == k
    assert res.fail_reason == (oracle.FAIL_MISSING if mode == "missing" else oracle.FAIL_CORRUPT)
    assert res.q == [0]
    assert res.n_windows == k // 2 + 1


def test_group_fault_in_one_group_collapses_every_group():
    """A fault in group B only still invalidates group A's blocks (HMA rule)."""
    from workloads.configs import Workload
    w0 = get_config(2)
    w = Workload(index=2, name="c2-small", n_tokens=6 * 256, chunk_tokens=256,
                 groups=w0.groups, windows=(2,), base_records=w0.base_records)
    wi = generate(w)
    case = build_case(wi)
    n, _, keys = _probe(case, wi)
    case.store.remove(keys[3], 1)
    res = oracle.windowed_restore(case.layout, case.store, keys, n, 2, wi.block_tables,
                                  case.pools, case.valid)
    _check_invalidated(case, wi, n, res)
    assert res.q == [1, 0] and res.first_failed_chunk == 3


@pytest.mark.parametrize("reason", [oracle.FAIL_TIMEOUT, oracle.FAIL_TRANSFER])
def test_host_side_faults(reason):
    wi = generate(get_config(1))
    case = build_case(wi)
    n, _, keys = _probe(case, wi)
    res = oracle.windowed_restore(case.layout, case.store, keys, n, 2, wi.block_tables,
                                  case.pools, case.valid, faults={7: reason})
    _check_invalidated(case, wi, n, res)
    assert res.fail_reason == reason and res.first_failed_chunk == 7


def test_abort_after_window():
    wi = generate(get_config(1))
    case = build_case(wi)
    n, _, keys = _probe(case, wi)
    res = oracle.windowed_restore(case.layout, case.store, keys, n, 2, wi.block_tables,
                                  case.pools, case.valid, abort_after_windows=3)
    _check_invalidated(case, wi, n, res)
    assert res.fail_reason == oracle.FAIL_ABORT and res.q == [1]


def test_failure_outcome_table():
    """§6.4 outcome table, single rank: full / zero via probe / zero after a window."""
    wi = generate(get_config(1))
    # healthy
    case = build_case(wi)
    rt = oracle.Runtime(case.layout, case.store, W=2)
    n, _, keys = rt.probe(1, wi.tokens, wi.salt)
    res = rt.restore(1, keys, n, wi.block_tables, case.pools, case.valid)
    assert res.exposed_tokens == 1024
    # both tiers absent: the probe finds nothing, nothing is restored
    empty = oracle.Runtime(case.layout, oracle.OracleStore(1), W=2)
    n0, _, keys0 = empty.probe(2, wi.tokens, wi.salt)
    res0 = empty.restore(2, keys0, n0, wi.block_tables, case.pools, case.valid)
    assert n0 == 0 and res0.exposed_tokens == 0 and res0.fallback == 0
    # fault after one window (W = 2): chunk 2 missing
    case = build_case(wi)
    rt = oracle.Runtime(case.layout, case.store, W=2)
    n, _, keys = rt.probe(3, wi.tokens, wi.salt)
    case.store.remove(keys[2], 0)
    res = rt.restore(3, keys, n, wi.block_tables, case.pools, case.valid)
    assert res.exposed_tokens == 0 and res.fallback == 1 and res.n_windows == 2


def test_force_local_marker_lifecycle():
    wi = generate(get_config(1))
    case = build_case(wi)
    rt = oracle.Runtime(case.layout, case.store, W=2)
    n, _, keys = rt.probe(9, wi.tokens, wi.salt)
    case.store.corrupt(keys[4], 0, 10, 1)
    res = rt.restore(9, keys, n, wi.block_tables, case.pools, case.valid)
    assert res.fallback == 1
    assert rt.probe(9, wi.tokens, wi.salt)[0] == 0          # next admission: no external tokens
    assert rt.probe(10, wi.tokens, wi.salt)[0] == 16        # other requests unaffected
    rt.request_running(9)
    assert rt.probe(9, wi.tokens, wi.salt)[0] == 16
    res = rt.restore(9, keys, n, wi.block_tables, case.pools, case.valid)
    rt.request_end(9)
    assert rt.probe(9, wi.tokens, wi.salt)[0] == 16


def test_missing_beyond_k_before_probe_commits_shorter_prefix():
    wi = generate(get_config(1))
    case = build_case(wi)
    k = 6
    for i in range(k + 1, 16):
        case.store.remove(case.keys[i], -1)
    n, _, keys = _probe(case, wi)
    assert n == k + 1
    res = oracle.windowed_restore(case.layout, case.store, keys, n, 2, wi.block_tables,
                                  case.pools, case.valid)
    assert res.exposed_tokens == (k + 1) * 64 and res.fallback == 0
    nb = oracle.request_blocks(n, 64, 16)
    assert (case.valid[0][wi.block_tables[0][:nb]] == 1).all()


@settings(max_examples=25, deadline=None)
@given(seed=st.integers(0, 40), W=st.integers(0, 6), pos=st.floats(0, 0.999),
       mode=st.sampled_from(["none", "missing", "corrupt", "timeout", "transfer", "abort"]))
def test_exposure_is_all_or_nothing(seed, W, pos, mode):
    """Prop. 2 under random layouts, windows and injected faults."""
    w = random_workload(seed)
    wi = generate(w)
    case = build_case(wi)
    n, _, keys = _probe(case, wi)
    k = int(pos * n) if n else 0
    G = len(w.groups)
    kw = {}
    if n and mode == "missing":
        case.store.remove(keys[k], seed % G)
    elif n and mode == "corrupt":
        g = seed % G
        case.store.corrupt(keys[k], g, byte=(seed * 7) % case.layout.payload_bytes(g), mask=3)
    elif n and mode == "timeout":
        kw["faults"] = {k: oracle.FAIL_TIMEOUT}
    elif n and mode == "transfer":
        kw["faults"] = {k: oracle.FAIL_TRANSFER}
    elif n and mode == "abort":
        kw["abort_after_windows"] = 1
    res = oracle.windowed_restore(case.layout, case.store, keys, n, W, wi.block_tables,
                                  case.pools, case.valid, **kw)
    assert res.exposed_tokens in (0, n * w.chunk_tokens)
    if n > 0 and mode != "none":
        _check_invalidated(case, wi, n, res)
    else:
        assert res.exposed_tokens == n * w.chunk_tokens and res.fallback == 0
    assert res.peak_live_staging_bytes <= (W if W else max(n, 1)) * case.layout.slot_bytes


def test_group_reported_invalid_without_window_failure():
    """Eq. 6: a group with q_g = 0 alone forbids exposure, no window failure needed."""
    from workloads.configs import Workload
    w0 = get_config(2)
    w = Workload(index=2, name="c2-small", n_tokens=4 * 256, chunk_tokens=256,
                 groups=w0.groups, windows=(2,), base_records=w0.base_records)
    wi = generate(w)
    case = build_case(wi)
    n, _, keys = _probe(case, wi)
    res = oracle.windowed_restore(case.layout, case.store, keys, n, 2, wi.block_tables,
                                  case.pools, case.valid, invalid_groups=[1])
    assert res.fail_reason == oracle.FAIL_NONE and res.q == [1, 0]
    _check_invalidated(case, wi, n, res)
