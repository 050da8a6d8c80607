"""The file-backed lower tier on the GPU path against the oracle (GPU).

§4 "System topology" (remote store over a lower local tier), §4
"Storage-side concurrency is orthogonal" (load concurrency inside a window)
and the §6.4 outcome table, checked through the C ABI: restores served by
the file tier install exactly the oracle's bytes at any load concurrency,
with or without O_DIRECT; the probe's per-chunk tier choice matches the
oracle's; a tier lost after the probe fails the restore closed.
"""

import gc as pygc

import numpy as np
import pytest
import torch

import oracle
from gpu_side import GpuCase, say
from oracle_side import build_case
from paper_2608_17826_amd import bsr
from workloads import generate, get_config

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


def _free(gc):
    gc.close()
    gc.dev = None
    gc.session = None
    pygc.collect()
    torch.cuda.empty_cache()


def _oracle_tiers(wi, in_remote, in_file, avail=(True, True), W=32, after_probe=None):
    case = build_case(wi, held=0)
    G = len(wi.workload.groups)
    remote, files = oracle.OracleStore(G), oracle.OracleStore(G)
    for i in in_remote:
        remote.put_chunk(case.keys[i], wi.payloads(i))
    for i in in_file:
        files.put_chunk(case.keys[i], wi.payloads(i))
    tiers = [oracle.Tier(remote, avail[0]), oracle.Tier(files, avail[1])]
    n, bm, keys, ct = oracle.probe_tiers(tiers, wi.tokens, wi.workload.chunk_tokens, wi.salt, G)
    if after_probe:
        after_probe(tiers, keys)
    res = oracle.windowed_restore(case.layout, oracle.PlannedStore(tiers, keys, ct), keys, n, W,
                                  wi.block_tables, case.pools, case.valid)
    return case, n, ct, res


@pytest.mark.parametrize("conc,direct", [(1, False), (4, False), (4, True)])
def test_file_tier_only_32k(tmp_path, conc, direct):
    say(f"case: workload 2 (32K) from the file tier only, load concurrency {conc}, O_DIRECT={direct}")
    wi = generate(get_config(2))
    allc = range(128)
    case, n, ct, res = _oracle_tiers(wi, [], allc)
    assert n == 128 and (ct == 1).all()
    gc = GpuCase(wi, W=32, pinned_chunks=[])
    try:
        gc.put_files(str(tmp_path), allc, concurrency=conc, direct=direct)
        gn, bm, _ = gc.probe(1)
        assert gn == n and (bsr.bsr_plan_tiers(gc.ctx, 1, 128) == ct).all()
        out = gc.restore(1, gn)
        assert out.window_errors == [] and out.exposed_tokens == res.exposed_tokens and out.fallback == 0
        st = out.stats
        assert st["file_tier_chunks"] == 128
        assert st["peak_live_staging_bytes"] == res.peak_live_staging_bytes == 32 * 9_707_520
        slot = 9_707_520
        assert st["host_bounce_bytes"] == 2 * conc * (4096 + (slot + 4095) // 4096 * 4096)
        for g in range(2):
            np.testing.assert_array_equal(gc.pool_host(g), case.pools[g])
            np.testing.assert_array_equal(gc.valid_host(g), case.valid[g])
    finally:
        _free(gc)


def test_mixed_tiers_32k(tmp_path):
    say("case: workload 2 (32K), chunks 0-63 pinned, 48-127 in files")
    wi = generate(get_config(2))
    case, n, ct, res = _oracle_tiers(wi, range(64), range(48, 128))
    assert n == 128 and list(ct[:64]) == [0] * 64 and list(ct[64:]) == [1] * 64
    gc = GpuCase(wi, W=32, pinned_chunks=range(64))
    try:
        gc.put_files(str(tmp_path), range(48, 128), concurrency=3)
        gn = gc.probe(2)[0]
        assert gn == 128 and (bsr.bsr_plan_tiers(gc.ctx, 2, 128) == ct).all()
        out = gc.restore(2, gn)
        assert out.exposed_tokens == res.exposed_tokens and out.stats["file_tier_chunks"] == 64
        for g in range(2):
            np.testing.assert_array_equal(gc.pool_host(g), case.pools[g])
            np.testing.assert_array_equal(gc.valid_host(g), case.valid[g])
    finally:
        _free(gc)


def test_outcome_table_through_the_abi(tmp_path):
    """§6.4: remote healthy -> full; remote unavailable, lower tier healthy ->
    full from the lower tier; both absent -> zero; remote lost after the
    probe -> zero (fail closed)."""
    wi = generate(get_config(1))
    allc = range(16)
    gc = GpuCase(wi, W=2)
    try:
        gc.put_files(str(tmp_path), allc, concurrency=2)
        # remote healthy
        out = gc.restore(10, gc.probe(10)[0])
        assert out.exposed_tokens == 1024 and out.stats["file_tier_chunks"] == 0
        bsr.bsr_request_end(gc.ctx, 10)
        # remote unavailable, lower tier healthy
        bsr.bsr_tier_set_available(gc.ctx, bsr.BSR_TIER_PINNED, 0)
        case, n, ct, res = _oracle_tiers(wi, allc, allc, avail=(False, True), W=2)
        gn = gc.probe(11)[0]
        assert gn == n == 16 and (bsr.bsr_plan_tiers(gc.ctx, 11, 16) == 1).all()
        out = gc.restore(11, gn)
        assert out.exposed_tokens == res.exposed_tokens == 1024 and out.stats["file_tier_chunks"] == 16
        np.testing.assert_array_equal(gc.pool_host(0), case.pools[0])
        bsr.bsr_request_end(gc.ctx, 11)
        # both absent
        bsr.bsr_tier_set_available(gc.ctx, bsr.BSR_TIER_FILE, 0)
        assert gc.probe(12)[0] == 0
        out = gc.restore(12, 0)
        assert out.exposed_tokens == 0 and out.fallback == 0
        bsr.bsr_request_end(gc.ctx, 12)
        # remote lost after the probe: fail closed, force-local next time
        bsr.bsr_tier_set_available(gc.ctx, bsr.BSR_TIER_PINNED, 1)
        bsr.bsr_tier_set_available(gc.ctx, bsr.BSR_TIER_FILE, 1)
        case, n, ct, res = _oracle_tiers(wi, allc, allc, W=2,
                                         after_probe=lambda ts, keys: setattr(ts[0], "available", False))
        gn = gc.probe(13)[0]
        bsr.bsr_tier_set_available(gc.ctx, bsr.BSR_TIER_PINNED, 0)
        out = gc.restore(13, gn)
        assert out.exposed_tokens == res.exposed_tokens == 0 and out.fallback == res.fallback == 1
        assert out.status["fail"] == bsr.BSR_FAIL_MISSING and out.status["first_failed_chunk"] == res.first_failed_chunk == 0
        np.testing.assert_array_equal(gc.valid_host(0), case.valid[0])
        assert gc.probe(13)[0] == 0
        bsr.bsr_request_end(gc.ctx, 13)
    finally:
        _free(gc)


@pytest.mark.parametrize("k", [0, 5, 15])
def test_file_entry_removed_after_probe(tmp_path, k):
    say(f"case: workload 1 from files, chunk {k} removed after the probe")
    wi = generate(get_config(1))
    allc = range(16)

    def drop(ts, keys):
        ts[1].store.remove(keys[k], 0)

    case, n, ct, res = _oracle_tiers(wi, [], allc, W=2, after_probe=drop)
    gc = GpuCase(wi, W=2, pinned_chunks=[])
    try:
        gc.put_files(str(tmp_path), allc, concurrency=2, readahead=4)
        n_g, _, keys = gc.probe(20)
        bsr.bsr_file_tier_remove(gc.ctx, int(keys[k]), 0)
        out = gc.restore(20, n_g)
        assert out.exposed_tokens == 0 and out.fallback == 1
        assert out.status["fail"] == bsr.BSR_FAIL_MISSING
        assert out.status["first_failed_chunk"] == res.first_failed_chunk == k
        np.testing.assert_array_equal(gc.valid_host(0), case.valid[0])
    finally:
        _free(gc)


@pytest.mark.parametrize("k", [3, 15])
def test_file_truncated_after_probe(tmp_path, k):
    """A chunk file cut short after the probe holds no complete object: its
    window fails as missing (§4: a retrieve requires complete presence)."""
    say(f"case: workload 1 from files, chunk {k}'s file truncated after the probe")
    wi = generate(get_config(1))
    allc = range(16)

    def drop(ts, keys):
        for g in range(len(wi.workload.groups)):
            ts[1].store.remove(keys[k], g)

    case, n, ct, res = _oracle_tiers(wi, [], allc, W=2, after_probe=drop)
    gc = GpuCase(wi, W=2, pinned_chunks=[])
    try:
        gc.put_files(str(tmp_path), allc, concurrency=2, readahead=4)
        n_g, _, keys = gc.probe(21)
        path = tmp_path / f"{int(keys[k]):016x}.bsr"
        with open(path, "r+b") as f:
            f.truncate(4096 + 1000)                  # the header survives, the body does not
        out = gc.restore(21, n_g)
        assert out.exposed_tokens == 0 and out.fallback == 1
        assert out.status["fail"] == bsr.BSR_FAIL_MISSING
        assert out.status["first_failed_chunk"] == res.first_failed_chunk == k
        np.testing.assert_array_equal(gc.valid_host(0), case.valid[0])
    finally:
        _free(gc)
