"""Pins of the oracle's windowed restore, commit and failure handling (CPU).

What pins the install image, other than the oracle itself:
  * brute force, one token and one tensor at a time, on tiny inputs;
  * W-independence: every window size, including the legacy whole-plan
    W = 0, yields the same image (BSR installs the same bytes as a
    whole-plan restore, §2 Prop. 1 and the discussion after it);
  * a gather with numpy fancy indexing through the block table, which reads
    back the token-ordered records of every tensor (the inverse mapping);
  * with an identity block table and block = chunk, the pool of one tensor
    is exactly numpy.concatenate of that tensor's records over the chunks.
"""

import numpy as np
import pytest

import oracle
from oracle_side import build_case, oracle_layout
from workloads import generate, get_config
from workloads.configs import GroupSpec, Workload
from workloads.gen import random_workload


def _restore(wi, W, **kw):
    case = build_case(wi)
    n, _, keys = oracle.probe(case.store, wi.tokens, wi.workload.chunk_tokens, wi.salt)
    res = oracle.windowed_restore(case.layout, case.store, keys, n, W, wi.block_tables,
                                  case.pools, case.valid, **kw)
    return case, n, res


def _bruteforce_pools(wi, n):
    """Per token, per tensor, per byte-range placement from the mapping rule."""
    w = wi.workload
    C = w.chunk_tokens
    pools = [wi.sentinel_pool(g) for g in range(len(w.groups))]
    for g, spec in enumerate(w.groups):
        B, r = spec.block_tokens, spec.record_bytes
        for tau in range(n * C):
            i, q = divmod(tau, C)
            k, o = divmod(tau, B)
            b = int(wi.block_tables[g][k])
            ent = wi.payload(i, g).reshape(spec.n_tensors, C, r)
            for t in range(spec.n_tensors):
                rec = ent[t, q]
                blk = pools[g][t, b]
                if spec.kind == "contig":
                    for j in range(r):
                        blk[o * r + j] = rec[j]
                else:
                    s = spec.split_bytes
                    for j in range(s):
                        blk[o * s + j] = rec[j]
                    for j in range(r - s):
                        blk[B * s + o * (r - s) + j] = rec[s + j]
    return pools


def _gather(wi, pools, n):
    """Token-ordered records of every (group, tensor), read back by block table."""
    w = wi.workload
    out = []
    for g, spec in enumerate(w.groups):
        B, r = spec.block_tokens, spec.record_bytes
        tau = np.arange(n * w.chunk_tokens)
        blocks = wi.block_tables[g][tau // B]
        pos = tau % B
        per_t = []
        for t in range(spec.n_tensors):
            p = pools[g][t]
            if spec.kind == "contig":
                per_t.append(p.reshape(p.shape[0], B, r)[blocks, pos])
            else:
                s = spec.split_bytes
                p1 = p[:, :B * s].reshape(p.shape[0], B, s)[blocks, pos]
                p2 = p[:, B * s:].reshape(p.shape[0], B, r - s)[blocks, pos]
                per_t.append(np.concatenate([p1, p2], axis=1))
        out.append(per_t)
    return out


def _records_in_order(wi, n):
    w = wi.workload
    out = []
    for g, spec in enumerate(w.groups):
        per_t = []
        for t in range(spec.n_tensors):
            per_t.append(np.concatenate(
                [wi.payload(i, g).reshape(spec.n_tensors, w.chunk_tokens, spec.record_bytes)[t]
                 for i in range(n)]) if n else np.zeros((0, spec.record_bytes), np.uint8))
        out.append(per_t)
    return out


def test_config1_bruteforce_and_counters():
    wi = generate(get_config(1))
    case, n, res = _restore(wi, W=2)
    assert n == 16
    expect = _bruteforce_pools(wi, n)
    for g in range(1):
        np.testing.assert_array_equal(case.pools[g], expect[g])
    slot = 2 * 64 * 1152
    assert case.layout.slot_bytes == slot == 147_456
    assert res.exposed_tokens == 1024 and res.fallback == 0 and res.fail_reason == 0
    assert res.n_windows == 8
    assert res.peak_live_staging_bytes == 2 * slot == 294_912
    assert res.h2d_bytes == 16 * slot
    assert res.installed_bytes == 16 * slot == 2_359_296
    assert (case.valid[0] == 1).all()   # the permutation table covers the whole pool


@pytest.mark.parametrize("seed", range(6))
def test_random_layout_bruteforce(seed):
    w = random_workload(seed)
    wi = generate(w)
    case, n, res = _restore(wi, W=w.windows[1])
    expect = _bruteforce_pools(wi, n)
    for g in range(len(w.groups)):
        np.testing.assert_array_equal(case.pools[g], expect[g])


@pytest.mark.parametrize("seed", range(8))
def test_window_size_independence(seed):
    """Every W (and the whole-plan W = 0) installs byte-identical state."""
    w = random_workload(seed)
    wi = generate(w)
    images = []
    for W in tuple(w.windows) + (0,):
        case, n, res = _restore(wi, W=W)
        assert res.fallback == 0
        assert res.peak_live_staging_bytes == oracle.peak_live_staging(n, W, case.layout.slot_bytes)
        assert max(res.trace) <= (W if W else n) * case.layout.slot_bytes
        images.append((case.pools, case.valid))
    for pools, valid in images[1:]:
        for g in range(len(w.groups)):
            np.testing.assert_array_equal(pools[g], images[0][0][g])
            np.testing.assert_array_equal(valid[g], images[0][1][g])


@pytest.mark.parametrize("seed", range(8))
def test_gather_round_trip_and_untouched_bytes(seed):
    w = random_workload(seed)
    wi = generate(w)
    case, n, res = _restore(wi, W=w.windows[0])
    got = _gather(wi, case.pools, n)
    want = _records_in_order(wi, n)
    installed = 0
    for g, spec in enumerate(w.groups):
        for t in range(spec.n_tensors):
            np.testing.assert_array_equal(got[g][t], want[g][t])
            installed += want[g][t].size
        # blocks outside the advertised prefix keep their sentinel bytes
        nb = oracle.request_blocks(n, w.chunk_tokens, spec.block_tokens)
        touched = set(int(b) for b in wi.block_tables[g][:nb])
        untouched = [b for b in range(wi.pool_blocks[g]) if b not in touched]
        sent = wi.sentinel_pool(g)
        np.testing.assert_array_equal(case.pools[g][:, untouched], sent[:, untouched])
        np.testing.assert_array_equal(case.valid[g][untouched], wi.valid_init[g][untouched])
        assert (case.valid[g][sorted(touched)] == 1).all()
    # Theta(|S|): exactly n chunks' record bytes were installed
    assert res.installed_bytes == installed == n * case.layout.chunk_payload_bytes


def test_identity_table_block_equals_chunk_is_concatenate():
    C = 32
    w = Workload(index=77, name="ident", n_tokens=5 * C, chunk_tokens=C,
                 groups=(GroupSpec("x", C, 3, 12, value_kind="bytes"),),
                 windows=(2,), pool_factor=1)
    wi = generate(w)
    wi.block_tables[0] = np.arange(5, dtype=np.int32)
    case, n, res = _restore(wi, W=2)
    assert n == 5
    for t in range(3):
        cat = np.concatenate([wi.payload(i, 0).reshape(3, C, 12)[t].reshape(-1) for i in range(5)])
        np.testing.assert_array_equal(case.pools[0][t].reshape(-1), cat)


def test_planar_block_layout_config2_shape():
    """Config-2 layout, first 3 chunks: planar index-key blocks split values/scales."""
    w0 = get_config(2)
    w = Workload(index=2, name="c2-small", n_tokens=3 * 256, chunk_tokens=256,
                 groups=w0.groups, windows=(2,), base_records=w0.base_records)
    wi = generate(w)
    case, n, res = _restore(wi, W=2)
    assert case.layout.slot_bytes == 9_707_520
    assert case.layout.group_offsets() == [0, 9_437_184]
    got = _gather(wi, case.pools, n)
    want = _records_in_order(wi, n)
    for t in range(8):
        np.testing.assert_array_equal(got[1][t], want[1][t])
    # block 0 of tensor 0 of group B: first 128*128 bytes are fp8 values
    b = int(wi.block_tables[1][0])
    blk = case.pools[1][0, b]
    recs = wi.payload(0, 1).reshape(8, 256, 132)[0, :128]
    np.testing.assert_array_equal(blk[:128 * 128].reshape(128, 128), recs[:, :128])
    np.testing.assert_array_equal(blk[128 * 128:].reshape(128, 4), recs[:, 128:])


def test_expected_block_matches_full_restore():
    w = random_workload(3)
    wi = generate(w)
    case, n, res = _restore(wi, W=2)
    for g, spec in enumerate(w.groups):
        for t in range(spec.n_tensors):
            for b in range(wi.pool_blocks[g]):
                e = oracle.expected_block(case.layout, case.store, case.keys, n, wi.block_tables[g],
                                          g, t, b, wi.sentinel_pool(g)[t, b])
                np.testing.assert_array_equal(e, case.pools[g][t, b])


def test_slot_offsets_align_every_group_to_256():
    """Slot layout reading: each group's entry starts 256-byte aligned inside a
    staged chunk; worked by hand for payloads that are not 256 multiples."""
    from oracle.layout import OracleGroup, OracleLayout
    L = OracleLayout(8, (OracleGroup(4, 3, 12, "contig", 0), OracleGroup(8, 1, 20, "planar", 16)))
    # payloads: 3 tensors x 8 tokens x 12 B = 288 B, then 1 x 8 x 20 = 160 B
    assert [L.payload_bytes(0), L.payload_bytes(1)] == [288, 160]
    assert L.group_offsets() == [0, 512]
    assert L.slot_bytes == 768
    assert L.chunk_payload_bytes == 448
