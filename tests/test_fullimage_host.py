"""The sliced whole-image comparison itself, on the CPU.

The GPU tests at 512K compare every pool byte through ``fullimage`` in
slices.  Here the same code runs on CPU tensors holding the oracle's own
whole-plan image (``oracle.windowed_restore`` into whole pools): it must
accept that image with any slice size, and reject a single changed byte in a
request block, in a block outside the prefix, and a swap of two request
blocks' contents (which a sum or XOR digest would not see).
"""

import numpy as np
import pytest
import torch

import oracle
from fullimage import compare_full_image, compare_untouched_blocks, slice_unit
from oracle_side import build_case
from workloads import generate, get_config
from workloads.configs import Workload
from workloads.gen import random_workload


def _restored(wi, n=None, W=4):
    case = build_case(wi)
    n0, _, keys = oracle.probe(case.store, wi.tokens, wi.workload.chunk_tokens, wi.salt)
    n = n0 if n is None else n
    res = oracle.windowed_restore(case.layout, case.store, keys, n, W, wi.block_tables, case.pools, case.valid)
    assert res.fallback == 0
    pools = [[torch.from_numpy(case.pools[g][t].copy()) for t in range(case.pools[g].shape[0])]
             for g in range(case.layout.n_groups)]
    return case, keys, n, pools


def _small_mtp_layout():
    w5 = get_config(5)
    return Workload(index=5, name="mtp-6", n_tokens=6 * 256 + 100, chunk_tokens=256, groups=w5.groups,
                    windows=(2,), base_records=w5.base_records)


@pytest.mark.parametrize("slice_bytes", [1, 20_000_000, 1 << 40])
def test_accepts_the_oracle_image(slice_bytes):
    wi = generate(_small_mtp_layout())
    case, keys, n, pools = _restored(wi)
    assert n == 6 and slice_unit(case.layout) == 1
    total = compare_full_image(pools, wi, keys, n, store=case.store, log=lambda s: None,
                               slice_bytes=slice_bytes)
    assert total == sum(p.nbytes for p in case.pools)


@pytest.mark.parametrize("seed", range(6))
def test_random_layouts_and_partial_prefix(seed):
    """Ragged layouts (blocks that do not divide the chunk) and a prefix
    shorter than the held chunks."""
    wi = generate(random_workload(seed))
    n_full = wi.workload.n_full_chunks
    case, keys, n, pools = _restored(wi, n=max(1, n_full - 1), W=2)
    compare_full_image(pools, wi, keys, n, store=case.store, log=lambda s: None, slice_bytes=1)


def _first_request_block(wi, g):
    return int(wi.block_tables[g][0])


def test_rejects_one_changed_request_byte():
    wi = generate(_small_mtp_layout())
    case, keys, n, pools = _restored(wi)
    b = int(wi.block_tables[1][3])
    pools[1][57][b, 16_000] ^= 1
    with pytest.raises(AssertionError, match="group 1"):
        compare_full_image(pools, wi, keys, n, store=case.store, log=lambda s: None, slice_bytes=1)


def test_rejects_one_changed_untouched_byte():
    wi = generate(_small_mtp_layout())
    case, keys, n, pools = _restored(wi)
    nreq = oracle.request_blocks(n, 256, wi.workload.groups[2].block_tokens)
    other = int(np.setdiff1d(np.arange(wi.pool_blocks[2]), wi.block_tables[2][:nreq])[5])
    pools[2][20][other, 3] ^= 0x80
    with pytest.raises(AssertionError, match="outside the prefix"):
        compare_untouched_blocks(pools, wi, n, log=lambda s: None)


def test_rejects_two_request_blocks_swapped():
    """Same multiset of words in the group, different placement."""
    wi = generate(_small_mtp_layout())
    case, keys, n, pools = _restored(wi)
    b0, b1 = int(wi.block_tables[0][0]), int(wi.block_tables[0][9])
    p = pools[0][4]
    tmp = p[b0].clone()
    p[b0] = p[b1]
    p[b1] = tmp
    with pytest.raises(AssertionError, match="group 0"):
        compare_full_image(pools, wi, keys, n, store=case.store, log=lambda s: None)
