"""Legacy whole-plan mode (W = 0) against the oracle and against bounded W (GPU).

§4 "Restore-window configuration": zero keeps the legacy whole-plan path,
whose staging holds the complete selected plan (Eq. 2), while a bounded
window holds W chunks (Eqs. 3-5).  Both must install the same bytes (§2: BSR
changes residency, not what is restored).
"""

import gc as pygc

import numpy as np
import pytest
import torch

import oracle
from fullimage import compare_full_image
from gpu_side import GpuCase, measured_restore, say
from paper_2608_17826_amd import bsr
from oracle_side import GeneratorStore, build_case, oracle_layout
from workloads import generate, get_config
from workloads.gen import random_workload

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]


def _free(gc):
    gc.close()
    gc.dev = None
    gc.session = None
    pygc.collect()
    torch.cuda.empty_cache()


def _oracle(wi, W):
    case = build_case(wi)
    n, _, keys = oracle.probe(case.store, wi.tokens, wi.workload.chunk_tokens, wi.salt)
    res = oracle.windowed_restore(case.layout, case.store, keys, n, W, wi.block_tables,
                                  case.pools, case.valid)
    return case, n, res


def test_whole_plan_32k_parity_and_same_image_as_bounded():
    say("case: workload 2 (32K), whole-plan W=0 vs oracle W=0 and vs bounded W=32")
    wi = generate(get_config(2))
    case, n, res = _oracle(wi, 0)
    assert res.peak_live_staging_bytes == 128 * 9_707_520
    images = []
    for W in (0, 32):
        gc = GpuCase(wi, W=W)
        try:
            assert gc.probe(1)[0] == n == 128
            if W == 0:
                # the ring the session allocates for this plan, measured alone
                m0 = torch.cuda.memory_allocated()
                gc.session._ring(bsr.bsr_plan_staging_bytes(gc.ctx, n))
                ring_delta = torch.cuda.memory_allocated() - m0
            out = gc.restore(1, n)
            assert out.exposed_tokens == res.exposed_tokens and out.fallback == 0
            st = out.stats
            want_peak = oracle.peak_live_staging(n, W, case.layout.slot_bytes)
            assert st["peak_live_staging_bytes"] == want_peak
            assert st["staging_required_bytes"] == want_peak
            if W == 0:
                assert gc.session.staging_bytes == gc.session.staging.numel() == 128 * 9_707_520
                # torch's caching allocator places a 1.24 GB block in a 2 MiB-rounded
                # segment and keeps a remainder of at most 1 MiB unsplit
                assert 0 <= ring_delta - 128 * 9_707_520 <= 1 << 20
            images.append([gc.pool_host(g) for g in range(2)] + [gc.valid_host(g) for g in range(2)])
        finally:
            _free(gc)
    for g in range(2):
        np.testing.assert_array_equal(images[0][g], case.pools[g])
        np.testing.assert_array_equal(images[0][2 + g], case.valid[g])
    for a, b in zip(images[0], images[1]):
        np.testing.assert_array_equal(a, b)


@pytest.mark.parametrize("seed", [0, 3, 7])
def test_whole_plan_random_layouts(seed):
    w = random_workload(seed)
    wi = generate(w)
    say(f"case: random layout seed={seed}, whole-plan W=0")
    case, n, res = _oracle(wi, 0)
    gc = GpuCase(wi, W=0)
    try:
        out = gc.restore(2, gc.probe(2)[0])
        assert out.exposed_tokens == res.exposed_tokens
        assert out.stats["peak_live_staging_bytes"] == res.peak_live_staging_bytes
        for g in range(len(w.groups)):
            np.testing.assert_array_equal(gc.pool_host(g), case.pools[g])
            np.testing.assert_array_equal(gc.valid_host(g), case.valid[g])
    finally:
        _free(gc)


def test_capacity_contrast_128k():
    """Whole-plan staging = n x c; bounded = W x c, each measured across its
    restore; both leave every pool byte equal to the oracle's image, so the
    two images are the same byte for byte (§6.1 against §6.2: the same state
    at different capacity)."""
    say("case: workload 3 (128K, 384 held), whole-plan vs W=32")
    wi = generate(get_config(3))
    layout = oracle_layout(wi)
    keys = oracle.chain_keys(wi.tokens, 256, wi.salt)
    store = GeneratorStore(wi, keys)
    peaks = {}
    for W in (0, 32):
        gc = GpuCase(wi, W=W)
        try:
            n = gc.probe(3)[0]
            assert n == 384
            out, m = measured_restore(gc, 3, n)
            assert out.exposed_tokens == 98_304 and out.fallback == 0
            peaks[W] = out.stats["peak_live_staging_bytes"]
            ring = (W or n) * layout.slot_bytes
            assert m["peak_requested_delta"] == ring, m
            # torch may keep a remainder of at most 1 MiB unsplit in the ring's segment
            assert 0 <= m["peak_alloc_delta"] - ring <= 1 << 20, m
            assert m["free_after_commit"] == m["free_after_bind"], m
            valid = [v.copy() for v in wi.valid_init]
            oracle.set_request_valid(layout, n, wi.block_tables, valid, 1)
            for g in range(2):
                np.testing.assert_array_equal(gc.valid_host(g), valid[g])
            compare_full_image(gc.dev.pools, wi, keys, n, store=store, log=say)
        finally:
            _free(gc)
    assert peaks[0] == oracle.peak_live_staging(384, 0, layout.slot_bytes) == 384 * 9_707_520
    assert peaks[32] == oracle.peak_live_staging(384, 32, layout.slot_bytes) == 32 * 9_707_520
