"""Both staging-copy paths against the oracle (GPU).

By default a library kernel stages each run of chunks from pinned host memory
into the ring; BSR_FLAG_SDMA_COPIES selects the copy engine instead, and a
store arena that HIP does not report pinned is always copied by the copy
engine.  Each path must leave the same bytes as the oracle.
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_side import GpuCase, layout_of, say
from oracle_side import build_case
from paper_2608_17826_amd import bsr
from paper_2608_17826_amd.session import RestoreSession, group_dsts
from workloads import generate, get_config
from workloads.device import place
from workloads.gen import random_workload

pytestmark = pytest.mark.gpu


def _oracle(wi, W):
    case = build_case(wi)
    n, _, keys = oracle.probe(case.store, wi.tokens, wi.workload.chunk_tokens, wi.salt)
    res = oracle.windowed_restore(case.layout, case.store, keys, n, W, wi.block_tables, case.pools, case.valid)
    return case, n, res


def _check(wi, case, res, out, pools, valid):
    assert out.exposed_tokens == res.exposed_tokens and out.fallback == 0
    assert out.stats["h2d_bytes"] == res.h2d_bytes
    for g in range(len(wi.workload.groups)):
        np.testing.assert_array_equal(valid[g].cpu().numpy(), case.valid[g])
        got = np.stack([p.cpu().numpy() for p in pools[g]])
        np.testing.assert_array_equal(got, case.pools[g], err_msg=f"pool of group {g}")


@pytest.mark.parametrize("W,batch", [(32, 0), (8, 0), (8, 8)])
def test_copy_engine_staging_parity(W, batch):
    wi = generate(get_config(2))
    say(f"case: workload 2 (32K), W={W}, batch={batch}, copy-engine staging")
    case, n, res = _oracle(wi, W)
    gc = GpuCase(wi, W=W, install_batch=batch, flags=bsr.BSR_FLAG_SDMA_COPIES)
    try:
        assert gc.probe(1)[0] == n
        out = gc.restore(1, n)
        _check(wi, case, res, out, gc.dev.pools, gc.dev.valid)
        assert out.stats["n_stage_launches"] == 0
    finally:
        gc.close()


@pytest.mark.parametrize("seed", [1, 4, 9, 13])
def test_copy_engine_staging_random_layouts(seed):
    w = random_workload(seed)
    wi = generate(w)
    W = w.windows[0]
    say(f"case: random layout seed={seed}, W={W}, copy-engine staging")
    case, n, res = _oracle(wi, W)
    gc = GpuCase(wi, W=W, flags=bsr.BSR_FLAG_SDMA_COPIES)
    try:
        out = gc.restore(2, gc.probe(2)[0])
        _check(wi, case, res, out, gc.dev.pools, gc.dev.valid)
    finally:
        gc.close()


@pytest.mark.parametrize("arena", ["pageable", "pinned"])
def test_adopted_arena(arena):
    """A caller arena: pageable memory (numpy) is copied by the copy engine;
    pinned memory (torch's pinned allocator) by the staging kernel.  Either
    way the image is the oracle's."""
    wi = generate(get_config(2))
    w = wi.workload
    say(f"case: workload 2 (32K), W=32, adopted {arena} arena")
    case, n, res = _oracle(wi, 32)
    layout = layout_of(wi)
    ctx = bsr.bsr_ctx_create(layout, 32, hip_device=0)
    try:
        stride = (bsr.bsr_slot_bytes(layout) + 4095) // 4096 * 4096
        nbytes = stride * (w.held_chunks + 1)
        if arena == "pageable":
            buf = np.zeros(nbytes, dtype=np.uint8)
            addr = buf.ctypes.data
        else:
            buf = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
            addr = buf.data_ptr()
        bsr.bsr_store_adopt(ctx, addr, nbytes)
        keys = bsr.bsr_chunk_keys(wi.salt, wi.tokens, w.chunk_tokens)
        bsr.bsr_store_put_chunks(ctx, [int(k) for k in keys[:w.held_chunks]],
                                 [wi.payloads(i) for i in range(w.held_chunks)])
        dev = place(wi)
        torch.cuda.synchronize()
        sess = RestoreSession(ctx)
        got_n = bsr.bsr_probe(ctx, 3, wi.salt, wi.tokens)[0]
        assert got_n == n
        out = sess.restore(3, n, group_dsts(dev.block_tables, dev.tensor_bases, dev.valid, wi.pool_blocks))
        _check(wi, case, res, out, dev.pools, dev.valid)
        if arena == "pageable":
            assert out.stats["n_stage_launches"] == 0
        else:
            assert out.stats["n_stage_launches"] > 0 and out.stats["stage_bytes"] == res.h2d_bytes
        bsr.bsr_request_end(ctx, 3)
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_staging_kernel_link_rate_reported():
    """The staging kernel's own link measurement runs and reports a rate in
    the range of the copy engine's (both read the same pinned memory)."""
    wi = generate(get_config(1))
    ctx = bsr.bsr_ctx_create(layout_of(wi), 2, hip_device=0)
    try:
        k = bsr.bsr_measure_stage(ctx, 256 << 20, 3)
        e = bsr.bsr_measure_h2d(ctx, 256 << 20, 1, 3)
        say(f"staging kernel {k:.1f} GB/s, copy engine {e:.1f} GB/s")
        assert k > 0.5 * e and e > 0
        with pytest.raises(bsr.BsrError):
            bsr.bsr_measure_stage(ctx, 1000, 1)      # not a multiple of 16
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_scatter_ceiling_measurement():
    """The plain scattered-copy ceiling runs for the layouts' block sizes,
    cold and warm, and rejects block sizes that are not 16-byte multiples."""
    wi = generate(get_config(1))
    ctx = bsr.bsr_ctx_create(layout_of(wi), 2, hip_device=0)
    try:
        for bb in (73_728, 16_896, 16_384):
            cold = bsr.bsr_measure_scatter(ctx, bb, 64 << 20, 2, 1)
            warm = bsr.bsr_measure_scatter(ctx, bb, 64 << 20, 2, 1, bsr.BSR_SCATTER_WARM_SOURCE)
            say(f"{bb} B blocks: {cold:.0f} GB/s cold, {warm:.0f} GB/s warm")
            assert cold > 100 and warm > 100
        with pytest.raises(bsr.BsrError):
            bsr.bsr_measure_scatter(ctx, 1000, 64 << 20, 1, 1)
        with pytest.raises(bsr.BsrError):
            bsr.bsr_measure_scatter(ctx, 16_384, 64 << 20, 1, 1, 2)     # unknown flag
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_timing_flags_are_taken_at_bind():
    """BSR_FLAG_TIME_INSTALL stamps installs only, BSR_FLAG_TIME_STAGE the
    staging launches only; bsr_set_timing changes them for requests bound
    afterwards, never for one already bound."""
    wi = generate(get_config(2))
    say("case: workload 2 (32K), W=32, timing flags per request")
    case, n, res = _oracle(wi, 32)
    gc = GpuCase(wi, W=32, flags=bsr.BSR_FLAG_TIME_INSTALL)
    try:
        def restore(rid, **kw):
            assert gc.probe(rid)[0] == n
            out = gc.restore(rid, n, **kw)
            _check(wi, case, res, out, gc.dev.pools, gc.dev.valid)
            bsr.bsr_request_end(gc.ctx, rid)
            return out.stats

        st = restore(31)
        assert st["install_ms_total"] > 0 and st["n_stage_launches"] > 0 and st["stage_ms_total"] == 0
        bsr.bsr_set_timing(gc.ctx, bsr.BSR_FLAG_TIME_STAGE)
        st = restore(32)
        assert st["install_ms_total"] == 0 and st["stage_ms_total"] > 0
        # changed while bound: this request keeps the flags of its bind
        st = restore(33, after_bind=lambda: bsr.bsr_set_timing(gc.ctx, bsr.BSR_FLAG_TIME_INSTALL))
        assert st["install_ms_total"] == 0 and st["stage_ms_total"] > 0
        st = restore(34)
        assert st["install_ms_total"] > 0 and st["stage_ms_total"] == 0
        with pytest.raises(bsr.BsrError):
            bsr.bsr_set_timing(gc.ctx, bsr.BSR_FLAG_SDMA_COPIES)
    finally:
        gc.close()
