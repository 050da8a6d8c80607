"""The context that allocates nothing against the ordinary one (GPU).

``bsr_ctx_create_static`` gives a context whose device scratch (the install
kernel's tag partials and the verify words) is the library's static per-GPU
array instead of memory allocated at context creation.  Through the C ABI,
one such context restores several requests in a row, each checked byte for
byte against the same request restored by an ordinary context
(``bsr_ctx_create``) and against the oracle:
  * the whole 32K workload, then a smaller prefix of it (the array keeps the
    first request's contents);
  * then a request with a corrupt entry (verify words left set by a
    mismatch), and the whole workload again (the next bind clears them).
Also: a second such context on the same GPU is refused while the first
exists, a layout whose scratch exceeds the array is refused, and creating
the context changes neither torch's allocations nor the device's free bytes.
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
from workloads.configs import GroupSpec, Workload
from workloads.device import place

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]


def _oracle(wi, n, W, mutate=None):
    case = build_case(wi)
    n0, _, keys = oracle.probe(case.store, wi.tokens, wi.workload.chunk_tokens, wi.salt)
    assert n <= n0
    if mutate:
        mutate(case, keys)
    res = oracle.windowed_restore(case.layout, case.store, keys, n, W, wi.block_tables, case.pools, case.valid)
    return case, res


def _fresh_pools(gc):
    gc.dev = place(gc.wi)
    torch.cuda.synchronize()


def _same(gs, go, case, res, G, success):
    """The static context's outcome and image equal the ordinary one's and the oracle's."""
    (out_s, gc_s), (out_o, gc_o) = gs, go
    for k in ("exposed_tokens", "fallback"):
        assert getattr(out_s, k) == getattr(out_o, k)
    assert out_s.exposed_tokens == res.exposed_tokens and out_s.fallback == res.fallback
    for k in ("fail", "first_failed_chunk", "q", "exposed_tokens", "fallback", "phase"):
        assert out_s.status[k] == out_o.status[k], k
    assert out_s.status["q"][:G] == res.q
    assert out_s.status["first_failed_chunk"] == res.first_failed_chunk
    for k in ("h2d_bytes", "installed_bytes", "peak_live_staging_bytes", "n_windows", "n_install_launches"):
        assert out_s.stats[k] == out_o.stats[k], k
    for g in range(G):
        np.testing.assert_array_equal(gc_s.valid_host(g), gc_o.valid_host(g))
        np.testing.assert_array_equal(gc_s.valid_host(g), case.valid[g])
        a, b = gc_s.pool_host(g), gc_o.pool_host(g)
        if success:
            np.testing.assert_array_equal(a, b, err_msg=f"pool of group {g}")
            np.testing.assert_array_equal(a, case.pools[g], err_msg=f"pool of group {g} vs oracle")
        else:   # request blocks are unspecified after a failure; the rest is not
            nreq = oracle.request_blocks(out_s.stats["n_hit_chunks"], 256, gc_s.wi.workload.groups[g].block_tokens)
            others = np.setdiff1d(np.arange(gc_s.wi.pool_blocks[g]), gc_s.wi.block_tables[g][:nreq])
            np.testing.assert_array_equal(a[:, others], b[:, others])
            np.testing.assert_array_equal(a[:, others], case.pools[g][:, others])


def test_static_context_matches_ordinary_on_requests_in_a_row():
    wi = generate(get_config(2))
    G = len(wi.workload.groups)
    say("case: workload 2 (32K), W=32: static and ordinary contexts side by side")
    go = GpuCase(wi, W=32)
    gs = GpuCase(wi, W=32, static=True)
    try:
        plan = [("full", 128, None), ("smaller", 40, None), ("corrupt", 128, (70, 1, 4321, 0x5A)),
                ("full again", 128, None)]
        for j, (name, n, bad) in enumerate(plan):
            say(f"  request {j}: {name}, {n} chunks")
            rid = 500 + j
            outs = []
            for gc in (gs, go):
                _fresh_pools(gc)
                n_probe, _, keys = gc.probe(rid)
                assert n_probe == 128
                if bad:
                    gc.corrupt(int(keys[bad[0]]), bad[1], bad[2], bad[3])
                outs.append((gc.restore(rid, n), gc))
                if bad:   # put the byte back for the next request
                    gc.corrupt(int(keys[bad[0]]), bad[1], bad[2], bad[3])
                bsr.bsr_request_end(gc.ctx, rid)
            mutate = (lambda c, k: c.store.corrupt(k[bad[0]], bad[1], bad[2], bad[3])) if bad else None
            case, res = _oracle(wi, n, 32, mutate)
            if bad:
                assert res.fail_reason == oracle.FAIL_CORRUPT and res.first_failed_chunk == bad[0]
            _same(outs[0], outs[1], case, res, G, success=bad is None)
    finally:
        gs.close()
        go.close()


def test_one_static_context_per_device_and_no_allocation():
    wi = generate(get_config(1))
    say("case: workload 1: a second static context is refused; creation allocates nothing")
    gc = GpuCase(wi, W=2, static=True)
    try:
        with pytest.raises(bsr.BsrError) as e:
            bsr.bsr_ctx_create_static(gc.layout, 2, hip_device=0)
        assert e.value.code == bsr.BSR_E_BUSY
        out = gc.restore(1, gc.probe(1)[0])
        assert out.exposed_tokens == 1024 and out.fallback == 0
    finally:
        gc.close()
    # the array's address is known now: a new context only claims it again
    torch.cuda.synchronize()
    m0, f0 = torch.cuda.memory_allocated(), torch.cuda.mem_get_info()[0]
    ctx = bsr.bsr_ctx_create_static(gc.layout, 2, hip_device=0)
    try:
        torch.cuda.synchronize()
        assert torch.cuda.memory_allocated() == m0
        assert torch.cuda.mem_get_info()[0] == f0
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_scratch_above_the_array_is_refused():
    """One group of 256 tensors of 1,152-byte records in 64-token blocks:
    9,216 install workgroups per chunk, 32-chunk launches need 4.7 MB of
    tag partials, more than the 2 MiB array."""
    w = Workload(index=900, name="wide", n_tokens=256, chunk_tokens=256,
                 groups=(GroupSpec("wide", 64, 256, 1152),), windows=(32,))
    layout = bsr.make_layout(256, [(64, 256, 1152, bsr.BSR_KIND_CONTIG, 0)])
    with pytest.raises(bsr.BsrError) as e:
        bsr.bsr_ctx_create_static(layout, 32, hip_device=0, install_batch=32)
    assert e.value.code == bsr.BSR_E_ARG and "static array" in str(e.value)
    ctx = bsr.bsr_ctx_create_static(layout, 32, hip_device=0, install_batch=8)   # 1.2 MB: fits
    bsr.bsr_ctx_destroy(ctx)
    assert w.n_full_chunks == 1
