"""Parity of the HIP path with the CPU oracle (GPU).

Small cases compare every destination byte, every valid byte, the status
words and the byte counters.  Failure cases compare what the commit rule
fixes: exposure, fallback, every valid byte, every block outside the
advertised prefix, the first failed chunk and the reason (request blocks
themselves are unspecified after a failure: they are never exposed).
"""

import numpy as np
import pytest
import torch

import oracle
from gpu_side import GpuCase, layout_of, say
from oracle_side import build_case
from paper_2608_17826_amd import bsr
from workloads import generate, get_config
from workloads.configs import GroupSpec, Workload
from workloads.gen import random_workload

pytestmark = pytest.mark.gpu

FAIL_NAME = {oracle.FAIL_MISSING: bsr.BSR_FAIL_MISSING, oracle.FAIL_CORRUPT: bsr.BSR_FAIL_CORRUPT,
             oracle.FAIL_TIMEOUT: bsr.BSR_FAIL_TIMEOUT, oracle.FAIL_TRANSFER: bsr.BSR_FAIL_TRANSFER,
             oracle.FAIL_ABORT: bsr.BSR_FAIL_ABORT, oracle.FAIL_NONE: bsr.BSR_FAIL_NONE}


def _oracle(wi, W, mutate=None, **kw):
    case = build_case(wi)
    n, bm, keys = oracle.probe(case.store, wi.tokens, wi.workload.chunk_tokens, wi.salt)
    if mutate:
        mutate(case, keys)
    res = oracle.windowed_restore(case.layout, case.store, keys, n, W, wi.block_tables,
                                  case.pools, case.valid, **kw)
    return case, n, bm, keys, res


def _compare_success(gc, case, res, out, full_pools=True):
    G = len(gc.wi.workload.groups)
    assert out.window_errors == []
    assert out.exposed_tokens == res.exposed_tokens
    assert out.fallback == res.fallback == 0
    st = out.stats
    assert st["h2d_bytes"] == res.h2d_bytes
    assert st["installed_bytes"] == res.installed_bytes
    assert st["peak_live_staging_bytes"] == res.peak_live_staging_bytes
    assert st["n_windows"] == res.n_windows
    assert out.status["fail"] == 0 and out.status["phase"] == 2
    assert out.status["q"][:G] == res.q
    for g in range(G):
        np.testing.assert_array_equal(gc.valid_host(g), case.valid[g])
        if full_pools:
            np.testing.assert_array_equal(gc.pool_host(g), case.pools[g])


def _compare_failure(gc, case, res, out):
    wi = gc.wi
    G = len(wi.workload.groups)
    assert out.exposed_tokens == res.exposed_tokens == 0
    assert out.fallback == res.fallback == 1
    assert out.status["fail"] == FAIL_NAME[res.fail_reason]
    assert out.status["first_failed_chunk"] == res.first_failed_chunk
    assert out.status["q"][:G] == res.q
    n_hit = out.stats["n_hit_chunks"]
    assert out.stats["installed_bytes"] <= n_hit * case.layout.chunk_payload_bytes
    for g, spec in enumerate(wi.workload.groups):
        np.testing.assert_array_equal(gc.valid_host(g), case.valid[g])
        nreq = oracle.request_blocks(n_hit, wi.workload.chunk_tokens, spec.block_tokens)
        others = np.setdiff1d(np.arange(wi.pool_blocks[g]), wi.block_tables[g][:nreq])
        np.testing.assert_array_equal(gc.pool_host(g)[:, others], case.pools[g][:, others])


def test_keys_and_probe_bit_exact():
    wi = generate(get_config(1))
    gc = GpuCase(wi, W=2)
    try:
        case = build_case(wi)
        n, bm, keys = gc.probe(11)
        on, obm, okeys = oracle.probe(case.store, wi.tokens, 64, wi.salt)
        assert n == on == 16
        np.testing.assert_array_equal(bm, obm)
        assert [int(k) for k in keys] == okeys
    finally:
        gc.close()


def test_config1_full_parity():
    say("case: workload 1, W=2, full parity")
    wi = generate(get_config(1))
    case, n, _, _, res = _oracle(wi, 2)
    gc = GpuCase(wi, W=2)
    try:
        assert gc.probe(1)[0] == n == 16
        out = gc.restore(1, n)
        _compare_success(gc, case, res, out)
    finally:
        gc.close()


@pytest.mark.parametrize("seed", range(10))
def test_random_layout_parity(seed):
    w = random_workload(seed)
    wi = generate(w)
    for W in w.windows:
        say(f"case: random layout seed={seed} W={W} groups={[(s.kind, s.block_tokens, s.record_bytes) for s in w.groups]} C={w.chunk_tokens}")
        case, n, _, _, res = _oracle(wi, W)
        gc = GpuCase(wi, W=W)
        try:
            assert gc.probe(5)[0] == n
            out = gc.restore(5, n)
            _compare_success(gc, case, res, out)
        finally:
            gc.close()


@pytest.mark.parametrize("seed", range(10, 110))
def test_random_layout_batch_and_flags_parity(seed):
    """Random layouts with a seeded window, install batch size and block-table
    check (host readback or device check), against the oracle image."""
    w = random_workload(seed)
    wi = generate(w)
    rng = np.random.default_rng(900 + seed)
    W = int(rng.choice(w.windows))
    batch = int(rng.integers(1, min(W, bsr.BSR_MAX_INSTALL_BATCH) + 1))
    flags = bsr.BSR_FLAG_TRUSTED_TABLES if rng.random() < 0.5 else 0
    if rng.random() < 0.5:   # these requests are small: force the two-stream path on half of them
        flags |= bsr.BSR_FLAG_TWO_STREAMS
    say(f"case: random layout seed={seed} W={W} install_batch={batch} flags={flags}")
    case, n, _, _, res = _oracle(wi, W)
    gc = GpuCase(wi, W=W, install_batch=batch, flags=flags)
    try:
        assert gc.probe(41)[0] == n
        out = gc.restore(41, n)
        _compare_success(gc, case, res, out)
        assert out.stats["install_batch"] == batch
        assert out.stats["n_install_launches"] == -(-n // batch) if n else True
    finally:
        gc.close()


@pytest.mark.parametrize("batch", [1, 3, 16, 32])
def test_config2_full_parity(batch):
    say(f"case: workload 2 (32K), W=32, install batch {batch}, full parity")
    wi = generate(get_config(2))
    case, n, _, _, res = _oracle(wi, 32)
    gc = GpuCase(wi, W=32, install_batch=batch)
    try:
        assert gc.probe(2)[0] == n == 128
        out = gc.restore(2, n)
        _compare_success(gc, case, res, out)
        assert out.stats["staging_required_bytes"] == 32 * 9_707_520 == 310_640_640
    finally:
        gc.close()


@pytest.mark.parametrize("workload,W,batch", [(1, 2, 1), (2, 32, 0)])
@pytest.mark.parametrize("slow", ["compute", "copy"])
def test_slot_reuse_gated_by_events_not_timing(workload, W, batch, slow):
    """(Both workloads on two streams: the small one is forced there, since a
    request that small is otherwise staged on the compute stream.)"""
    """Slot reuse is ordered by HIP events, not by how fast either stream
    runs.  Before every window a bounded spin kernel is queued on one of the
    session's streams: on the compute stream the installs lag far behind the
    copies, so a copy into a reused slot must wait for the release of the
    chunk installed from it; on the copy stream the copies lag, so each
    install must wait for its chunks' copies.  Either missing wait would
    install the wrong bytes.  The image must be the oracle's."""
    say(f"case: workload {workload}, W={W}, batch={batch}, slow {slow} stream")
    wi = generate(get_config(workload))
    case, n, _, _, res = _oracle(wi, W)
    gc = GpuCase(wi, W=W, install_batch=batch, flags=bsr.BSR_FLAG_TWO_STREAMS)
    try:
        assert gc.probe(61)[0] == n
        sess = gc.session
        stream = sess.compute_stream if slow == "compute" else sess.copy_stream
        torch.cuda.synchronize()
        sess.bind(61, n, gc.dsts())
        for first, cnt in sess.next_windows(61):
            with torch.cuda.stream(stream):
                torch.cuda._sleep(4_000_000)  # a spin kernel of a fixed cycle count
            bsr.bsr_restore_window(gc.ctx, 61, first, cnt)
        out = sess.commit(61)
        _compare_success(gc, case, res, out)
    finally:
        gc.close()


@pytest.mark.parametrize("mode,k", [("missing", 0), ("missing", 5), ("corrupt", 1), ("corrupt", 15),
                                    ("timeout", 7), ("transfer", 3), ("abort", 2)])
def test_config1_failure_parity(mode, k):
    say(f"case: workload 1 failure {mode} at {k}")
    wi = generate(get_config(1))
    kw = {}
    gkw = {}
    if mode == "missing":
        mut = lambda case, keys: case.store.remove(keys[k], 0)  # noqa: E731
    elif mode == "corrupt":
        mut = lambda case, keys: case.store.corrupt(keys[k], 0, 777, 0x24)  # noqa: E731
    else:
        mut = None
    if mode == "timeout":
        kw["faults"] = {k: oracle.FAIL_TIMEOUT}
    if mode == "transfer":
        kw["faults"] = {k: oracle.FAIL_TRANSFER}
    if mode == "abort":
        kw["abort_after_windows"] = k
    case, n, _, okeys, res = _oracle(wi, 2, mutate=mut, **kw)
    gc = GpuCase(wi, W=2, timeout_ms=50 if mode == "timeout" else 0)
    try:
        n_g, _, keys = gc.probe(3)
        if mode == "missing":
            bsr.bsr_store_remove(gc.ctx, int(keys[k]), 0)
        elif mode == "corrupt":
            gc.corrupt(int(keys[k]), 0, 777, 0x24)
        elif mode == "timeout":
            bsr.bsr_debug_inject(gc.ctx, bsr.BSR_INJECT_DELAY_MS, k, 200)
        elif mode == "transfer":
            bsr.bsr_debug_inject(gc.ctx, bsr.BSR_INJECT_TRANSFER_ERROR, k, 0)
        out = gc.restore(3, n_g, abort_after_windows=kw.get("abort_after_windows"))
        _compare_failure(gc, case, res, out)
        # force-local: the next admission sees no external tokens until RUNNING/teardown
        assert gc.probe(3)[0] == 0
        bsr.bsr_request_running(gc.ctx, 3)
        assert gc.probe(3)[0] == oracle.probe(case.store, wi.tokens, 64, wi.salt)[0]
        bsr.bsr_request_end(gc.ctx, 3)
    finally:
        gc.close()


@pytest.mark.parametrize("seed", range(50))
def test_random_layout_failure_parity(seed):
    """Random layouts x a seeded fault (missing / corrupt entry in a random
    group, timeout, transfer error, abort) at a seeded chunk."""
    w = random_workload(seed)
    wi = generate(w)
    rng = np.random.default_rng(500 + seed)
    W = int(rng.choice(w.windows))
    G = len(w.groups)
    n_full = w.n_full_chunks
    k = int(rng.integers(0, n_full))
    g = int(rng.integers(0, G))
    n_windows = -(-n_full // W)
    mode = ["missing", "corrupt", "timeout", "transfer", "abort"][seed % 5]
    if mode == "abort" and n_windows < 2:
        W = max(1, n_full // 2)                 # at least two windows to abort after the first
        n_windows = -(-n_full // W)
        if n_windows < 2:
            mode = "missing"
    layout = oracle.OracleLayout.from_specs(w.chunk_tokens, w.groups)
    byte = int(rng.integers(0, layout.payload_bytes(g)))
    mask = int(rng.integers(1, 256))
    abort_k = int(rng.integers(1, n_windows)) if mode == "abort" else None
    say(f"case: random layout seed={seed} W={W} fault {mode} chunk {k} group {g}")
    kw = {}
    if mode == "missing":
        mut = lambda case, keys: case.store.remove(keys[k], g)  # noqa: E731
    elif mode == "corrupt":
        mut = lambda case, keys: case.store.corrupt(keys[k], g, byte, mask)  # noqa: E731
    else:
        mut = None
    if mode in ("timeout", "transfer"):
        kw["faults"] = {k: oracle.FAIL_TIMEOUT if mode == "timeout" else oracle.FAIL_TRANSFER}
    if mode == "abort":
        kw["abort_after_windows"] = abort_k
    case, n, _, _, res = _oracle(wi, W, mutate=mut, **kw)
    assert n == n_full
    gc = GpuCase(wi, W=W, timeout_ms=50 if mode == "timeout" else 0)
    try:
        n_g, _, keys = gc.probe(40)
        assert n_g == n
        if mode == "missing":
            bsr.bsr_store_remove(gc.ctx, int(keys[k]), g)
        elif mode == "corrupt":
            gc.corrupt(int(keys[k]), g, byte, mask)
        elif mode == "timeout":
            bsr.bsr_debug_inject(gc.ctx, bsr.BSR_INJECT_DELAY_MS, k, 200)
        elif mode == "transfer":
            bsr.bsr_debug_inject(gc.ctx, bsr.BSR_INJECT_TRANSFER_ERROR, k, 0)
        out = gc.restore(40, n_g, abort_after_windows=abort_k)
        _compare_failure(gc, case, res, out)
        assert gc.probe(40)[0] == 0
    finally:
        gc.close()


def test_failed_install_launch_fails_closed_and_refuses_retries():
    """A launch failure inside a window (forced from the host: the flush of the
    batch holding chunk 40 reports a failed launch and launches nothing) marks
    the request failed: a retried window is refused, and commit invalidates
    before it commits, so nothing is exposed (Prop. 2)."""
    wi = generate(get_config(2))
    layout = oracle.OracleLayout.from_specs(wi.workload.chunk_tokens, wi.workload.groups)
    say("case: workload 2, W=32, install launch failure injected at the batch holding chunk 40")
    gc = GpuCase(wi, W=32)
    try:
        n = gc.probe(50)[0]
        assert n == 128
        bsr.bsr_debug_inject(gc.ctx, bsr.BSR_INJECT_LAUNCH_ERROR, 40, 0)
        torch.cuda.synchronize()
        gc.session.bind(50, n, gc.dsts())
        bsr.bsr_restore_window(gc.ctx, 50, 0, 32)
        with pytest.raises(bsr.BsrError) as e:
            bsr.bsr_restore_window(gc.ctx, 50, 32, 32)
        assert e.value.code == bsr.BSR_E_TRANSFER
        with pytest.raises(bsr.BsrError) as e:
            bsr.bsr_restore_window(gc.ctx, 50, 32, 32)      # the same window again
        assert e.value.code == bsr.BSR_E_STATE
        out = gc.session.commit(50)
        assert out.exposed_tokens == 0 and out.fallback == 1
        assert out.status["fail"] == bsr.BSR_FAIL_TRANSFER
        for g in range(2):
            want = [v.copy() for v in wi.valid_init]
            oracle.set_request_valid(layout, n, wi.block_tables, want, 0)
            np.testing.assert_array_equal(gc.valid_host(g), want[g])
            req = wi.block_tables[g]
            others = np.setdiff1d(np.arange(wi.pool_blocks[g]), req)
            np.testing.assert_array_equal(gc.pool_host(g)[:, others], wi.sentinel_pool(g)[:, others])
        assert gc.probe(50)[0] == 0
    finally:
        gc.close()


def test_group_fault_collapses_all_groups_and_mark_invalid():
    say("case: workload-2 layout, 6 chunks, group B missing at 3; then group marked invalid")
    w0 = get_config(2)
    w = Workload(index=2, name="c2-small", n_tokens=6 * 256, chunk_tokens=256,
                 groups=w0.groups, windows=(2,), base_records=w0.base_records)
    wi = generate(w)
    case, n, _, _, res = _oracle(wi, 2, mutate=lambda c, keys: c.store.remove(keys[3], 1))
    gc = GpuCase(wi, W=2)
    try:
        n_g, _, keys = gc.probe(4)
        bsr.bsr_store_remove(gc.ctx, int(keys[3]), 1)
        out = gc.restore(4, n_g)
        _compare_failure(gc, case, res, out)
        assert out.window_errors == [(2, bsr.BSR_E_MISSING)]
        bsr.bsr_request_end(gc.ctx, 4)
    finally:
        gc.close()
    # engine-reported invalid group, no window failure (Eq. 6's q_g term)
    case, n, _, _, res = _oracle(wi, 2, invalid_groups=[1])
    gc = GpuCase(wi, W=2)
    try:
        n_g = gc.probe(6)[0]
        out = gc.restore(6, n_g, before_commit=lambda: bsr.bsr_mark_group_invalid(gc.ctx, 6, 1))
        assert res.fail_reason == oracle.FAIL_NONE
        _compare_failure(gc, case, res, out)
    finally:
        gc.close()


@pytest.mark.parametrize("after", [1, 2])
def test_group_marked_invalid_between_windows(after):
    """Eq. 6's q_g reported 0 by the engine after window ``after`` of four
    (workload 2, W = 32, default batch of 28, so an install batch is still
    pending when the mark arrives): the later chunks are past the valid prefix
    and install nothing, and their empty tag partials are no corruption.  The
    commit falls back with fail NONE, no failed chunk and q = [1, 0], as the
    oracle's engine-reported invalid group gives."""
    wi = generate(get_config(2))
    say(f"case: workload 2 (32K), W=32, group 1 marked invalid after window {after} of 4")
    case, n, _, _, res = _oracle(wi, 32, invalid_groups=[1])
    assert n == 128 and res.fail_reason == oracle.FAIL_NONE and res.q == [1, 0]
    assert res.first_failed_chunk == 0xFFFFFFFF
    gc = GpuCase(wi, W=32)
    try:
        n_g = gc.probe(8)[0]
        assert n_g == n

        def mark(j):
            if j + 1 == after:
                bsr.bsr_mark_group_invalid(gc.ctx, 8, 1)
        out = gc.restore(8, n_g, after_window=mark)
        assert out.window_errors == []
        _compare_failure(gc, case, res, out)
        assert out.status["first_failed_chunk"] == 0xFFFFFFFF
        assert gc.probe(8)[0] == 0      # the fallback sets the force-local marker
    finally:
        gc.close()


def test_corruption_before_a_mark_stays_the_recorded_failure():
    """A corrupt entry in window 0, then the engine marks group 0 invalid
    after window 1: the corruption was verified before the mark and stays the
    first failure (CORRUPT at its chunk, q = 0 for both groups), as in the
    oracle given the same corrupt entry and invalid group."""
    wi = generate(get_config(2))
    k, g_bad, byte, mask = 5, 1, 777, 0x21
    say(f"case: workload 2 (32K), W=32, group {g_bad} corrupt at chunk {k}, group 0 marked after window 1")
    case, n, _, _, res = _oracle(wi, 32, mutate=lambda c, keys: c.store.corrupt(keys[k], g_bad, byte, mask),
                                 invalid_groups=[0])
    assert res.fail_reason == oracle.FAIL_CORRUPT and res.first_failed_chunk == k and res.q == [0, 0]
    gc = GpuCase(wi, W=32)
    try:
        n_g, _, keys = gc.probe(9)
        gc.corrupt(int(keys[k]), g_bad, byte, mask)
        out = gc.restore(9, n_g, after_window=lambda j: j == 0 and bsr.bsr_mark_group_invalid(gc.ctx, 9, 0))
        _compare_failure(gc, case, res, out)
    finally:
        gc.close()


# the first twelve random layouts with at least two chunks (a window boundary)
_MARK_SEEDS = [s for s in range(40) if random_workload(s).n_full_chunks >= 2][:12]


@pytest.mark.parametrize("seed", _MARK_SEEDS)
def test_random_layout_group_marked_mid_restore(seed):
    """Random layouts: a seeded group is marked invalid after a seeded window
    (never the last), with a seeded install batch."""
    w = random_workload(seed)
    rng = np.random.default_rng(900 + seed)
    n_full = w.n_full_chunks
    W = int(rng.integers(1, n_full))           # at least two windows
    n_windows = -(-n_full // W)
    after = int(rng.integers(1, n_windows))
    g = int(rng.integers(0, len(w.groups)))
    batch = int(rng.integers(1, W + 1))
    wi = generate(w)
    say(f"case: random layout seed={seed} W={W} batch={batch} group {g} marked after window {after} of {n_windows}")
    case, n, _, _, res = _oracle(wi, W, invalid_groups=[g])
    gc = GpuCase(wi, W=W, install_batch=batch)
    try:
        n_g = gc.probe(10)[0]
        assert n_g == n == n_full
        out = gc.restore(10, n_g, after_window=lambda j: j + 1 == after and bsr.bsr_mark_group_invalid(gc.ctx, 10, g))
        assert out.window_errors == []
        _compare_failure(gc, case, res, out)
    finally:
        gc.close()


def _eight_group_workload():
    """BSR_MAX_GROUPS groups mixing planar and contiguous kinds and block sizes
    that divide the chunk, exceed it, or neither; a ragged token tail."""
    from workloads.configs import GroupSpec
    specs = [GroupSpec("c0", 8, 2, 64, value_kind="bytes"),
             GroupSpec("p1", 16, 1, 36, kind="planar", split_bytes=32, value_kind="bytes"),
             GroupSpec("c2", 64, 3, 20, value_kind="bytes"),
             GroupSpec("p3", 24, 2, 132, kind="planar", split_bytes=128, value_kind="bytes"),
             GroupSpec("c4", 32, 1, 1152, value_kind="bytes"),
             GroupSpec("c5", 5, 2, 12, value_kind="bytes"),
             GroupSpec("p6", 48, 1, 24, kind="planar", split_bytes=8, value_kind="bytes"),
             GroupSpec("c7", 128, 2, 512, value_kind="bytes")]
    return Workload(index=300, name="eight-groups", n_tokens=40 * 32 + 7, chunk_tokens=32,
                    groups=tuple(specs), windows=(32,), pool_factor=2)


def test_max_groups_and_max_install_batch():
    wi = generate(_eight_group_workload())
    assert len(wi.workload.groups) == bsr.BSR_MAX_GROUPS
    say("case: eight groups, W=32, install batch 32 (both maxima)")
    case, n, _, _, res = _oracle(wi, 32)
    assert n == 40
    gc = GpuCase(wi, W=32, install_batch=bsr.BSR_MAX_INSTALL_BATCH)
    try:
        assert gc.probe(12)[0] == n
        out = gc.restore(12, n)
        _compare_success(gc, case, res, out)
        assert out.stats["install_batch"] == 32 and out.stats["n_install_launches"] == 2
    finally:
        gc.close()


def _serpentine_workload():
    """Five groups whose 28-chunk install launches exceed 256 MiB, so that the
    groups at odd dispatch positions take a launch's chunks last to first:
    three contiguous groups with equal piece sizes and different block sizes
    (one not dividing the chunk), two planar groups, a ragged token tail."""
    from workloads.configs import GroupSpec
    specs = [GroupSpec("a", 64, 24, 1152, value_kind="bytes"),
             GroupSpec("b", 128, 40, 132, kind="planar", split_bytes=128, value_kind="bytes"),
             GroupSpec("c", 32, 8, 512, value_kind="bytes"),
             GroupSpec("d", 96, 2, 1152, value_kind="bytes"),
             GroupSpec("e", 64, 16, 132, kind="planar", split_bytes=128, value_kind="bytes")]
    return Workload(index=301, name="serpentine-5g", n_tokens=40 * 256 + 100, chunk_tokens=256,
                    groups=tuple(specs), windows=(32,), pool_factor=2, base_records=1 << 14)


def test_serpentine_launches_full_parity():
    """Launches of 28 (the default batch) or 32 chunks take the serpentine
    order, the last, ragged launch (12 or 8 chunks) does not; the whole image
    is the oracle's either way."""
    wi = generate(_serpentine_workload())
    slot = bsr.bsr_slot_bytes(layout_of(wi))
    assert 28 * slot > (256 << 20) and 12 * slot <= (256 << 20)
    case, n, _, _, res = _oracle(wi, 32)
    assert n == 40
    for rid, batch in ((14, 0), (15, 32)):
        say(f"case: five groups, {slot} B chunks, W=32, install batch {batch or 28}, serpentine launches")
        gc = GpuCase(wi, W=32, install_batch=batch)
        try:
            assert gc.probe(rid)[0] == n
            out = gc.restore(rid, n)
            _compare_success(gc, case, res, out)
            assert out.stats["n_install_launches"] == 2
        finally:
            gc.close()


def test_copy_runs_follow_the_arena_layout():
    """Chunks stored back to back are copied in runs; a run breaks wherever
    the arena is not contiguous (shuffled single puts, a replaced chunk)."""
    wi = generate(get_config(2))
    say("case: workload 2, W=32, store half bulk, half shuffled, chunk 10 replaced")
    case, n, _, _, res = _oracle(wi, 32)
    gc = GpuCase(wi, W=32, pinned_chunks=[], arena_chunks=130)
    try:
        keys = [int(k) for k in gc.keys]
        bsr.bsr_store_put_chunks(gc.ctx, keys[:64], [wi.payloads(i) for i in range(64)])
        for i in np.random.default_rng(7).permutation(np.arange(64, 128)):
            bsr.bsr_store_put_chunk(gc.ctx, keys[i], wi.payloads(int(i)))
        bsr.bsr_store_put_chunk(gc.ctx, keys[10], wi.payloads(10))   # moves to another block
        assert gc.probe(21)[0] == n == 128
        out = gc.restore(21, n)
        _compare_success(gc, case, res, out)
    finally:
        gc.close()


@pytest.mark.parametrize("seed", [0, 4, 9])
def test_trusted_tables_parity(seed):
    """BSR_FLAG_TRUSTED_TABLES: no block-table readback at bind; same image."""
    w = random_workload(seed)
    wi = generate(w)
    W = w.windows[1]
    say(f"case: trusted tables, random layout seed={seed} W={W}")
    case, n, _, _, res = _oracle(wi, W)
    gc = GpuCase(wi, W=W, flags=bsr.BSR_FLAG_TRUSTED_TABLES)
    try:
        assert gc.probe(31)[0] == n
        out = gc.restore(31, n)
        _compare_success(gc, case, res, out)
    finally:
        gc.close()


@pytest.mark.parametrize("bad", ["past_pool", "negative"])
def test_trusted_tables_bad_id_fails_closed(bad):
    """An advertised id outside its pool, unchecked at bind, fails the request
    on the device: nothing is written, nothing is exposed (Prop. 2)."""
    wi = generate(get_config(1))
    say(f"case: trusted tables, workload 1, block_table[37] {bad}")
    gc = GpuCase(wi, W=2, flags=bsr.BSR_FLAG_TRUSTED_TABLES)
    try:
        pb = wi.pool_blocks[0]
        gc.dev.block_tables[0][37] = pb if bad == "past_pool" else -5
        torch.cuda.synchronize()
        n = gc.probe(32)[0]
        out = gc.restore(32, n)
        assert out.exposed_tokens == 0 and out.fallback == 1
        assert out.status["fail"] == bsr.BSR_FAIL_BLOCK_TABLE
        assert out.status["first_failed_chunk"] == 37 * 16 // 64
        assert out.status["q"][0] == 0
        # no install ran: every pool byte keeps its sentinel
        np.testing.assert_array_equal(gc.pool_host(0), wi.sentinel_pool(0))
        # every advertised in-range block is invalid, the rest untouched
        want = wi.valid_init[0].copy()
        bt = wi.block_tables[0]
        want[np.delete(bt, 37)] = 0
        np.testing.assert_array_equal(gc.valid_host(0), want)
        assert gc.probe(32)[0] == 0          # force-local after the fallback
    finally:
        gc.close()


@pytest.mark.parametrize("W", [2, 0])
def test_empty_prefix_and_new_salt(W):
    """n = 0: nothing staged, nothing exposed, no fallback; in whole-plan mode
    (W = 0) the ring of an empty plan is one slot."""
    wi = generate(get_config(1))
    gc = GpuCase(wi, W=W)
    try:
        n, bm, _ = gc.probe(8, salt=wi.salt + 2)
        assert n == 0 and not bm.any()
        out = gc.restore(8, 0)
        assert out.exposed_tokens == 0 and out.fallback == 0
        assert out.stats["staging_required_bytes"] == max(W, 1) * 147_456
        assert out.stats["peak_live_staging_bytes"] == 0 and out.stats["h2d_bytes"] == 0
        for g in range(1):
            np.testing.assert_array_equal(gc.valid_host(g), wi.valid_init[g])
            np.testing.assert_array_equal(gc.pool_host(g), wi.sentinel_pool(g))
    finally:
        gc.close()


@pytest.mark.parametrize("W,fault", [(0, None), (2, None), (3, None), (8, None), (3, 4)])
def test_next_window_is_the_oracles_plan(W, fault):
    """bsr_next_window hands out exactly the oracle's windows, each after the
    one before is restored, then (n, 0); after a transfer error at chunk
    `fault` it hands out nothing more, and the outcome is the oracle's."""
    say(f"case: workload 1, W={W}, next-window plan, transfer fault at {fault}")
    wi = generate(get_config(1))
    kw = {"faults": {fault: oracle.FAIL_TRANSFER}} if fault is not None else {}
    case, n, _, _, res = _oracle(wi, W, **kw)
    gc = GpuCase(wi, W=W)
    try:
        assert gc.probe(9)[0] == n
        if fault is not None:
            bsr.bsr_debug_inject(gc.ctx, bsr.BSR_INJECT_TRANSFER_ERROR, fault, 0)
        torch.cuda.synchronize()
        gc.session.bind(9, n, gc.dsts())
        got, errors = [], []
        while True:
            first, cnt = bsr.bsr_next_window(gc.ctx, 9)
            if cnt == 0:
                break
            got.append(range(first, first + cnt))
            try:
                bsr.bsr_restore_window(gc.ctx, 9, first, cnt)
            except bsr.BsrError as e:
                errors.append((first, e.code))
        plan = oracle.plan_windows(n, W)
        if fault is None:
            assert got == plan and first == n and not errors
        else:
            j = fault // W
            assert got == plan[:j + 1] and len(errors) == 1 and errors[0][0] == plan[j].start
        out = gc.session.commit(9, errors)
        if fault is None:
            _compare_success(gc, case, res, out)
        else:
            _compare_failure(gc, case, res, out)
    finally:
        gc.close()


def test_bind_refuses_prefixes_past_the_32_bit_token_range():
    """The install works on 32-bit token positions: bind refuses a prefix
    whose tokens plus two of the largest blocks reach 2^32, and lets the
    largest prefix below that through to its next check (here the missing
    destinations, so nothing is bound)."""
    wi = generate(get_config(1))             # 64-token chunks, 16-token blocks
    gc = GpuCase(wi, W=2)
    try:
        C, B = 64, 16
        limit = (2**32 - 2 * B) // C         # largest n with n*C + 2B < 2^32 (n*C + 2B = 2^32 - 64 + 32)
        assert limit * C + 2 * B < 2**32 <= (limit + 1) * C + 2 * B
        say(f"case: bind bound at n_hit={limit + 1} (refused) and {limit} (passes the bound)")
        with pytest.raises(bsr.BsrError) as e:
            bsr.bsr_request_bind(gc.ctx, 91, limit + 1, [], 0, 0, 0, 0, 0)
        assert e.value.code == bsr.BSR_E_ARG and "2^32" in str(e.value)
        with pytest.raises(bsr.BsrError) as e:
            bsr.bsr_request_bind(gc.ctx, 91, limit, [], 0, 0, 0, 0, 0)
        assert e.value.code == bsr.BSR_E_ARG and "2^32" not in str(e.value) and "NULL" in str(e.value)
        assert bsr.bsr_admission_get(gc.ctx)["n_bound"] == 0
    finally:
        gc.close()


XCD_SPAN_LAYOUT = Workload(
    index=200, name="xcd-span", n_tokens=34 * 16 + 5, chunk_tokens=16,
    groups=(GroupSpec("c36", 16, 36, 512, value_kind="bytes"),), windows=(32,), pool_factor=2)


@pytest.mark.parametrize("batch,grid", [(7, 252), (8, 288), (9, 324), (17, 612)])
def test_xcd_work_order_spans_and_ragged_tail(batch, grid):
    """The install issues its work items in runs across the XCDs for whole
    spans of the grid and in plain order for the ragged rest.  One 8 KiB
    piece per (tensor, chunk) gives 36 work items per chunk, so these batch
    sizes make launches below one span, of exactly one span, and of one or
    two spans plus a ragged tail (a span is 36 x the XCD count, 288 on
    eight XCDs); every image must still equal the oracle's."""
    wi = generate(XCD_SPAN_LAYOUT)
    assert 36 * batch == grid
    say(f"case: XCD spans, install batch {batch} (grid {grid})")
    case, n, _, _, res = _oracle(wi, 32)
    gc = GpuCase(wi, W=32, install_batch=batch)
    try:
        assert gc.probe(61)[0] == n == 34
        out = gc.restore(61, n)
        _compare_success(gc, case, res, out)
        assert out.stats["n_install_launches"] == -(-n // batch)
    finally:
        gc.close()
