"""Global admission budget B (§7 "Current concurrency is conservative") on the GPU.

Several requests are bound to one context at once, each with its own staging
ring, status block, streams and destination pools, and their windows are
interleaved.  What must hold:
  * admission follows the oracle's replay of the same bind/end events
    (``oracle.admission``): the lock when B = 0, else the summed rings of the
    bound requests never exceed B;
  * each request's destination image, valid bytes, exposure and counters
    equal the oracle's restore of that request alone (§2: BSR changes
    residency, not what is restored), whatever else is bound beside it;
  * a failure in one bound request leaves the others untouched (Prop. 2 per
    request).
"""

import ctypes
import dataclasses
import random
import threading
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from gpu_side import layout_of, say
from oracle_side import build_case
from paper_2608_17826_amd import bsr
from paper_2608_17826_amd.session import RestoreSession, group_dsts
from workloads import generate, get_config
from workloads.device import place

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(600)]

adm = oracle.admission


def _variant(k, index, n_tokens=None):
    w = get_config(k)
    kw = {"index": index}
    if n_tokens:
        kw["n_tokens"] = n_tokens
    return generate(dataclasses.replace(w, **kw))


class Tenant:
    """One request: its inputs, its oracle case, its device pools and session."""

    def __init__(self, ctx, wi, rid, W, mutate=None, n_hit=None, **okw):
        self.wi, self.rid, self.ctx = wi, rid, ctx
        w = wi.workload
        self.case = build_case(wi)
        n, _, keys = oracle.probe(self.case.store, wi.tokens, w.chunk_tokens, wi.salt)
        self.keys = keys
        if mutate:
            mutate(self.case, keys)
        self.n = n if n_hit is None else n_hit
        self.res = oracle.windowed_restore(self.case.layout, self.case.store, keys, self.n, W,
                                           wi.block_tables, self.case.pools, self.case.valid, **okw)
        self.dev = place(wi)
        self.sess = RestoreSession(ctx)
        self.errors = []
        self.out = None

    def probe(self):
        return bsr.bsr_probe(self.ctx, self.rid, self.wi.salt, self.wi.tokens)[0]

    def dsts(self):
        d = self.dev
        return group_dsts(d.block_tables, d.tensor_bases, d.valid, self.wi.pool_blocks)

    def bind(self):
        torch.cuda.synchronize()
        self.sess.bind(self.rid, self.n, self.dsts())

    def step(self):
        """Restore the next window; False when none is left or the request failed."""
        if self.errors:
            return False
        first, n = bsr.bsr_next_window(self.ctx, self.rid)
        if n == 0:
            return False
        try:
            bsr.bsr_restore_window(self.ctx, self.rid, first, n)
        except bsr.BsrError as e:
            self.errors.append((first, e.code))
        return True

    def commit(self):
        self.out = self.sess.commit(self.rid, self.errors)
        return self.out

    def pool_host(self, g):
        return np.stack([p.cpu().numpy() for p in self.dev.pools[g]])

    def check_success(self):
        out, res = self.out, self.res
        assert out.window_errors == []
        assert out.exposed_tokens == res.exposed_tokens > 0 and out.fallback == 0
        st = out.stats
        assert st["request_id"] == self.rid
        assert st["h2d_bytes"] == res.h2d_bytes
        assert st["installed_bytes"] == res.installed_bytes
        assert st["peak_live_staging_bytes"] == res.peak_live_staging_bytes
        assert out.status["phase"] == 2 and out.status["fail"] == 0
        for g in range(len(self.wi.workload.groups)):
            np.testing.assert_array_equal(self.dev.valid[g].cpu().numpy(), self.case.valid[g])
            np.testing.assert_array_equal(self.pool_host(g), self.case.pools[g])

    def check_failure(self, fail_code):
        out, res = self.out, self.res
        assert out.exposed_tokens == res.exposed_tokens == 0
        assert out.fallback == res.fallback == 1
        assert out.status["fail"] == fail_code
        assert out.status["first_failed_chunk"] == res.first_failed_chunk
        w = self.wi.workload
        for g, spec in enumerate(w.groups):
            np.testing.assert_array_equal(self.dev.valid[g].cpu().numpy(), self.case.valid[g])
            nreq = oracle.request_blocks(self.n, w.chunk_tokens, spec.block_tokens)
            others = np.setdiff1d(np.arange(self.wi.pool_blocks[g]), self.wi.block_tables[g][:nreq])
            np.testing.assert_array_equal(self.pool_host(g)[:, others], self.case.pools[g][:, others])


def _ctx(wis, W, budget, max_bound=0):
    layout = layout_of(wis[0])
    ctx = bsr.bsr_ctx_create(layout, W, hip_device=0, staging_budget_bytes=budget,
                             max_bound_requests=max_bound)
    slot = bsr.bsr_slot_bytes(layout)
    stride = (slot + 4095) // 4096 * 4096
    bsr.bsr_store_reserve(ctx, stride * (sum(wi.workload.held_chunks for wi in wis) + 2))
    for wi in wis:
        keys = bsr.bsr_chunk_keys(wi.salt, wi.tokens, wi.workload.chunk_tokens)
        held = wi.workload.held_chunks
        bsr.bsr_store_put_chunks(ctx, keys[:held], [wi.payloads(i) for i in range(held)])
    return ctx, slot


def _bind(t, log):
    """Bind and record the admission outcome in the oracle's vocabulary."""
    try:
        t.bind()
        log.append(adm.OK)
        return True
    except bsr.BsrError as e:
        if e.code not in (bsr.BSR_E_BUSY, bsr.BSR_E_STAGING):
            raise
        log.append(adm.BUSY if e.code == bsr.BSR_E_BUSY else adm.TOO_LARGE)
        return False


def _interleave(tenants):
    while any([t.step() for t in tenants]):
        pass


def test_two_bound_interleaved_third_waits_for_budget():
    W = 8
    wis = [_variant(2, 2 + 100 * j, n_tokens=8192) for j in range(3)]
    ctx, slot = _ctx(wis, W, budget=2 * W * 9_707_520 + W * 9_707_520 // 2)
    try:
        ring = W * slot
        B = 2 * ring + ring // 2
        ts = [Tenant(ctx, wi, 10 + j, W) for j, wi in enumerate(wis)]
        a, b, c = ts
        for t in ts:
            assert t.probe() == t.n == 32
        say("case: config-2 layout 8K x3, W=8, B=2.5 rings: bind a, b; c waits")
        log = []
        assert _bind(a, log) and _bind(b, log)
        assert not _bind(c, log)
        st = bsr.bsr_admission_get(ctx)
        assert st["n_bound"] == 2 and st["bound_staging_bytes"] == 2 * ring
        assert st["max_bound_requests"] == 2   # automatic: B / ring
        _interleave([a, b])
        a.commit()
        assert _bind(c, log)
        _interleave([b, c])
        b.commit()
        c.commit()
        # runs staged while another request was bound went to the copy engine
        assert a.out.stats["n_stage_launches"] == b.out.stats["n_stage_launches"] == 0
        events = [("bind", 10, 32), ("bind", 11, 32), ("bind", 12, 32), ("end", 10), ("bind", 12, 32),
                  ("end", 11), ("end", 12)]
        want = adm.replay(B, st["max_bound_requests"], W, slot, events)
        assert log == want.outcomes
        st = bsr.bsr_admission_get(ctx)
        assert st["peak_bound_staging_bytes"] == want.peak_bound_bytes == 2 * ring <= B
        assert st["peak_n_bound"] == want.peak_bound == 2
        assert st["n_refused"] == want.refused_busy == 1
        assert st["n_bound"] == 0 and st["bound_staging_bytes"] == 0
        for t in ts:
            t.check_success()
            assert bsr.bsr_request_stats(ctx, t.rid)["exposed_tokens"] == 8192
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_failure_in_one_request_leaves_the_others_intact():
    W = 8
    wis = [_variant(2, 2 + 100 * j, n_tokens=8192) for j in range(3)]
    ctx, slot = _ctx(wis, W, budget=3 * W * 9_707_520)
    try:
        corrupt = lambda case, keys: case.store.corrupt(keys[5], 1, 1001, 0x5A)   # noqa: E731
        missing = lambda case, keys: case.store.remove(keys[12], 0)               # noqa: E731
        good = Tenant(ctx, wis[0], 20, W)
        bad = Tenant(ctx, wis[1], 21, W, mutate=corrupt)
        gone = Tenant(ctx, wis[2], 22, W, mutate=missing)
        for t in (good, bad, gone):
            assert t.probe() == 32
        # the same faults, made after the probe on the library's tiers
        addr, nbytes, _ = bsr.bsr_store_payload(ctx, int(bad.keys[5]), 1)
        assert 1001 < nbytes
        ctypes.c_uint8.from_address(addr + 1001).value ^= 0x5A
        bsr.bsr_store_remove(ctx, int(gone.keys[12]), 0)
        say("case: three bound, one corrupt entry (device-detected), one missing (host-detected)")
        log = []
        assert all(_bind(t, log) for t in (good, bad, gone))
        _interleave([good, bad, gone])
        assert gone.errors == [(8, bsr.BSR_E_MISSING)]
        for t in (bad, gone, good):
            t.commit()
        good.check_success()
        bad.check_failure(bsr.BSR_FAIL_CORRUPT)
        gone.check_failure(bsr.BSR_FAIL_MISSING)
        # force-local only for the failed requests
        assert bad.probe() == 0 and gone.probe() == 0
        bsr.bsr_request_end(ctx, good.rid)
        assert good.probe() == 32
        assert bsr.bsr_admission_get(ctx)["peak_n_bound"] == 3
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_staging_path_changes_mid_request():
    """A request staged by the staging kernel while bound alone switches to
    the copy engine when a second one binds, and back once the second one
    has committed; both images are the oracle's."""
    W = 8
    wis = [_variant(2, 2 + 100 * j, n_tokens=8192) for j in range(2)]
    ctx, slot = _ctx(wis, W, budget=2 * W * 9_707_520)
    try:
        x = Tenant(ctx, wis[0], 70, W)
        y = Tenant(ctx, wis[1], 71, W)
        assert x.probe() == y.probe() == 32
        say("case: config-2 layout 8K x2, W=8: x alone, then with y, then alone again")
        log = []
        assert _bind(x, log)
        assert x.step() and x.step()          # windows 0-1 of x alone: staging kernel
        assert _bind(y, log)
        assert x.step() and y.step()          # x's window 2 beside y: copy engine
        while y.step():
            pass
        y.commit()
        while x.step():                       # x's window 3 alone again
            pass
        x.commit()
        x.check_success()
        y.check_success()
        runs_x, runs_y = x.out.stats["n_stage_launches"], y.out.stats["n_stage_launches"]
        assert runs_x > 0 and runs_y == 0
        assert 0 < x.out.stats["stage_bytes"] < x.out.stats["h2d_bytes"]
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_budget_zero_keeps_the_lock_and_slot_count_limits():
    W = 2
    wis = [_variant(1, 1 + 100 * j) for j in range(3)]
    ctx, slot = _ctx(wis, W, budget=0)
    try:
        ts = [Tenant(ctx, wi, 30 + j, W) for j, wi in enumerate(wis)]
        for t in ts:
            assert t.probe() == 16
        say("case: B=0 lock, workload 1 x3")
        log = []
        assert _bind(ts[0], log)
        assert not _bind(ts[1], log)
        _interleave([ts[0]])
        bsr.bsr_request_end(ctx, ts[0].rid)     # teardown releases the lock without exposing
        assert ts[0].dev.valid[0].cpu().numpy()[ts[0].wi.block_tables[0]].sum() == 0
        assert _bind(ts[1], log)
        _interleave([ts[1]])
        ts[1].commit()
        ts[1].check_success()
        want = adm.replay(0, 1, W, slot, [("bind", 30, 16), ("bind", 31, 16), ("end", 30), ("bind", 31, 16)])
        assert log == want.outcomes
        a = bsr.bsr_admission_get(ctx)
        assert a["max_bound_requests"] == 1 and a["peak_n_bound"] == 1 and a["n_refused"] == 1
    finally:
        bsr.bsr_ctx_destroy(ctx)
    # a budget for ten rings but two session slots: the slots bind first
    ctx, slot = _ctx(wis, W, budget=10 * W * 147_456, max_bound=2)
    try:
        ts = [Tenant(ctx, wi, 40 + j, W) for j, wi in enumerate(wis)]
        for t in ts:
            t.probe()
        log = []
        assert _bind(ts[0], log) and _bind(ts[1], log) and not _bind(ts[2], log)
        want = adm.replay(10 * W * slot, 2, W, slot, [("bind", r, 16) for r in (40, 41, 42)])
        assert log == want.outcomes
        _interleave(ts[:2])
        for t in ts[:2]:
            t.commit()
            t.check_success()
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_whole_plan_rings_count_against_the_budget():
    """W = 0: a request's ring is its whole plan (Eq. 2), so B admits by plan length."""
    wis = [_variant(2, 2 + 100 * j, n_tokens=8192) for j in range(3)]
    c5 = 9_707_520
    ctx, slot = _ctx(wis, 0, budget=30 * c5)
    try:
        assert slot == c5
        say("case: whole-plan W=0, B=30 slots, plans 32 (too large), 24, 6, 1")
        big = Tenant(ctx, wis[0], 50, 0, n_hit=32)
        a = Tenant(ctx, wis[0], 51, 0, n_hit=24)
        b = Tenant(ctx, wis[1], 52, 0, n_hit=6)
        c = Tenant(ctx, wis[2], 53, 0, n_hit=1)
        for t in (big, a, b, c):
            assert t.probe() == 32
        log = []
        assert not _bind(big, log)
        assert _bind(a, log) and _bind(b, log)
        assert not _bind(c, log)
        assert bsr.bsr_admission_get(ctx)["bound_staging_bytes"] == 30 * c5
        _interleave([a, b])
        a.commit()
        b.commit()
        a.check_success()
        b.check_success()
        assert a.out.stats["peak_live_staging_bytes"] == 24 * c5
        want = adm.replay(30 * c5, bsr.bsr_admission_get(ctx)["max_bound_requests"], 0, c5,
                          [("bind", 50, 32), ("bind", 51, 24), ("bind", 52, 6), ("bind", 53, 1)])
        assert log == want.outcomes == [adm.TOO_LARGE, adm.OK, adm.OK, adm.BUSY]
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_requests_driven_from_threads():
    """Four requests bound together, each driven start to finish by its own thread."""
    W = 4
    wis = [_variant(2, 2 + 100 * j, n_tokens=4096) for j in range(4)]
    ctx, slot = _ctx(wis, W, budget=4 * W * 9_707_520)
    try:
        ts = [Tenant(ctx, wi, 60 + j, W) for j, wi in enumerate(wis)]
        for t in ts:
            assert t.probe() == 16
        torch.cuda.synchronize()
        barrier = threading.Barrier(len(ts))
        say("case: 4 threads, W=4, B=4 rings")

        def run(t):
            t.sess.bind(t.rid, t.n, t.dsts())
            barrier.wait(timeout=60)          # all four are bound at once
            while t.step():
                pass
            return t.commit()

        with ThreadPoolExecutor(len(ts)) as ex:
            list(ex.map(run, ts))
        for t in ts:
            t.check_success()
        a = bsr.bsr_admission_get(ctx)
        assert a["peak_n_bound"] == 4 and a["peak_bound_staging_bytes"] == 4 * W * slot
    finally:
        bsr.bsr_ctx_destroy(ctx)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_random_event_sequences_follow_the_oracle(seed):
    rng = random.Random(seed)
    W = 2
    wis = [_variant(1, 1 + 100 * j) for j in range(4)]
    B = 2 * W * 147_456 + 147_456          # two rings and a slot
    ctx, slot = _ctx(wis, W, budget=B)
    try:
        ts = {40 + j: Tenant(ctx, wi, 40 + j, W) for j, wi in enumerate(wis)}
        for t in ts.values():
            t.probe()
        say(f"case: random bind/end sequence seed={seed}, B = 2 rings + 1 slot")
        events, log, bound, done = [], [], set(), set()
        for _ in range(14):
            rid = rng.choice(sorted(ts))
            if rid in done:
                continue
            t = ts[rid]
            if rid in bound:
                if rng.random() < 0.5:
                    t.step()
                    continue
                while t.step():
                    pass
                t.commit()
                events.append(("end", rid))
                bound.discard(rid)
                done.add(rid)
            else:
                events.append(("bind", rid, t.n))
                if _bind(t, log):
                    bound.add(rid)
        for rid in sorted(bound):
            t = ts[rid]
            while t.step():
                pass
            t.commit()
            events.append(("end", rid))
            done.add(rid)
        want = adm.replay(B, bsr.bsr_admission_get(ctx)["max_bound_requests"], W, slot, events)
        assert log == want.outcomes
        assert bsr.bsr_admission_get(ctx)["peak_bound_staging_bytes"] == want.peak_bound_bytes <= B
        for rid in done:
            ts[rid].check_success()
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_file_tier_requests_share_the_bounce_pool(tmp_path):
    """Two requests served by the file tier, bound together: their windows
    alternate over one pool of two pinned bounce buffers."""
    W = 4
    wis = [_variant(2, 2 + 100 * j, n_tokens=4096) for j in range(2)]
    layout = layout_of(wis[0])
    ctx = bsr.bsr_ctx_create(layout, W, hip_device=0, staging_budget_bytes=2 * W * 9_707_520)
    try:
        slot = bsr.bsr_slot_bytes(layout)
        bsr.bsr_store_reserve(ctx, (slot + 4095) // 4096 * 4096)   # the pinned tier stays empty
        bsr.bsr_file_tier_open(ctx, str(tmp_path), 2, 2, 0)
        for wi in wis:
            keys = bsr.bsr_chunk_keys(wi.salt, wi.tokens, wi.workload.chunk_tokens)
            with ThreadPoolExecutor(8) as ex:
                list(ex.map(lambda i: bsr.bsr_file_tier_put_chunk(ctx, int(keys[i]), wi.payloads(i)),
                            range(wi.workload.held_chunks)))
        ts = [Tenant(ctx, wi, 70 + j, W) for j, wi in enumerate(wis)]
        for t in ts:
            assert t.probe() == 16
            assert set(bsr.bsr_plan_tiers(ctx, t.rid, 16).tolist()) == {bsr.BSR_TIER_FILE}
        say("case: file tier only, 2 requests bound together, 2 bounce buffers shared")
        log = []
        assert all(_bind(t, log) for t in ts)
        _interleave(ts)
        for t in ts:
            t.commit()
            t.check_success()
            assert t.out.stats["file_tier_chunks"] == 16
    finally:
        bsr.bsr_ctx_destroy(ctx)
