"""Full-size parity of the HIP path with the oracle (GPU).

Runs the workloads at their real sizes in the launch configuration bench.py
times (W from the workload, install batch = the library default).  Checks:
  * the probe (every chunk key bit-exact, the prefix length);
  * every valid byte of every group against the oracle's commit rule;
  * every byte of every destination pool: the advertised blocks against the
    oracle's install mapping of the prefix, and every other block against
    its bytes from before the restore, streamed back in slices of about
    1 GiB (``fullimage``); a few sampled blocks also against the oracle's
    separate whole-plan definition of one block (``expected_block``);
  * Eq. 1 measured across the restore: with the ring allocated inside the
    measured region, torch's peak allocated bytes grow by exactly W x chunk
    bytes, the device's free bytes do not change from bind to commit, and the
    library's peak live staging counter equals W x chunk bytes;
  * failures: the oracle walks the same failing restore (into sink pools,
    since request-block contents are unspecified after a failure) and fixes
    exposure, fallback, reason, first failed chunk, q_g and every valid byte;
    every byte of every block outside the prefix is compared unchanged.
"""

import gc as pygc
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from fullimage import compare_full_image, compare_untouched_blocks
from gpu_side import GpuCase, measured_restore, say
from oracle_side import GeneratorStore, SinkPools, build_case, oracle_layout
from paper_2608_17826_amd import bsr
from workloads import generate, get_config
from workloads.configs import Workload

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

FAIL = {oracle.FAIL_MISSING: bsr.BSR_FAIL_MISSING, oracle.FAIL_CORRUPT: bsr.BSR_FAIL_CORRUPT,
        oracle.FAIL_NONE: bsr.BSR_FAIL_NONE}


def _free(gc):
    gc.close()
    gc.dev = None
    gc.session = None
    pygc.collect()
    torch.cuda.empty_cache()


def _expected_valid(wi, layout, n, value):
    valid = [v.copy() for v in wi.valid_init]
    oracle.set_request_valid(layout, n, wi.block_tables, valid, value)
    return valid


def _sample_blocks(gc, wi, keys, n, per_group=40, seed=0, store=None):
    layout = oracle_layout(wi)
    store = store or GeneratorStore(wi, keys)
    rng = np.random.default_rng(seed)
    for g, spec in enumerate(wi.workload.groups):
        nreq = oracle.request_blocks(n, wi.workload.chunk_tokens, spec.block_tokens)
        req = wi.block_tables[g][:nreq]
        others = np.setdiff1d(np.arange(wi.pool_blocks[g]), req)
        picks = list(rng.choice(req, size=min(per_group, len(req)), replace=False))
        picks += list(rng.choice(others, size=min(per_group // 4, len(others)), replace=False))
        for b in picks:
            t = int(rng.integers(0, spec.n_tensors))
            got = gc.dev.pools[g][t][int(b)].cpu().numpy()
            want = oracle.expected_block(layout, store, keys, n, wi.block_tables[g], g, t, int(b),
                                         wi.sentinel_block(g, t, int(b)))
            np.testing.assert_array_equal(got, want, err_msg=f"group {g} tensor {t} block {b}")


def _check_valid(gc, wi, expected):
    for g in range(len(wi.workload.groups)):
        np.testing.assert_array_equal(gc.valid_host(g), expected[g], err_msg=f"valid bytes of group {g}")


def _check_staging_measured(m, W, slot_bytes):
    """Eq. 1 across the restore: the ring is the only device memory it adds."""
    assert m["peak_requested_delta"] == W * slot_bytes, m
    assert 0 <= m["peak_alloc_delta"] - W * slot_bytes <= 1 << 20, m   # torch's block rounding
    assert m["free_after_commit"] == m["free_after_bind"], m


@pytest.mark.parametrize("W", [8, 16, 32, 64])
def test_128k_window_law_and_prefix(W):
    """Workload 3: 75% of chunks held; peak staging = W x chunk bytes exactly,
    measured across the restore; every pool byte equals the oracle's."""
    say(f"case: workload 3 (128K, 384 of 512 held), W={W}")
    wi = generate(get_config(3))
    layout = oracle_layout(wi)
    keys = oracle.chain_keys(wi.tokens, 256, wi.salt)
    gc = GpuCase(wi, W=W)
    try:
        n, bm, gkeys = gc.probe(30 + W)
        assert [int(k) for k in gkeys] == keys
        ostore = GeneratorStore(wi, keys)
        on, obm, _ = oracle.probe(ostore, wi.tokens, 256, wi.salt)
        assert n == on == 384
        np.testing.assert_array_equal(bm, obm)
        assert bsr.bsr_staging_bytes(gc.layout, W) == W * layout.slot_bytes == W * 9_707_520
        out, m = measured_restore(gc, 30 + W, n)
        assert out.exposed_tokens == 384 * 256 == 98_304 and out.fallback == 0
        _check_staging_measured(m, W, layout.slot_bytes)
        st = out.stats
        assert st["peak_live_staging_bytes"] == oracle.peak_live_staging(n, W, layout.slot_bytes) == W * 9_707_520
        assert st["h2d_bytes"] == n * layout.slot_bytes
        assert st["installed_bytes"] == n * layout.chunk_payload_bytes
        assert st["n_windows"] == len(oracle.plan_windows(n, W))
        _check_valid(gc, wi, _expected_valid(wi, layout, n, 1))
        compare_full_image(gc.dev.pools, wi, keys, n, store=ostore, log=say)
        _sample_blocks(gc, wi, keys, n, per_group=8, seed=W, store=ostore)
    finally:
        _free(gc)


@pytest.mark.parametrize("k", [4, 5])
def test_512k_success(k):
    """512K tokens, W = 32, full hit: every pool byte of every group (40 GB of
    pools for workload 4, 67 GB for workload 5) equals the oracle's."""
    say(f"case: workload {k} (512K), W=32, full hit")
    wi = generate(get_config(k))
    layout = oracle_layout(wi)
    keys = oracle.chain_keys(wi.tokens, 256, wi.salt)
    gc = GpuCase(wi, W=32)
    try:
        n, bm, gkeys = gc.probe(40 + k)
        assert [int(x) for x in gkeys] == keys and n == 2048 and bm.all()
        out, m = measured_restore(gc, 40 + k, n)
        assert out.window_errors == [] and out.fallback == 0 and out.exposed_tokens == 524_288
        _check_staging_measured(m, 32, layout.slot_bytes)
        st = out.stats
        assert st["peak_live_staging_bytes"] == 32 * layout.slot_bytes
        assert st["h2d_bytes"] == n * layout.slot_bytes
        assert st["installed_bytes"] == n * layout.chunk_payload_bytes
        _check_valid(gc, wi, _expected_valid(wi, layout, n, 1))
        store = GeneratorStore(wi, keys)
        total = compare_full_image(gc.dev.pools, wi, keys, n, store=store, log=say)
        say(f"  all {total} pool bytes equal the oracle's")
        _sample_blocks(gc, wi, keys, n, per_group=8, seed=k, store=store)
    finally:
        _free(gc)


def test_mtp_layout_64_chunks_full_image():
    """The 4-group layout (MLA @64, planar index keys @128, sliding window
    @32, MTP @64) at 64 chunks, W = 32 with the default 28-chunk install
    batch (launches that span windows): the whole image, every valid byte and
    the counters against the oracle's windowed restore into whole pools."""
    w5 = get_config(5)
    w = Workload(index=5, name="512k-mtp-64-chunks", n_tokens=64 * 256, chunk_tokens=256,
                 groups=w5.groups, windows=(32,), base_records=w5.base_records)
    wi = generate(w)
    say("case: 4-group layout, 64 chunks, W=32, default install batch")
    case = build_case(wi)
    n, _, keys = oracle.probe(case.store, wi.tokens, 256, wi.salt)
    res = oracle.windowed_restore(case.layout, case.store, keys, n, 32, wi.block_tables, case.pools, case.valid)
    assert n == 64 and res.fallback == 0
    gc = GpuCase(wi, W=32)
    try:
        assert gc.probe(45)[0] == n
        out, m = measured_restore(gc, 45, n)
        assert out.stats["install_batch"] == 28 and out.stats["n_install_launches"] == 3
        assert out.exposed_tokens == res.exposed_tokens and out.fallback == 0
        assert out.status["q"][:4] == res.q == [1, 1, 1, 1]
        _check_staging_measured(m, 32, case.layout.slot_bytes)
        st = out.stats
        assert st["peak_live_staging_bytes"] == res.peak_live_staging_bytes == 32 * 16_404_480
        assert st["h2d_bytes"] == res.h2d_bytes and st["installed_bytes"] == res.installed_bytes
        for g in range(4):
            np.testing.assert_array_equal(gc.valid_host(g), case.valid[g], err_msg=f"valid bytes of group {g}")
            np.testing.assert_array_equal(gc.pool_host(g), case.pools[g], err_msg=f"pool of group {g}")
    finally:
        _free(gc)


def _oracle_failure(wi, keys, n, mutate):
    layout = oracle_layout(wi)
    store = GeneratorStore(wi, keys)
    mutate(store)
    valid = [v.copy() for v in wi.valid_init]
    res = oracle.windowed_restore(layout, store, keys, n, 32, wi.block_tables, SinkPools(wi), valid)
    return res, valid


class _CorruptingStore(GeneratorStore):
    """Generator-backed store with one stored byte flipped (tag unchanged)."""

    def __init__(self, wi, keys, chunk, g, byte, mask):
        super().__init__(wi, keys)
        self.bad = (chunk, g, byte, mask)

    def get(self, key, g):
        p, tag = super().get(key, g)
        i = self.index[int(key)]
        if (i, g) == self.bad[:2]:
            p = np.array(p, copy=True)
            p[self.bad[2]] ^= self.bad[3]
        return p, tag


@pytest.mark.parametrize("mode", ["missing", "corrupt"])
def test_512k_group_a_fault_after_probe(mode):
    """Workload 4: a seeded chunk's group-A entry goes missing or corrupt after
    the probe: whole-prefix invalidation in both groups, zero exposure."""
    wi = generate(get_config(4))
    f = wi.failure
    say(f"case: workload 4 (512K), W=32, group A {mode} at chunk {f['chunk']}")
    keys = oracle.chain_keys(wi.tokens, 256, wi.salt)
    layout = oracle_layout(wi)
    if mode == "missing":
        res, valid = _oracle_failure(wi, keys, 2048, lambda s: s.remove(keys[f["chunk"]], f["group"]))
    else:
        store = _CorruptingStore(wi, keys, f["chunk"], f["group"], f["byte"], f["mask"])
        valid = [v.copy() for v in wi.valid_init]
        res = oracle.windowed_restore(layout, store, keys, 2048, 32, wi.block_tables, SinkPools(wi), valid)
    assert res.fallback == 1 and res.first_failed_chunk == f["chunk"]
    gc = GpuCase(wi, W=32)
    try:
        n, _, _ = gc.probe(50)
        assert n == 2048
        if mode == "missing":
            bsr.bsr_store_remove(gc.ctx, int(keys[f["chunk"]]), f["group"])
        else:
            gc.corrupt(int(keys[f["chunk"]]), f["group"], f["byte"], f["mask"])
        out = gc.restore(50, n)
        assert out.exposed_tokens == res.exposed_tokens == 0
        assert out.fallback == 1
        assert out.status["fail"] == FAIL[res.fail_reason]
        assert out.status["first_failed_chunk"] == res.first_failed_chunk
        assert out.status["q"][:2] == res.q == [0, 1]
        if mode == "missing":
            assert out.window_errors == [(f["chunk"] // 32 * 32, bsr.BSR_E_MISSING)]
        _check_valid(gc, wi, valid)
        # every block outside the advertised prefix keeps its bytes
        compare_untouched_blocks(gc.dev.pools, wi, n, log=say)
        assert gc.probe(50)[0] == 0      # force-local until RUNNING admission or teardown
        bsr.bsr_request_end(gc.ctx, 50)
    finally:
        _free(gc)


@pytest.mark.parametrize("which", ["one_window", "seeded"])
def test_512k_mtp_group_missing_beyond_k(which):
    """Workload 5: group G3's entries beyond chunk k are removed after the
    probe (k = W-1, i.e. a fault after one window, and a seeded k)."""
    wi = generate(get_config(5))
    k = 31 if which == "one_window" else wi.failure["seeded_k"]
    g3 = wi.failure["group"]
    say(f"case: workload 5 (512K MTP), W=32, G3 entries beyond chunk {k} removed")
    keys = oracle.chain_keys(wi.tokens, 256, wi.salt)

    def mutate(s):
        for i in range(k + 1, 2048):
            s.remove(keys[i], g3)

    res, valid = _oracle_failure(wi, keys, 2048, mutate)
    assert res.first_failed_chunk == k + 1 and res.fail_reason == oracle.FAIL_MISSING
    gc = GpuCase(wi, W=32)
    try:
        n, _, _ = gc.probe(60)
        assert n == 2048
        for i in range(k + 1, 2048):
            bsr.bsr_store_remove(gc.ctx, int(keys[i]), g3)
        out = gc.restore(60, n)
        assert out.exposed_tokens == 0 and out.fallback == 1
        assert out.status["fail"] == bsr.BSR_FAIL_MISSING
        assert out.status["first_failed_chunk"] == k + 1
        assert out.status["q"][:4] == res.q
        _check_valid(gc, wi, valid)
        compare_untouched_blocks(gc.dev.pools, wi, n, log=say)
        # re-admission: force-local reports zero, then after RUNNING the
        # probe finds exactly the surviving prefix of k+1 chunks
        assert gc.probe(60)[0] == 0
        bsr.bsr_request_running(gc.ctx, 60)
        assert gc.probe(60)[0] == k + 1
        bsr.bsr_request_end(gc.ctx, 60)
    finally:
        _free(gc)


def test_prefix_never_exposed_before_commit():
    """Prop. 2 observed live: a third stream snapshots the status words and the
    advertised valid bytes while windows are in flight; exposure stays 0 and
    every advertised block reads invalid until commit."""
    say("case: workload 2 (32K), W=32, live snapshots from a third stream")
    wi = generate(get_config(2))
    gc = GpuCase(wi, W=32, install_batch=4)
    try:
        n, _, _ = gc.probe(70)
        s = gc.session
        torch.cuda.synchronize()
        s.bind(70, n, gc.dsts())
        s.compute_stream.synchronize()   # the begin kernel has cleared the advertised valid bytes
        watch = torch.cuda.Stream()
        layout = oracle_layout(wi)
        reqs = [wi.block_tables[g][:oracle.request_blocks(n, 256, spec.block_tokens)]
                for g, spec in enumerate(wi.workload.groups)]
        snaps = 0
        for first in range(0, n, 32):
            bsr.bsr_restore_window(gc.ctx, 70, first, min(32, n - first))
            with torch.cuda.stream(watch):
                st = s.status.cpu()
                vals = [v.cpu() for v in gc.dev.valid]
            watch.synchronize()
            raw = bsr.bsr_dev_status.from_buffer_copy(st.numpy().tobytes())
            assert raw.exposed_tokens == 0
            for g in range(len(reqs)):
                assert (vals[g].numpy()[reqs[g]] == 0).all()
            snaps += 1
        exposed, fallback = bsr.bsr_commit(gc.ctx, 70)
        assert exposed == n * 256 and fallback == 0 and snaps == 4
        _check_valid(gc, wi, _expected_valid(wi, layout, n, 1))
    finally:
        _free(gc)
