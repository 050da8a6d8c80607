"""Full-size parity of the HIP path with the oracle (GPU).

Runs the workloads at their real sizes in the launch configuration bench.py
times (W from the workload, install batch = the library default).  Checks:
  * the probe (every chunk key bit-exact, the prefix length);
  * every valid byte of every group against the oracle's commit rule;
  * sampled destination blocks (advertised and not) against the oracle's
    whole-plan definition of a block;
  * a property that holds at any size: in every group, the sum and XOR of
    all 32-bit words over the advertised blocks equal the sum and XOR of the
    oracle's entry tags (a block holds a permutation of its tokens' record
    words, planar or not);
  * the staging law: the ring the library requires is W x chunk bytes, the
    torch allocation delta of that ring equals it, and the library's peak
    live staging counter equals it;
  * failures: the oracle walks the same failing restore (into sink pools,
    since contents are unspecified after a failure) and fixes exposure,
    fallback, reason, first failed chunk, q_g and every valid byte; blocks
    outside the prefix are sampled unchanged.
"""

import gc as pygc
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from gpu_side import GpuCase, say
from oracle_side import GeneratorStore, SinkPools, oracle_layout
from paper_2608_17826_amd import bsr
from workloads import generate, get_config

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


def _word_sum_xor(t: torch.Tensor):
    w = t.reshape(-1).view(torch.int32)
    s = int(w.sum(dtype=torch.int64).item()) & 0xFFFFFFFF
    x = w.clone()
    while x.numel() > 1:
        if x.numel() % 2:
            x = torch.cat([x, torch.zeros(1, dtype=x.dtype, device=x.device)])
        h = x.numel() // 2
        x = torch.bitwise_xor(x[:h], x[h:])
    return s, int(x.item()) & 0xFFFFFFFF


def _check_pool_tags(gc, wi, keys, n):
    """Sum/XOR of all words over the advertised blocks == combination of the
    oracle's entry tags, per group."""
    layout = oracle_layout(wi)
    store = GeneratorStore(wi, keys)

    def tag(i_g):
        return oracle.entry_tag(wi.payload(*i_g))

    for g, spec in enumerate(wi.workload.groups):
        nreq = oracle.request_blocks(n, wi.workload.chunk_tokens, spec.block_tokens)
        assert (n * wi.workload.chunk_tokens) % spec.block_tokens == 0
        with ThreadPoolExecutor(16) as ex:
            tags = list(ex.map(tag, [(i, g) for i in range(n)]))
        es = sum(t & 0xFFFFFFFF for t in tags) & 0xFFFFFFFF
        ex_ = 0
        for t in tags:
            ex_ ^= t >> 32
        idx = gc.dev.block_tables[g][:nreq].long()
        gs, gx = 0, 0
        for p in gc.dev.pools[g]:
            s, x = _word_sum_xor(p.index_select(0, idx))
            gs = (gs + s) & 0xFFFFFFFF
            gx ^= x
        assert (gs, gx) == (es, ex_), f"group {g}: pool words do not match the entry tags"
    return store


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


@pytest.mark.parametrize("W", [8, 16, 32, 64])
def test_128k_window_law_and_prefix(W):
    """Workload 3: 75% of chunks held; peak staging = W x chunk bytes exactly."""
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
        # the ring alone, allocated as the session allocates it
        need = bsr.bsr_staging_bytes(gc.layout, W)
        m0 = torch.cuda.memory_allocated()
        ring = torch.empty(need, dtype=torch.uint8, device="cuda")
        delta = torch.cuda.memory_allocated() - m0
        del ring
        assert need == delta == W * layout.slot_bytes == W * 9_707_520
        out = gc.restore(30 + W, n)
        assert out.exposed_tokens == 384 * 256 == 98_304 and out.fallback == 0
        st = out.stats
        assert st["peak_live_staging_bytes"] == oracle.peak_live_staging(n, W, layout.slot_bytes) == W * 9_707_520
        assert st["h2d_bytes"] == n * layout.slot_bytes
        assert st["installed_bytes"] == n * layout.chunk_payload_bytes
        assert st["n_windows"] == len(oracle.plan_windows(n, W))
        _check_valid(gc, wi, _expected_valid(wi, layout, n, 1))
        _sample_blocks(gc, wi, keys, n, per_group=24, seed=W, store=ostore)
        if W == 32:
            _check_pool_tags(gc, wi, keys, n)
    finally:
        _free(gc)


@pytest.mark.parametrize("k", [4, 5])
def test_512k_success(k):
    say(f"case: workload {k} (512K), W=32, full hit")
    wi = generate(get_config(k))
    layout = oracle_layout(wi)
    keys = oracle.chain_keys(wi.tokens, 256, wi.salt)
    gc = GpuCase(wi, W=32)
    try:
        n, bm, gkeys = gc.probe(40 + k)
        assert [int(x) for x in gkeys] == keys and n == 2048 and bm.all()
        out = gc.restore(40 + k, n)
        assert out.window_errors == [] and out.fallback == 0 and out.exposed_tokens == 524_288
        st = out.stats
        assert st["peak_live_staging_bytes"] == 32 * layout.slot_bytes
        assert st["h2d_bytes"] == n * layout.slot_bytes
        assert st["installed_bytes"] == n * layout.chunk_payload_bytes
        _check_valid(gc, wi, _expected_valid(wi, layout, n, 1))
        store = _check_pool_tags(gc, wi, keys, n)
        _sample_blocks(gc, wi, keys, n, per_group=32, seed=k, store=store)
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
        # blocks outside the advertised prefix keep their sentinels
        rng = np.random.default_rng(7)
        for g, spec in enumerate(wi.workload.groups):
            others = np.setdiff1d(np.arange(wi.pool_blocks[g]), wi.block_tables[g])
            for b in rng.choice(others, size=12, replace=False):
                t = int(rng.integers(0, spec.n_tensors))
                np.testing.assert_array_equal(gc.dev.pools[g][t][int(b)].cpu().numpy(),
                                              wi.sentinel_block(g, t, int(b)))
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
