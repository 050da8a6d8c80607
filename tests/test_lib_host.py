"""Host-side checks of libbsr.so without a GPU (CPU).

The library loads, exports every function include/bsr.h declares, and its
host logic -- chunk keys, probe, slot geometry, store tags, argument and
state errors -- matches the oracle bit for bit on a host-only context
(hip_device = -1, caller-adopted arena).  No compute call is made.
"""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle
from oracle_side import build_case, oracle_layout
from paper_2608_17826_amd import bsr
from workloads import generate, get_config
from workloads.gen import random_workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
KIND = {"contig": bsr.BSR_KIND_CONTIG, "planar": bsr.BSR_KIND_PLANAR}


def _declared():
    src = open(os.path.join(ROOT, "include", "bsr.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(bsr_[a-z0-9_]+)\s*\(", src)))


def test_exports_every_declared_symbol():
    names = _declared()
    assert len(names) >= 25
    lib = ctypes.CDLL(bsr.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    nm = subprocess.run(["nm", "-D", "--defined-only", bsr.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (bsr_[a-z0-9_]+)", nm))
    assert set(names) <= exported
    assert bsr.bsr_abi_version() == bsr.BSR_ABI_VERSION == 4


def _layout(w):
    return bsr.make_layout(w.chunk_tokens, [(s.block_tokens, s.n_tensors, s.record_bytes, KIND[s.kind],
                                             s.split_bytes) for s in w.groups])


@pytest.mark.parametrize("k", [1, 2, 5])
def test_slot_bytes_match_oracle(k):
    w = get_config(k)
    ol = oracle.OracleLayout.from_specs(w.chunk_tokens, w.groups)
    assert bsr.bsr_slot_bytes(_layout(w)) == ol.slot_bytes
    assert bsr.bsr_staging_bytes(_layout(w), 32) == 32 * ol.slot_bytes
    # §8-layout numbers: 147,456 / 9,707,520 / 16,404,480
    assert ol.slot_bytes == {1: 147_456, 2: 9_707_520, 5: 16_404_480}[k]


@pytest.mark.parametrize("seed", range(30))
def test_slot_bytes_random_layouts(seed):
    w = random_workload(seed)
    ol = oracle.OracleLayout.from_specs(w.chunk_tokens, w.groups)
    assert bsr.bsr_slot_bytes(_layout(w)) == ol.slot_bytes


@pytest.mark.parametrize("C,n,salt", [(64, 1024, 1), (256, 32768 + 100, 2**64 - 1), (16, 5, 7), (7, 701, 0)])
def test_chunk_keys_bit_exact(C, n, salt):
    toks = np.random.default_rng(C + n).integers(-2**31, 2**31, n, dtype=np.int64).astype(np.int32)
    assert [int(x) for x in bsr.bsr_chunk_keys(salt, toks, C)] == oracle.chain_keys(toks, C, salt)


def _host_ctx(w, W=2):
    ctx = bsr.bsr_ctx_create(_layout(w), W, hip_device=-1)
    slot = bsr.bsr_slot_bytes(ctx.layout)
    stride = (slot + 4095) // 4096 * 4096
    arena = np.zeros(stride * (w.held_chunks + 2), np.uint8)
    bsr.bsr_store_adopt(ctx, arena.ctypes.data, arena.nbytes)
    return ctx, arena


def test_probe_and_tags_match_oracle():
    wi = generate(get_config(1))
    w = wi.workload
    ctx, arena = _host_ctx(w)
    try:
        case = build_case(wi)
        for i in range(w.held_chunks):
            bsr.bsr_store_put_chunk(ctx, case.keys[i], wi.payloads(i))
        n, bm, keys = bsr.bsr_probe(ctx, 1, wi.salt, wi.tokens)
        on, obm, okeys = oracle.probe(case.store, wi.tokens, w.chunk_tokens, wi.salt)
        assert n == on and [int(k) for k in keys] == okeys
        np.testing.assert_array_equal(bm, obm)
        for i in (0, 7, 15):
            addr, nbytes, tag = bsr.bsr_store_payload(ctx, case.keys[i], 0)
            assert tag == case.store.get(case.keys[i], 0)[1]
            got = np.ctypeslib.as_array((ctypes.c_uint8 * nbytes).from_address(addr))
            np.testing.assert_array_equal(got, wi.payload(i, 0))
        # hole at chunk 9: prefix 9, bitmap still shows later hits
        bsr.bsr_store_remove(ctx, case.keys[9], 0)
        case.store.remove(case.keys[9], 0)
        n, bm, _ = bsr.bsr_probe(ctx, 2, wi.salt, wi.tokens)
        on, obm, _ = oracle.probe(case.store, wi.tokens, w.chunk_tokens, wi.salt)
        assert n == on == 9
        np.testing.assert_array_equal(bm, obm)
        # a new salt finds nothing
        assert bsr.bsr_probe(ctx, 3, wi.salt ^ 0x10, wi.tokens)[0] == 0
        assert bsr.bsr_store_count(ctx)[0] == w.held_chunks - 1
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_multi_group_tags_and_partial_removal():
    w = random_workload(4)
    wi = generate(w)
    ctx, arena = _host_ctx(w)
    try:
        case = build_case(wi)
        for i in range(w.held_chunks):
            bsr.bsr_store_put_chunk(ctx, case.keys[i], wi.payloads(i))
        for i in range(w.held_chunks):
            for g in range(len(w.groups)):
                assert bsr.bsr_store_payload(ctx, case.keys[i], g)[2] == case.store.get(case.keys[i], g)[1]
        G = len(w.groups)
        bsr.bsr_store_remove(ctx, case.keys[1], G - 1)
        case.store.remove(case.keys[1], G - 1)
        assert bsr.bsr_probe(ctx, 1, wi.salt, wi.tokens)[0] == oracle.probe(
            case.store, wi.tokens, w.chunk_tokens, wi.salt)[0] == 1
        with pytest.raises(bsr.BsrError) as e:
            bsr.bsr_store_remove(ctx, case.keys[1], G - 1)
        assert e.value.code == bsr.BSR_E_NOTFOUND
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_store_replace_and_full_arena():
    w = get_config(1)
    wi = generate(w)
    ctx = bsr.bsr_ctx_create(_layout(w), 2, hip_device=-1)
    arena = np.zeros(2 * 147_456, np.uint8)
    try:
        bsr.bsr_store_adopt(ctx, arena.ctypes.data, arena.nbytes)
        bsr.bsr_store_put_chunk(ctx, 5, wi.payloads(0))
        bsr.bsr_store_put_chunk(ctx, 6, wi.payloads(1))
        with pytest.raises(bsr.BsrError) as e:
            bsr.bsr_store_put_chunk(ctx, 7, wi.payloads(2))
        assert e.value.code == bsr.BSR_E_NOMEM
        bsr.bsr_store_remove(ctx, 6)
        bsr.bsr_store_put_chunk(ctx, 5, wi.payloads(2))   # replace: old block freed
        bsr.bsr_store_put_chunk(ctx, 7, wi.payloads(3))
        assert bsr.bsr_store_payload(ctx, 5, 0)[2] == oracle.entry_tag(wi.payload(2, 0))
        assert bsr.bsr_store_count(ctx) == (2, 2 * 147_456)
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_argument_and_state_errors():
    w = get_config(2)
    L = _layout(w)
    bad = bsr.make_layout(256, [(64, 32, 1150, 0, 0)])          # record not a multiple of 4
    with pytest.raises(bsr.BsrError):
        bsr.bsr_slot_bytes(bad)
    with pytest.raises(bsr.BsrError):
        bsr.bsr_slot_bytes(bsr.make_layout(256, [(128, 8, 132, 1, 132)]))   # split == record
    with pytest.raises(bsr.BsrError):
        bsr.bsr_staging_bytes(L, 0)
    with pytest.raises(bsr.BsrError):
        bsr.bsr_ctx_create(L, 4, hip_device=-1, install_batch=5)
    with pytest.raises(bsr.BsrError) as e:
        bsr.bsr_ctx_create(L, 0, hip_device=-1, install_batch=bsr.BSR_MAX_INSTALL_BATCH + 1)
    assert e.value.code == bsr.BSR_E_ARG
    # W = 0 is the whole-plan mode: the ring holds the whole plan (Eq. 2)
    whole = bsr.bsr_ctx_create(L, 0, hip_device=-1)
    try:
        assert bsr.bsr_plan_staging_bytes(whole, 2048) == 2048 * 9_707_520
        assert bsr.bsr_plan_staging_bytes(whole, 7) == 7 * 9_707_520
    finally:
        bsr.bsr_ctx_destroy(whole)
    bounded = bsr.bsr_ctx_create(L, 32, hip_device=-1)
    try:
        assert bsr.bsr_plan_staging_bytes(bounded, 2048) == bsr.bsr_plan_staging_bytes(bounded, 3) == 32 * 9_707_520
    finally:
        bsr.bsr_ctx_destroy(bounded)
    ctx = bsr.bsr_ctx_create(L, 4, hip_device=-1)
    try:
        with pytest.raises(bsr.BsrError) as e:
            bsr.bsr_store_reserve(ctx, 1 << 20)
        assert e.value.code == bsr.BSR_E_DEVICE
        with pytest.raises(bsr.BsrError) as e:
            bsr.bsr_restore_window(ctx, 1, 0, 1)
        assert e.value.code == bsr.BSR_E_DEVICE
        with pytest.raises(bsr.BsrError) as e:
            bsr.bsr_store_put_chunk(ctx, 1, [np.zeros(9437184, np.uint8), np.zeros(270336, np.uint8)])
        assert e.value.code == bsr.BSR_E_STATE
        assert "arena" in bsr.bsr_last_error()
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_admission_config_errors_and_defaults():
    """Global admission budget B (§7): argument checks and the automatic slot count."""
    w = get_config(2)
    L = _layout(w)
    c = 9_707_520
    with pytest.raises(bsr.BsrError) as e:
        bsr.bsr_ctx_create(L, 4, hip_device=-1, max_bound_requests=2)         # lock: one slot
    assert e.value.code == bsr.BSR_E_ARG
    with pytest.raises(bsr.BsrError) as e:
        bsr.bsr_ctx_create(L, 4, hip_device=-1, staging_budget_bytes=4 * c - 1)  # holds no ring
    assert e.value.code == bsr.BSR_E_ARG
    with pytest.raises(bsr.BsrError) as e:
        bsr.bsr_ctx_create(L, 4, hip_device=-1, staging_budget_bytes=1 << 40,
                           max_bound_requests=bsr.BSR_MAX_BOUND_REQUESTS + 1)
    assert e.value.code == bsr.BSR_E_ARG
    for W, B, M, want in [(4, 0, 0, 1), (4, 0, 1, 1), (4, 4 * c, 0, 1), (4, 14 * c, 0, 3),
                          (4, 1 << 40, 0, bsr.BSR_MAX_BOUND_REQUESTS), (4, 14 * c, 7, 7),
                          (0, c, 0, 1), (0, 5 * c + 1, 0, 5), (0, 1 << 40, 0, bsr.BSR_MAX_BOUND_REQUESTS)]:
        ctx = bsr.bsr_ctx_create(L, W, hip_device=-1, staging_budget_bytes=B, max_bound_requests=M)
        try:
            a = bsr.bsr_admission_get(ctx)
            assert a["staging_budget_bytes"] == B and a["max_bound_requests"] == want
            assert a["n_bound"] == a["bound_staging_bytes"] == a["peak_n_bound"] == a["n_refused"] == 0
            assert a["aux_device_bytes"] == 0          # host-only context: no session resources
            with pytest.raises(bsr.BsrError) as e:
                bsr.bsr_request_stats(ctx, 7)
            assert e.value.code == bsr.BSR_E_NOTFOUND
            assert bsr.bsr_stats_get(ctx)["window_chunks"] == W
        finally:
            bsr.bsr_ctx_destroy(ctx)


def test_install_grid_limit():
    """One install launch runs install_batch x (workgroups per chunk) workgroups
    of 128 threads (the install kernel's workgroup size); a layout and batch
    whose grid would pass 2^32 - 1 work-items is refused at creation, and a
    smaller batch is accepted."""
    def layout(n_tensors):   # one token per chunk and per block, 4-byte records: one workgroup per tensor
        return bsr.make_layout(1, [(1, n_tensors, 4, bsr.BSR_KIND_CONTIG, 0)])
    limit = (1 << 32) // (32 * 128)          # 1,048,576 tensors at the automatic batch of 32 (W = 64)
    with pytest.raises(bsr.BsrError) as e:
        bsr.bsr_ctx_create(layout(limit), 64, hip_device=-1)
    assert e.value.code == bsr.BSR_E_ARG and "grid limit" in bsr.bsr_last_error()
    for n, W, b in [(limit - 1, 64, 0), (limit, 64, 16), (limit, 0, 16)]:
        bsr.bsr_ctx_destroy(bsr.bsr_ctx_create(layout(n), W, hip_device=-1, install_batch=b))
    with pytest.raises(bsr.BsrError) as e:
        bsr.bsr_ctx_create(layout(limit), 0, hip_device=-1)      # whole-plan mode: batch 32
    assert e.value.code == bsr.BSR_E_ARG


def test_put_chunks_matches_put_chunk_and_keeps_a_prefix_contiguous():
    """Bulk insertion: same entries and tags as one put per chunk; the chunks
    of one call sit in consecutive arena blocks; all or nothing when full."""
    w = random_workload(6)
    wi = generate(w)
    G = len(w.groups)
    case = build_case(wi)
    n = w.held_chunks
    ctx = bsr.bsr_ctx_create(_layout(w), 2, hip_device=-1)
    slot = bsr.bsr_slot_bytes(ctx.layout)
    stride = (slot + 4095) // 4096 * 4096
    arena = np.zeros(stride * (n + 3), np.uint8)
    try:
        bsr.bsr_store_adopt(ctx, arena.ctypes.data, arena.nbytes)
        bsr.bsr_store_put_chunk(ctx, 12345, wi.payloads(0))          # one block used first
        bsr.bsr_store_put_chunks(ctx, case.keys[:n], [wi.payloads(i) for i in range(n)])
        addrs = []
        for i in range(n):
            for g in range(G):
                addr, nbytes, tag = bsr.bsr_store_payload(ctx, case.keys[i], g)
                assert tag == case.store.get(case.keys[i], g)[1]
                got = np.ctypeslib.as_array((ctypes.c_uint8 * nbytes).from_address(addr))
                np.testing.assert_array_equal(got, wi.payload(i, g))
            addrs.append(bsr.bsr_store_payload(ctx, case.keys[i], 0)[0])
        assert all(b - a == stride for a, b in zip(addrs, addrs[1:]))
        assert bsr.bsr_store_count(ctx) == (G * (n + 1), stride * (n + 1))
        pn, _, _ = bsr.bsr_probe(ctx, 1, wi.salt, wi.tokens)
        assert pn == oracle.probe(case.store, wi.tokens, w.chunk_tokens, wi.salt)[0]
        # three more chunks do not fit the two free blocks: nothing is stored
        with pytest.raises(bsr.BsrError) as e:
            bsr.bsr_store_put_chunks(ctx, [7, 8, 9], [wi.payloads(0)] * 3)
        assert e.value.code == bsr.BSR_E_NOMEM
        assert bsr.bsr_store_count(ctx)[0] == G * (n + 1)
        # a key repeated within one call: the later payload wins, one block kept
        bsr.bsr_store_put_chunks(ctx, [7, 7], [wi.payloads(0), wi.payloads(1)])
        assert bsr.bsr_store_payload(ctx, 7, 0)[2] == oracle.entry_tag(wi.payload(1, 0))
        assert bsr.bsr_store_count(ctx) == (G * (n + 2), stride * (n + 2))
    finally:
        bsr.bsr_ctx_destroy(ctx)


def test_unknown_config_flags_are_rejected():
    w = get_config(2)
    with pytest.raises(bsr.BsrError) as e:
        bsr.bsr_ctx_create(_layout(w), 4, hip_device=-1, flags=0x80)
    assert e.value.code == bsr.BSR_E_ARG
    ctx = bsr.bsr_ctx_create(_layout(w), 4, hip_device=-1,
                             flags=bsr.BSR_FLAG_TIME_INSTALL | bsr.BSR_FLAG_TRUSTED_TABLES)
    bsr.bsr_ctx_destroy(ctx)
