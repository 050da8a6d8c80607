"""Whole destination pools compared byte for byte with the oracle, in slices.

At 512K tokens the pools hold 40-67 GB, too much for one host image.  The
comparison therefore walks the advertised prefix in slices of whole chunks.
For each slice, the oracle's install mapping (``oracle.install_chunk``)
writes the slice's staged chunks into a pool restricted to the physical
blocks those chunks reach, each holding its bytes from before the restore.
The same blocks are gathered from the device pools and compared.  Blocks
outside the advertised prefix are compared, in slices too, with their bytes
from before the restore.  The two passes together cover every byte of every
pool, and the valid bytes are compared whole.

Pools are lists (per group) of torch tensors [pool_blocks, block_bytes] per
tensor, on the GPU in the GPU tests; the CPU tests run the same code on CPU
tensors.
"""

from __future__ import annotations

import math
import threading
import time
from concurrent.futures import ThreadPoolExecutor
from typing import Callable, List, Optional, Sequence

import numpy as np
import torch

import oracle
from oracle_side import oracle_layout

SLICE_BYTES = 1 << 30        # about this many pool bytes per slice
_CMP_PIECE = 32 << 20        # bytes compared per task


class _SlicePool:
    """One group's pool, restricted to a set of physical blocks.

    The oracle's install mapping indexes it as ``pool[t, b]``; a write to a
    block outside the set means the slice was cut wrong, and raises.
    """

    def __init__(self, arr: np.ndarray, pos: np.ndarray):
        self.arr, self.pos = arr, pos

    def __getitem__(self, idx):
        t, b = idx
        p = int(self.pos[int(b)])
        if p < 0:
            raise IndexError(f"block {b} is outside the slice")
        return self.arr[t, p]


def _slot(layout: oracle.OracleLayout, store, key: int) -> np.ndarray:
    """Staged bytes of one chunk: every group's entry at its slot offset."""
    slot = np.zeros(layout.slot_bytes, np.uint8)
    for g, off in enumerate(layout.group_offsets()):
        data = store.payload(key, g) if hasattr(store, "payload") else store.get(key, g)[0]
        slot[off:off + data.size] = data
    return slot


def slice_unit(layout: oracle.OracleLayout) -> int:
    """Chunks per slice unit: slices start on a block boundary in every group."""
    C = layout.chunk_tokens
    u = 1
    for gr in layout.groups:
        u = math.lcm(u, math.lcm(C, gr.block_tokens) // C)
    return u


def expected_request_slice(layout, wi, store, keys, c0: int, c1: int, n: int):
    """Per group: (physical blocks, expected bytes [T, nb, bb]) of the request
    blocks that chunks [c0, c1) of an n-chunk prefix reach, after a successful
    restore."""
    C = layout.chunk_tokens
    out, pools = [], []
    for g, gr in enumerate(layout.groups):
        B = gr.block_tokens
        assert (c0 * C) % B == 0, "slices start on a block boundary"
        k0 = c0 * C // B
        k1 = -(-(min(c1, n) * C) // B)
        phys = np.asarray(wi.block_tables[g][k0:k1], dtype=np.int64)
        arr = wi.sentinel_blocks(g, phys)
        pos = np.full(wi.pool_blocks[g], -1, np.int64)
        pos[phys] = np.arange(len(phys))
        pools.append(_SlicePool(arr, pos))
        out.append((phys, arr))
    for i in range(c0, min(c1, n)):
        oracle.install_chunk(layout, i, _slot(layout, store, keys[i]), wi.block_tables, pools)
    return out


_tls = threading.local()


def _host_buffer(nbytes: int, pinned: bool) -> np.ndarray:
    """A per-thread host landing buffer (pinned when the pools are on a GPU)."""
    buf = getattr(_tls, "buf", None)
    if buf is None or buf.numel() < nbytes:
        _tls.buf = None
        _tls.buf = torch.empty(max(nbytes, 1), dtype=torch.uint8, pin_memory=pinned)
        buf = _tls.buf
    return buf


def gather(pools_g: Sequence[torch.Tensor], phys: np.ndarray) -> np.ndarray:
    """Blocks ``phys`` of every tensor of one group, on the host: [T, nb, bb]."""
    dev = pools_g[0].device
    idx = torch.from_numpy(np.ascontiguousarray(phys, dtype=np.int64)).to(dev)
    got = torch.stack([p.index_select(0, idx) for p in pools_g])
    n = got.numel()
    host = _host_buffer(n, dev.type == "cuda")[:n].view(got.shape)
    host.copy_(got)
    if dev.type == "cuda":
        torch.cuda.current_stream(dev).synchronize()
    return host.numpy()


def assert_same(got: np.ndarray, want: np.ndarray, what: str, ex: ThreadPoolExecutor) -> None:
    assert got.shape == want.shape, f"{what}: shape {got.shape} != {want.shape}"
    a, b = got.reshape(-1), want.reshape(-1)
    spans = [(s, min(s + _CMP_PIECE, a.size)) for s in range(0, a.size, _CMP_PIECE)]
    ok = list(ex.map(lambda s: bool(np.array_equal(a[s[0]:s[1]], b[s[0]:s[1]])), spans))
    if all(ok):
        return
    s = spans[ok.index(False)]
    j = s[0] + int(np.flatnonzero(a[s[0]:s[1]] != b[s[0]:s[1]])[0])
    idx = np.unravel_index(j, got.shape)
    raise AssertionError(f"{what}: first difference at [tensor, block slot, byte] = {tuple(int(x) for x in idx)}: "
                         f"device {int(a[j])} != oracle {int(b[j])}")


def compare_request_blocks(pools, wi, keys, n: int, store=None, log: Callable[[str], None] = print,
                           slice_bytes: int = SLICE_BYTES, workers: int = 4) -> int:
    """Every advertised block of every group against the oracle's install of
    the n-chunk prefix (a successful restore).  Returns the bytes compared."""
    from oracle_side import GeneratorStore
    layout = oracle_layout(wi)
    store = store or GeneratorStore(wi, keys)
    unit = slice_unit(layout)
    per = max(unit, slice_bytes // max(1, layout.chunk_payload_bytes) // unit * unit)
    slices = [(c0, min(c0 + per, n)) for c0 in range(0, n, per)]
    done = [0]
    t0 = time.time()
    with ThreadPoolExecutor(16) as cmp_ex, ThreadPoolExecutor(workers) as ex:
        def one(sl):
            c0, c1 = sl
            exp = expected_request_slice(layout, wi, store, keys, c0, c1, n)
            nbytes = 0
            for g, (phys, arr) in enumerate(exp):
                got = gather(pools[g], phys)
                assert_same(got, arr, f"group {g}, chunks [{c0}, {c1}), request blocks", cmp_ex)
                nbytes += arr.nbytes
            return sl, nbytes
        for (c0, c1), nb in ex.map(one, slices):
            done[0] += nb
            log(f"  request blocks of chunks [{c0}, {c1}) equal the oracle "
                f"({done[0] / 1e9:.1f} GB, {time.time() - t0:.0f}s)")
    return done[0]


def compare_untouched_blocks(pools, wi, n: int, log: Callable[[str], None] = print,
                             slice_bytes: int = SLICE_BYTES, workers: int = 4) -> int:
    """Every block outside the advertised prefix against its bytes before the
    restore.  Returns the bytes compared."""
    layout = oracle_layout(wi)
    C = layout.chunk_tokens
    jobs = []
    for g, gr in enumerate(layout.groups):
        nreq = oracle.request_blocks(n, C, gr.block_tokens)
        others = np.setdiff1d(np.arange(wi.pool_blocks[g]), np.asarray(wi.block_tables[g][:nreq]))
        per = max(1, slice_bytes // (gr.n_tensors * layout.block_bytes(g)))
        jobs += [(g, others[s:s + per]) for s in range(0, len(others), per)]
    done = [0]
    t0 = time.time()
    with ThreadPoolExecutor(16) as cmp_ex, ThreadPoolExecutor(workers) as ex:
        def one(job):
            g, blocks = job
            want = wi.sentinel_blocks(g, blocks)
            assert_same(gather(pools[g], blocks), want, f"group {g}, blocks outside the prefix", cmp_ex)
            return want.nbytes
        for i, nb in enumerate(ex.map(one, jobs)):
            done[0] += nb
            if i % 8 == 7 or i + 1 == len(jobs):
                log(f"  blocks outside the prefix unchanged ({done[0] / 1e9:.1f} GB, {time.time() - t0:.0f}s)")
    return done[0]


def compare_full_image(pools, wi, keys, n: int, store=None, log: Callable[[str], None] = print,
                       slice_bytes: int = SLICE_BYTES) -> int:
    """Every byte of every pool after a successful restore of n chunks."""
    a = compare_request_blocks(pools, wi, keys, n, store=store, log=log, slice_bytes=slice_bytes)
    b = compare_untouched_blocks(pools, wi, n, log=log, slice_bytes=slice_bytes)
    total = sum(len(p) * p[0].numel() for p in pools)
    assert a + b == total, f"compared {a + b} of {total} pool bytes"
    return total
