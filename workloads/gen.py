"""Seeded generators for a :class:`~workloads.configs.Workload`.

Seeds: workload ``k`` draws its integers (tokens, block tables, salt, payload
offsets, initial valid bytes, pool sentinels, failure points, in that order)
from ``numpy.random.Generator(PCG64(k - 1))`` and its values from
``torch.Generator().manual_seed(1000 + k)``.  Workload 1's tokens therefore
come from seed 0.

The external tier holds, for every held chunk ``i`` and group ``g``, one
payload of ``n_tensors x chunk_tokens`` records in tensor-major, token-minor
order: record (t, q) is tensor t's bytes for token ``i * chunk_tokens + q``.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np
import torch

from .configs import GroupSpec, VOCAB, Workload

SENTINEL_STRIDE = 37  # byte j of a pool block holds (seed + 37 * j) mod 256


def _bf16_records(n_records: int, record_bytes: int, gen: torch.Generator) -> np.ndarray:
    n_vals = n_records * record_bytes // 2
    x = torch.randn(n_vals, generator=gen, dtype=torch.float32).to(torch.bfloat16)
    return x.view(torch.int16).numpy().view(np.uint8).reshape(n_records, record_bytes)


def _fp8_scaled_records(n_records: int, record_bytes: int, split_bytes: int,
                        gen: torch.Generator) -> np.ndarray:
    """Records of ``split_bytes`` fp8-e4m3fn values followed by their fp32 scale.

    scale = max|x| / 448 (448 is e4m3fn's largest finite value); the values
    are x / scale rounded by torch's CPU cast.
    """
    assert record_bytes == split_bytes + 4
    x = torch.randn(n_records, split_bytes, generator=gen, dtype=torch.float32)
    scale = x.abs().amax(dim=1) / 448.0
    q = (x / scale[:, None]).to(torch.float8_e4m3fn)
    out = np.empty((n_records, record_bytes), dtype=np.uint8)
    out[:, :split_bytes] = q.view(torch.uint8).numpy()
    out[:, split_bytes:] = scale.numpy().astype("<f4").view(np.uint8).reshape(n_records, 4)
    return out


def _records(spec: GroupSpec, n_records: int, gen: torch.Generator) -> np.ndarray:
    if spec.value_kind == "bf16":
        return _bf16_records(n_records, spec.record_bytes, gen)
    if spec.value_kind == "fp8_scaled":
        return _fp8_scaled_records(n_records, spec.record_bytes, spec.split_bytes, gen)
    if spec.value_kind == "bytes":  # uniform bytes, for random property-test layouts
        return torch.randint(0, 256, (n_records, spec.record_bytes), generator=gen,
                             dtype=torch.uint8).numpy()
    raise ValueError(spec.value_kind)


@dataclass
class WorkloadInputs:
    """Everything a restore of one workload consumes, generated once."""

    workload: Workload
    tokens: np.ndarray                      # int32 [n_tokens]
    salt: int                               # u64 key namespace of this run
    block_tables: List[np.ndarray]          # per group, int32 [needed_blocks]
    pool_blocks: List[int]                  # per group
    valid_init: List[np.ndarray]            # per group, uint8 [pool_blocks] of 0/1
    sentinel_seed: List[np.ndarray]         # per group, uint8 [n_tensors, pool_blocks]
    failure: Dict[str, int] = field(default_factory=dict)
    _base: List[np.ndarray] = field(default_factory=list, repr=False)
    _offsets: List[np.ndarray] = field(default_factory=list, repr=False)

    # ---- payloads held by the external tier -------------------------------
    def entry_records(self, g: int) -> int:
        spec = self.workload.groups[g]
        return spec.n_tensors * self.workload.chunk_tokens

    def payload(self, i: int, g: int) -> np.ndarray:
        """Bytes of chunk ``i``'s entry for group ``g`` (read-only view)."""
        if not 0 <= i < self.workload.held_chunks:
            raise IndexError(i)
        o = int(self._offsets[g][i])
        v = self._base[g][o:o + self.entry_records(g)].reshape(-1)
        v.flags.writeable = False
        return v

    def payloads(self, i: int) -> List[np.ndarray]:
        return [self.payload(i, g) for g in range(len(self.workload.groups))]

    # ---- destination pools -------------------------------------------------
    def block_bytes(self, g: int) -> int:
        spec = self.workload.groups[g]
        return spec.block_tokens * spec.record_bytes

    def sentinel_block(self, g: int, t: int, b: int) -> np.ndarray:
        ramp = (np.arange(self.block_bytes(g), dtype=np.int64) * SENTINEL_STRIDE)
        return ((int(self.sentinel_seed[g][t, b]) + ramp) & 0xFF).astype(np.uint8)

    def sentinel_blocks(self, g: int, blocks: np.ndarray) -> np.ndarray:
        """uint8 [n_tensors, len(blocks), block_bytes]: those pool blocks before restore."""
        bb = self.block_bytes(g)
        ramp = ((np.arange(bb, dtype=np.int64) * SENTINEL_STRIDE) & 0xFF).astype(np.uint8)
        s = self.sentinel_seed[g][:, np.asarray(blocks, dtype=np.int64)]
        out = np.empty(s.shape + (bb,), dtype=np.uint8)
        np.add(s[:, :, None], ramp[None, None, :], out=out)  # uint8 add wraps
        return out

    def sentinel_pool(self, g: int) -> np.ndarray:
        """uint8 [n_tensors, pool_blocks, block_bytes]: the pool before restore."""
        bb = self.block_bytes(g)
        ramp = ((np.arange(bb, dtype=np.int64) * SENTINEL_STRIDE) & 0xFF).astype(np.uint8)
        s = self.sentinel_seed[g]
        return (s[:, :, None] + ramp[None, None, :]).astype(np.uint8)  # uint8 add wraps


def needed_blocks(n_tokens: int, block_tokens: int) -> int:
    return -(-n_tokens // block_tokens)


def generate(w: Workload, values: bool = True) -> WorkloadInputs:
    rng = np.random.Generator(np.random.PCG64(w.index - 1))
    gen = torch.Generator().manual_seed(1000 + w.index)

    tokens = rng.integers(0, VOCAB, size=w.n_tokens, dtype=np.int32)

    block_tables, pool_blocks = [], []
    for spec in w.groups:
        need = needed_blocks(w.n_tokens, spec.block_tokens)
        pool = max(1, need * w.pool_factor)
        if w.permute_blocks and pool == need:
            bt = rng.permutation(pool).astype(np.int32)
        else:
            bt = rng.choice(pool, size=need, replace=False).astype(np.int32)
        block_tables.append(bt)
        pool_blocks.append(pool)

    salt = int(rng.integers(0, 2**63, dtype=np.int64)) * 2 + 1

    held = w.held_chunks
    bases, offsets = [], []
    for spec in w.groups:
        e = spec.n_tensors * w.chunk_tokens
        if w.base_records is None:
            n_base = max(1, held) * e
            offs = np.arange(held, dtype=np.int64) * e
        else:
            n_base = w.base_records
            span = n_base - e + 1
            if span < held:
                raise ValueError(f"base of {n_base} records too small for {held} distinct entries of {e}")
            offs = rng.choice(span, size=held, replace=False).astype(np.int64)
        offsets.append(offs)
        bases.append(_records(spec, n_base, gen) if values else
                     np.zeros((n_base, spec.record_bytes), np.uint8))

    valid_init = [rng.integers(0, 2, size=p, dtype=np.uint8) for p in pool_blocks]
    sentinel_seed = [rng.integers(0, 256, size=(spec.n_tensors, p), dtype=np.uint8)
                     for spec, p in zip(w.groups, pool_blocks)]

    failure: Dict[str, int] = {}
    if w.failure is not None and held > 0:
        g = int(w.failure_group)
        spec = w.groups[g]
        payload_bytes = spec.n_tensors * w.chunk_tokens * spec.record_bytes
        failure["group"] = g
        failure["chunk"] = int(rng.integers(0, held))
        failure["byte"] = int(rng.integers(0, payload_bytes))
        failure["mask"] = int(rng.integers(1, 256))
        failure["seeded_k"] = int(rng.integers(0, max(1, held - 1)))

    return WorkloadInputs(w, tokens, salt, block_tables, pool_blocks, valid_init,
                          sentinel_seed, failure, bases, offsets)


def random_workload(seed: int, max_groups: int = 4) -> Workload:
    """A small random layout for property tests: ragged chunk/block ratios,
    block sizes that do or do not divide the chunk, planar and contiguous
    groups, and a ragged token tail."""
    r = np.random.Generator(np.random.PCG64(10_000 + seed))
    n_groups = int(r.integers(1, max_groups + 1))
    chunk = int(r.choice([8, 16, 24, 32, 48, 64]))
    groups = []
    for gi in range(n_groups):
        bt = int(r.choice([4, 8, 16, 32, 64, 128]))
        nt = int(r.integers(1, 4))
        if r.random() < 0.35:
            split = 4 * int(r.integers(1, 9))
            rec = split + 4 * int(r.integers(1, 4))
            groups.append(GroupSpec(f"p{gi}", bt, nt, rec, kind="planar", split_bytes=split,
                                    value_kind="bytes"))
        else:
            rec = 4 * int(r.integers(1, 40))
            groups.append(GroupSpec(f"c{gi}", bt, nt, rec, value_kind="bytes"))
    n_chunks = int(r.integers(1, 12))
    n_tokens = n_chunks * chunk + int(r.integers(0, chunk))
    w_choices = sorted({1, 2, 3, max(1, n_chunks), n_chunks + 5})
    return Workload(index=100 + seed, name=f"random-{seed}", n_tokens=n_tokens,
                    chunk_tokens=chunk, groups=tuple(groups), windows=tuple(w_choices),
                    pool_factor=2)
