"""Build the CPU oracle's view of a generated workload (tests only)."""

from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional

import numpy as np

import oracle
from workloads import WorkloadInputs


@dataclass
class OracleCase:
    layout: oracle.OracleLayout
    store: oracle.OracleStore
    keys: List[int]
    pools: List[np.ndarray]
    valid: List[np.ndarray]


def oracle_layout(wi: WorkloadInputs) -> oracle.OracleLayout:
    return oracle.OracleLayout.from_specs(wi.workload.chunk_tokens, wi.workload.groups)


def build_case(wi: WorkloadInputs, held: Optional[int] = None, with_pools: bool = True,
               tiny_payloads: bool = False) -> OracleCase:
    """Fill an oracle store with the workload's held chunks.

    ``tiny_payloads`` stores 4-byte stand-ins (enough for probe-only tests,
    which never read payloads).
    """
    w = wi.workload
    layout = oracle_layout(wi)
    store = oracle.OracleStore(layout.n_groups)
    keys = oracle.chain_keys(wi.tokens, w.chunk_tokens, wi.salt)
    held = w.held_chunks if held is None else held
    for i in range(held):
        if tiny_payloads:
            store.put_chunk(keys[i], [np.zeros(4, np.uint8)] * layout.n_groups)
        else:
            store.put_chunk(keys[i], wi.payloads(i))
    pools = [wi.sentinel_pool(g) for g in range(layout.n_groups)] if with_pools else []
    valid = [v.copy() for v in wi.valid_init]
    return OracleCase(layout, store, keys, pools, valid)


class GeneratorStore:
    """Read-only stand-in for OracleStore over a workload's generated payloads.

    Presents the entries of chunks [0, held) under the oracle's chunk keys,
    minus removed ones, with tags computed by the oracle on first use; lets
    full-size checks call the oracle without copying the whole external tier.
    """

    def __init__(self, wi: WorkloadInputs, keys: List[int], held: Optional[int] = None):
        self.wi = wi
        self.n_groups = len(wi.workload.groups)
        held = wi.workload.held_chunks if held is None else held
        self.index = {int(k): i for i, k in enumerate(keys[:held])}
        self.removed = set()
        self._tags = {}

    def has(self, key: int, g: int) -> bool:
        return int(key) in self.index and (int(key), g) not in self.removed

    def payload(self, key: int, g: int) -> np.ndarray:
        """The entry's bytes alone (no tag computed)."""
        return self.wi.payload(self.index[int(key)], g)

    def get(self, key: int, g: int):
        i = self.index[int(key)]
        p = self.wi.payload(i, g)
        if (i, g) not in self._tags:
            self._tags[(i, g)] = oracle.entry_tag(p)
        return p, self._tags[(i, g)]

    def remove(self, key: int, g: int = -1) -> None:
        for gg in (range(self.n_groups) if g < 0 else [g]):
            self.removed.add((int(key), gg))


class _SinkTensor:
    def __init__(self, block_bytes: int):
        self.scratch = np.zeros(block_bytes, np.uint8)

    def __getitem__(self, idx):
        return self.scratch


class SinkPools(list):
    """Destination pools that accept every block write into one scratch block
    per group: lets the oracle walk a full-size failing restore (whose pool
    contents are unspecified) for its metadata without a 40-70 GB image."""

    def __init__(self, wi: WorkloadInputs):
        super().__init__(_SinkTensor(wi.block_bytes(g)) for g in range(len(wi.workload.groups)))
