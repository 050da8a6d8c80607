"""The external tier: retained entries keyed by (chunk key, group).

§2 "Knowledge versus residency" and §3 "Probe globally": the external tier
retains reusable state; probe asks which entries exist, restore fetches them.
Reading of the paper's object granularity: one entry per (chunk, allocator
group), so a fault can hit one group of one chunk; a chunk is a hit only if
every group's entry is present.  A tag is recorded with each entry when it
is stored.
"""

from typing import Dict, Sequence, Tuple

import numpy as np

from .tag import entry_tag


class OracleStore:
    def __init__(self, n_groups: int):
        self.n_groups = n_groups
        self._entries: Dict[Tuple[int, int], Tuple[np.ndarray, int]] = {}

    def put_chunk(self, key: int, payloads: Sequence[np.ndarray]) -> None:
        assert len(payloads) == self.n_groups
        for g, p in enumerate(payloads):
            b = np.array(p, dtype=np.uint8, copy=True).reshape(-1)
            self._entries[(key, g)] = (b, entry_tag(b))

    def has(self, key: int, g: int) -> bool:
        return (key, g) in self._entries

    def get(self, key: int, g: int) -> Tuple[np.ndarray, int]:
        return self._entries[(key, g)]

    def remove(self, key: int, g: int = -1) -> None:
        for gg in (range(self.n_groups) if g < 0 else [g]):
            self._entries.pop((key, gg), None)

    def corrupt(self, key: int, g: int, byte: int, mask: int) -> None:
        """Flip bits of one stored byte without updating the stored tag."""
        b, t = self._entries[(key, g)]
        b[byte] ^= mask
        self._entries[(key, g)] = (b, t)

    def __len__(self) -> int:
        return len(self._entries)
