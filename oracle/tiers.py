"""Ordered external tiers and the per-chunk tier choice of the probe.

§4 "System topology": the evaluated hierarchy keeps remote DRAM as the
external store and local SSD as a lower reusable tier; §3 "Recover without
re-entering the same fault" and Fig. "Evaluated hierarchy": when the remote
store is unavailable, restoration falls back to the lower valid tier (§6.4
outcome table: remote unavailable, SSD healthy -> the full prefix is reused
from SSD; both absent -> zero external reuse).

Reading: a chunk is a hit in the first *available* tier that holds every one
of its groups; the restore fetches each chunk from the tier the probe chose
and fails the window if that tier has become unavailable or lost the entry.
"""

from typing import List, Sequence, Tuple

import numpy as np

from .keys import chain_keys

NO_TIER = 255


class Tier:
    def __init__(self, store, available: bool = True):
        self.store = store
        self.available = available


def probe_tiers(tiers: Sequence[Tier], tokens: np.ndarray, chunk_tokens: int, salt: int,
                n_groups: int, force_local: bool = False) -> Tuple[int, np.ndarray, List[int], np.ndarray]:
    """(n_hit, bitmap, keys, tier of each chunk) over the tiers in order."""
    keys = chain_keys(tokens, chunk_tokens, salt)
    bitmap = np.zeros(len(keys), dtype=np.uint8)
    chunk_tier = np.full(len(keys), NO_TIER, dtype=np.uint8)
    if force_local:
        return 0, bitmap, keys, chunk_tier
    for i, h in enumerate(keys):
        for t, tier in enumerate(tiers):
            if tier.available and all(tier.store.has(h, g) for g in range(n_groups)):
                bitmap[i], chunk_tier[i] = 1, t
                break
    n_hit = 0
    while n_hit < len(keys) and bitmap[n_hit]:
        n_hit += 1
    return n_hit, bitmap, keys, chunk_tier


class PlannedStore:
    """The store a restore fetches from: each chunk's entries come from the
    tier its probe chose, while that tier is available and holds them."""

    def __init__(self, tiers: Sequence[Tier], keys: Sequence[int], chunk_tier: np.ndarray):
        self.tiers = tiers
        self.tier_of = {int(k): int(t) for k, t in zip(keys, chunk_tier)}

    def _tier(self, key):
        t = self.tier_of.get(int(key), NO_TIER)
        return None if t == NO_TIER else self.tiers[t]

    def has(self, key: int, g: int) -> bool:
        tier = self._tier(key)
        return tier is not None and tier.available and tier.store.has(key, g)

    def get(self, key: int, g: int):
        return self._tier(key).store.get(key, g)
