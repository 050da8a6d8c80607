"""Place a generated workload's destination state on the GPU with torch.

Allocates one pool tensor per (group, tensor) of ``pool_blocks x
block_bytes`` bytes, fills it with the workload's sentinel pattern, and
uploads block tables and initial valid bytes.  Input placement only.
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import List

import numpy as np
import torch

from .gen import SENTINEL_STRIDE, WorkloadInputs


@dataclass
class DeviceInputs:
    pools: List[List[torch.Tensor]]      # [group][tensor] uint8 [pool_blocks, block_bytes]
    tensor_bases: List[torch.Tensor]     # [group] int64 [n_tensors] device addresses
    block_tables: List[torch.Tensor]     # [group] int32 [needed_blocks]
    valid: List[torch.Tensor]            # [group] uint8 [pool_blocks]


def fill_sentinel(pool: torch.Tensor, seeds: np.ndarray) -> None:
    """pool[b, j] = (seeds[b] + 37 * j) mod 256, computed on the device."""
    pb, bb = pool.shape
    ramp = ((torch.arange(bb, device=pool.device, dtype=torch.int64) * SENTINEL_STRIDE) & 0xFF).to(torch.uint8)
    s = torch.from_numpy(np.ascontiguousarray(seeds)).to(pool.device)
    torch.add(s[:, None], ramp[None, :], out=pool)


def place(wi: WorkloadInputs, device: str = "cuda:0") -> DeviceInputs:
    pools, bases, tables, valid = [], [], [], []
    for g, spec in enumerate(wi.workload.groups):
        pb, bb = wi.pool_blocks[g], wi.block_bytes(g)
        per_t = []
        for t in range(spec.n_tensors):
            p = torch.empty((pb, bb), dtype=torch.uint8, device=device)
            fill_sentinel(p, wi.sentinel_seed[g][t])
            per_t.append(p)
        pools.append(per_t)
        bases.append(torch.tensor([p.data_ptr() for p in per_t], dtype=torch.int64, device=device))
        tables.append(torch.from_numpy(wi.block_tables[g]).to(device))
        valid.append(torch.from_numpy(wi.valid_init[g]).to(device))
    return DeviceInputs(pools, bases, tables, valid)
