"""The five restore workloads, stated as plain parameters.

Sizes follow the paper's evaluated registration: 256-token chunks (§4
"System topology"), DeepSeek-style MLA latent KV of 576 bf16 values per token
and layer, 128 fp8-e4m3 index-key values plus one fp32 scale per token, and a
sliding-window KV of 2 x 128 bf16 per token.  The model, its prompts and the
paper's evidence artifacts are not available, so every value is synthetic:
tokens are uniform int32 IDs, bf16 values are N(0, 1), and fp8 values are
N(0, 1) quantised with a per-record scale.

A record is the bytes one registered tensor holds for one token.  A group is
one allocator group of the paged KV cache: all its tensors share a block size
(tokens per paged block) and a block table.  ``kind`` says how a block stores
its tokens' records: ``"contig"`` keeps whole records in token order;
``"planar"`` keeps the first ``split_bytes`` of every record as one plane and
the remaining bytes as a second plane (values plane, then scales plane).
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

VOCAB = 129_280  # token IDs are uniform in [0, VOCAB)

BF16_LATENT_RECORD = 576 * 2          # MLA latent 512 + rope 64, bf16
FP8_INDEX_RECORD = 128 + 4            # 128 fp8-e4m3 values + one fp32 scale
SWA_RECORD = 2 * 128 * 2              # sliding-window K and V, 128 bf16 each


@dataclass(frozen=True)
class GroupSpec:
    name: str
    block_tokens: int
    n_tensors: int
    record_bytes: int
    kind: str = "contig"          # "contig" | "planar"
    split_bytes: int = 0          # planar only: bytes of the first plane per record
    value_kind: str = "bf16"      # "bf16" | "fp8_scaled"  (how record bytes are drawn)


@dataclass(frozen=True)
class Workload:
    """One restore workload.

    ``index`` is the workload number (1..5); seeds derive from it.
    ``hit_chunks`` is how many leading full chunks the external tier holds
    (None = all of them).  ``pool_factor`` oversubscribes each group's paged
    pool relative to the blocks the request needs; ``pool_factor == 1`` with
    ``permute_blocks`` gives a random permutation block table.
    ``base_records`` bounds value generation: when set, each (chunk, group)
    payload is a window of that many-record seeded base, at a seeded record
    offset drawn without replacement, so payloads stay N(0, 1), differ from
    each other, and large workloads generate in seconds.
    """

    index: int
    name: str
    n_tokens: int
    chunk_tokens: int
    groups: Tuple[GroupSpec, ...]
    windows: Tuple[int, ...]
    hit_chunks: Optional[int] = None
    pool_factor: int = 2
    permute_blocks: bool = False
    base_records: Optional[int] = None
    failure: Optional[str] = None       # description of the failure case, if any
    failure_group: Optional[int] = None
    note: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def n_full_chunks(self) -> int:
        return self.n_tokens // self.chunk_tokens

    @property
    def held_chunks(self) -> int:
        return self.n_full_chunks if self.hit_chunks is None else self.hit_chunks


GROUP_A = GroupSpec("A_mla_latent", 64, 32, BF16_LATENT_RECORD)
GROUP_B = GroupSpec("B_index_keys", 128, 8, FP8_INDEX_RECORD, kind="planar",
                    split_bytes=128, value_kind="fp8_scaled")

# 4-group split of 170 registered tensors for the MTP-style share: 30 MLA
# latent, 116 index-key, 21 sliding-window and 3 MTP tensors.
G1_MLA = GroupSpec("G1_mla_latent", 64, 30, BF16_LATENT_RECORD)
G2_IDX = GroupSpec("G2_index_keys", 128, 116, FP8_INDEX_RECORD, kind="planar",
                   split_bytes=128, value_kind="fp8_scaled")
G3_SWA = GroupSpec("G3_swa_kv", 32, 21, SWA_RECORD)
G4_MTP = GroupSpec("G4_mtp_latent", 64, 3, BF16_LATENT_RECORD)

BASE = 1 << 16  # records per seeded base (per group) for the large workloads

CONFIGS = {
    1: Workload(
        index=1, name="tiny-1k", n_tokens=1024, chunk_tokens=64,
        groups=(GroupSpec("A_mla_latent", 16, 2, BF16_LATENT_RECORD),),
        windows=(2,), pool_factor=1, permute_blocks=True,
        note="1,024 tokens, 64-token chunks, one group of 2 x 576 bf16 in 16-token blocks, W=2"),
    2: Workload(
        index=2, name="32k", n_tokens=32_768, chunk_tokens=256,
        groups=(GROUP_A, GROUP_B), windows=(32,), base_records=BASE,
        note="32K tokens, config-2 layout (A: 32 x 576 bf16 @64, B: 8 x (128 fp8 + fp32) @128), W=32"),
    3: Workload(
        index=3, name="128k-75pct", n_tokens=131_072, chunk_tokens=256,
        groups=(GROUP_A, GROUP_B), windows=(8, 16, 32, 64), hit_chunks=384,
        base_records=BASE,
        note="128K tokens, config-2 layout, first 75% of chunks held, W in {8,16,32,64}"),
    4: Workload(
        index=4, name="512k", n_tokens=524_288, chunk_tokens=256,
        groups=(GROUP_A, GROUP_B), windows=(32,), base_records=BASE,
        failure="seeded chunk in group A: missing or corrupt entry, injected after probe",
        failure_group=0,
        note="512K tokens (2,048 chunks), config-2 layout, W=32"),
    5: Workload(
        index=5, name="512k-mtp", n_tokens=524_288, chunk_tokens=256,
        groups=(G1_MLA, G2_IDX, G3_SWA, G4_MTP), windows=(32,), base_records=BASE,
        failure="group G3 entries beyond chunk k removed after probe (k = W-1 and a seeded k)",
        failure_group=2,
        note="512K tokens, 170 tensors in 4 groups (MLA @64, index keys @128, SWA @32, MTP @64), W=32"),
}


def get_config(index: int) -> Workload:
    return CONFIGS[index]
