"""Byte geometry of one chunk unit and of the destination blocks.

§2 "Restoration Capacity as a Resource": unit u_i occupies c_i bytes of local
staging while it is installed; with a fixed registration every chunk has the
same size c.  This build's reading of c ("slot bytes"): a staged chunk holds
each allocator group's entry back to back, group g starting at a 256-byte
aligned offset, so

    payload_g  = n_tensors_g * C * record_bytes_g
    off_0 = 0, off_{g+1} = off_g + align_up(payload_g, 256)
    c = slot_bytes = off_G

Inside group g's region the entry is [tensor][token][record] (tensor-major,
token-minor).  A destination block of group g holds block_tokens_g tokens of
one tensor: ``contig`` blocks keep the records in token order; ``planar``
blocks keep the first split_g bytes of every record as one plane followed by
the remaining bytes as a second plane.
"""

from dataclasses import dataclass
from typing import List, Sequence

ALIGN = 256


def align_up(x: int, a: int = ALIGN) -> int:
    return (x + a - 1) // a * a


@dataclass(frozen=True)
class OracleGroup:
    block_tokens: int
    n_tensors: int
    record_bytes: int
    kind: str          # "contig" | "planar"
    split_bytes: int


@dataclass(frozen=True)
class OracleLayout:
    chunk_tokens: int
    groups: tuple

    @staticmethod
    def from_specs(chunk_tokens: int, specs: Sequence) -> "OracleLayout":
        return OracleLayout(chunk_tokens, tuple(
            OracleGroup(s.block_tokens, s.n_tensors, s.record_bytes, s.kind, s.split_bytes)
            for s in specs))

    @property
    def n_groups(self) -> int:
        return len(self.groups)

    def payload_bytes(self, g: int) -> int:
        gr = self.groups[g]
        return gr.n_tensors * self.chunk_tokens * gr.record_bytes

    def group_offsets(self) -> List[int]:
        offs, o = [], 0
        for g in range(self.n_groups):
            offs.append(o)
            o += align_up(self.payload_bytes(g))
        return offs

    @property
    def slot_bytes(self) -> int:
        return sum(align_up(self.payload_bytes(g)) for g in range(self.n_groups))

    @property
    def chunk_payload_bytes(self) -> int:
        return sum(self.payload_bytes(g) for g in range(self.n_groups))

    def block_bytes(self, g: int) -> int:
        gr = self.groups[g]
        return gr.block_tokens * gr.record_bytes
