"""Integrity tag of one stored entry.

§3 "Commit at request semantics" and §4 "LMCache changes": the runtime must
know whether the transferred objects compose a valid request state; a
transfer that delivers wrong bytes must fail the retrieve.  The paper does
not define a checksum; this build's reading (a "corrupt" entry) uses

    tag = (XOR of the entry's little-endian u32 words) << 32
          | (sum of those words mod 2**32)

computed when the entry is stored.  Both halves are order-independent, so
any partition of the words may be reduced in any order.  A single flipped
byte with a non-zero mask always changes the 32-bit sum.
"""

import numpy as np


def entry_tag(payload: np.ndarray) -> int:
    words = np.ascontiguousarray(payload, dtype=np.uint8).view("<u4")
    s = int(words.sum(dtype=np.uint64)) & 0xFFFFFFFF
    x = int(np.bitwise_xor.reduce(words)) if words.size else 0
    return (x << 32) | s
