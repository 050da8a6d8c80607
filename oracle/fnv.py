"""FNV hashes, 64-bit, written from the FNV specification (Fowler, Noll, Vo).

FNV-1a processes one octet at a time: XOR the octet into the hash, then
multiply by the FNV prime modulo 2**64.  FNV-0 is the historic variant with
a zero offset basis and multiply-before-XOR; the specification derives the
FNV-1/FNV-1a 64-bit offset basis as the FNV-0 hash of a fixed 32-octet
string, which the tests use as an independent pin of the basis.

The paper does not name a hash for chunk keys (§3 "Probe globally" only
needs a retained hit set, and §5 "Experiment 2" a per-run salt); FNV-1a-64
is this build's reading.  Pure Python integers: slow and exact.
"""

MASK64 = (1 << 64) - 1
FNV64_PRIME = 0x00000100000001B3          # 2**40 + 2**8 + 0xb3
FNV64_OFFSET_BASIS = 0xCBF29CE484222325


def fnv1a64(data: bytes, h: int = FNV64_OFFSET_BASIS) -> int:
    """FNV-1a-64 of ``data`` (continuing from hash state ``h``)."""
    for octet in data:
        h ^= octet
        h = (h * FNV64_PRIME) & MASK64
    return h


def fnv0_64(data: bytes) -> int:
    """FNV-0-64: zero basis, multiply then XOR (used only to derive the basis)."""
    h = 0
    for octet in data:
        h = (h * FNV64_PRIME) & MASK64
        h ^= octet
    return h
