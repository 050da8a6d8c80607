"""Chunk keys of a token sequence: the key space of the restore plan.

§2 "Restoration Capacity as a Resource": a request's reusable state induces
an ordered restore plan of chunk units u_1..u_N; a chunk spans the
registered per-rank state of a fixed token range (256 tokens in the paper's
evaluation, §4 "System topology").  Reuse is a prefix, so a chunk's key must
name the whole token prefix up to and including that chunk.  The paper does
not fix the key function; this build's reading is a two-level FNV-1a-64:

    d_i = FNV1a64(little-endian int32 bytes of tokens[i*C : (i+1)*C])
    h_i = FNV1a64(LE64(h_{i-1}) || LE64(d_i)),   h_{-1} = salt

Only full chunks are keyed (N = floor(T / C)); a trailing partial chunk is
never a hit.  The salt is the per-run key namespace: §5 "Experiment 2" reruns
the largest state "with a new salt", which must find fresh keys.
"""

from typing import List

import numpy as np

from .fnv import fnv1a64


def chunk_digest(chunk_tokens: np.ndarray) -> int:
    return fnv1a64(np.ascontiguousarray(chunk_tokens, dtype="<i4").tobytes())


def chain_keys(tokens: np.ndarray, chunk_tokens: int, salt: int) -> List[int]:
    n_chunks = len(tokens) // chunk_tokens
    h = salt
    keys = []
    for i in range(n_chunks):
        d = chunk_digest(tokens[i * chunk_tokens:(i + 1) * chunk_tokens])
        h = fnv1a64(h.to_bytes(8, "little") + d.to_bytes(8, "little"))
        keys.append(h)
    return keys
