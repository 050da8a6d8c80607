"""Probe, windowed restore and request-level commit, in the paper's order.

* §3 "Probe globally" / §4 "LMCache changes": probe-only lookup returns the
  retained hit bitmap without staging anything; reuse is the leading run of
  hits (the restore plan is an ordered prefix, §2).
* §2 "Bounded installation" (Eqs. 3-4, Prop. 1): the confirmed prefix of n
  chunks is cut into ordered windows G_1..G_K with |G_j| <= W and
  K = ceil(n / W).  A window's staging is released before its capacity is
  reused, so at most W units are live (Eq. 3) and the peak staging is
  min(W, n) * c (the Eq. 5 law when n >= W).  W = 0 is the legacy
  whole-plan path (§4 "Restore-window configuration"): one window holding
  the whole plan, peak n * c (Eq. 2).
* §4 "LMCache changes": per window, fetch every entry and require complete
  presence, stage it, map it onto the destination blocks of the same chunk
  range, install, then release.  A missing entry, a timeout or a transfer
  error fails the retrieve; this build also fails it when a staged entry's
  tag differs from the tag recorded at store time (a corrupt entry).
* §3 "Commit at request semantics" (Eq. 6 with one rank) and §4 "vLLM
  failure integration": reuse is exposed only if no window failed and every
  group is valid; otherwise every destination block of the advertised prefix
  in every group is marked invalid, zero tokens are exposed and the request
  falls back.  Prop. 2: exposure is all or nothing.
* §3 "Recover without re-entering the same fault": a failed restore sets a
  force-local marker for the request; while it is set, probe reports zero
  external tokens.  Successful RUNNING admission or teardown clears it.

Destination validity is modelled by one byte per pool block per group
(1 = holds valid state).  Binding a request clears the valid bytes of its
advertised blocks; commit sets them to 1 only when Eq. 6 holds.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .keys import chain_keys
from .layout import OracleLayout
from .store import OracleStore
from .tag import entry_tag

FAIL_NONE = 0
FAIL_MISSING = 1     # an entry of the window is absent at fetch time
FAIL_CORRUPT = 2     # a staged entry's tag differs from its stored tag
FAIL_TIMEOUT = 3     # the window's fetch exceeded its deadline
FAIL_TRANSFER = 4    # the transfer of a chunk raised an error
FAIL_ABORT = 5       # the caller invalidated the restore

NO_CHUNK = 0xFFFFFFFF


# --------------------------------------------------------------------------
# probe
# --------------------------------------------------------------------------
def probe(store: OracleStore, tokens: np.ndarray, chunk_tokens: int, salt: int,
          force_local: bool = False) -> Tuple[int, np.ndarray, List[int]]:
    """Probe-only lookup: (n_hit, hit bitmap over the N full chunks, keys).

    bitmap_i = 1 iff every group's entry for chunk key h_i is retained.
    n_hit is the number of leading ones.  Nothing is staged and the store is
    not modified.  With the force-local marker set, the probe reports no
    external hit at all.
    """
    keys = chain_keys(tokens, chunk_tokens, salt)
    bitmap = np.zeros(len(keys), dtype=np.uint8)
    if force_local:
        return 0, bitmap, keys
    for i, h in enumerate(keys):
        bitmap[i] = all(store.has(h, g) for g in range(store.n_groups))
    n_hit = 0
    while n_hit < len(keys) and bitmap[n_hit]:
        n_hit += 1
    return n_hit, bitmap, keys


# --------------------------------------------------------------------------
# window plan and staging accounting
# --------------------------------------------------------------------------
def plan_windows(n: int, W: int) -> List[range]:
    """Ordered windows G_1..G_K of the n-chunk prefix, |G_j| <= W.

    W = 0 (legacy whole-plan mode) is a single window of all n chunks.
    """
    if n == 0:
        return []
    step = n if W == 0 else W
    return [range(s, min(s + step, n)) for s in range(0, n, step)]


def live_trace(windows: Sequence[range], slot_bytes: int) -> List[int]:
    """Live staging bytes after every stage/release event of the window loop.

    Each chunk becomes live when it is staged; a window's chunks are all
    released after the window is installed (Eq. 1 sums c_i over L(t)).
    """
    live, trace = 0, [0]
    for win in windows:
        for _ in win:
            live += slot_bytes
            trace.append(live)
        live = 0
        trace.append(live)
    return trace


def peak_live_staging(n: int, W: int, slot_bytes: int) -> int:
    """RWS of the windowed restore (Eq. 1): the maximum of the live trace."""
    return max(live_trace(plan_windows(n, W), slot_bytes))


def request_blocks(n_hit: int, chunk_tokens: int, block_tokens: int) -> int:
    """Destination blocks of one group that the advertised prefix touches."""
    return -(-(n_hit * chunk_tokens) // block_tokens)


# --------------------------------------------------------------------------
# install mapping (one staged chunk -> paged destination blocks)
# --------------------------------------------------------------------------
def _place(layout: OracleLayout, g: int, blk: np.ndarray, o: int, recs: np.ndarray) -> None:
    """Write records of consecutive tokens o, o+1, .. into one destination block."""
    gr = layout.groups[g]
    m, r = recs.shape
    if gr.kind == "contig":
        blk[o * r:(o + m) * r] = recs.reshape(-1)
    elif gr.kind == "planar":
        s = gr.split_bytes
        blk[o * s:(o + m) * s] = recs[:, :s].reshape(-1)
        p2 = gr.block_tokens * s
        blk[p2 + o * (r - s):p2 + (o + m) * (r - s)] = recs[:, s:].reshape(-1)
    else:
        raise ValueError(gr.kind)


def install_chunk(layout: OracleLayout, i: int, slot: np.ndarray,
                  block_tables: Sequence[np.ndarray], pools: Sequence[np.ndarray]) -> None:
    """Map staged chunk i onto every group's destination blocks.

    Token tau = i*C + q of tensor t goes to block k = tau // B_g at in-block
    position o = tau % B_g, in physical block block_tables[g][k].
    """
    C = layout.chunk_tokens
    offs = layout.group_offsets()
    for g, gr in enumerate(layout.groups):
        region = slot[offs[g]:offs[g] + layout.payload_bytes(g)].reshape(
            gr.n_tensors, C, gr.record_bytes)
        for t in range(gr.n_tensors):
            q = 0
            while q < C:
                k, o = divmod(i * C + q, gr.block_tokens)
                m = min(gr.block_tokens - o, C - q)
                b = int(block_tables[g][k])
                _place(layout, g, pools[g][t, b], o, region[t, q:q + m])
                q += m


# --------------------------------------------------------------------------
# windowed restore + commit
# --------------------------------------------------------------------------
@dataclass
class RestoreResult:
    exposed_tokens: int
    fallback: int
    fail_reason: int
    first_failed_chunk: int
    q: List[int]
    n_windows: int
    peak_live_staging_bytes: int
    h2d_bytes: int
    installed_bytes: int
    trace: List[int] = field(default_factory=list)


def set_request_valid(layout: OracleLayout, n_hit: int, block_tables: Sequence[np.ndarray],
                      valid: Sequence[np.ndarray], value: int) -> None:
    """Set the validity byte of every block the advertised prefix touches, in
    every group (bind clears them; commit sets them to Q, §3 Eq. 6 and §4
    failed-block / HMA-aware invalidation)."""
    for g, gr in enumerate(layout.groups):
        for k in range(request_blocks(n_hit, layout.chunk_tokens, gr.block_tokens)):
            valid[g][int(block_tables[g][k])] = value


def windowed_restore(layout: OracleLayout, store: OracleStore, keys: Sequence[int],
                     n_hit: int, W: int, block_tables: Sequence[np.ndarray],
                     pools: Sequence[np.ndarray], valid: Sequence[np.ndarray],
                     faults: Optional[Dict[int, int]] = None,
                     abort_after_windows: Optional[int] = None,
                     invalid_groups: Sequence[int] = ()) -> RestoreResult:
    """Restore the first ``n_hit`` chunks through a W-slot staging pool.

    ``pools[g]`` is uint8 [n_tensors, pool_blocks, block_bytes] and
    ``valid[g]`` uint8 [pool_blocks]; both are updated in place.
    ``faults`` maps a chunk index to FAIL_TIMEOUT or FAIL_TRANSFER, raised
    when that chunk is fetched.  ``abort_after_windows`` models the caller
    invalidating the restore after that many windows have been installed.
    ``invalid_groups`` are groups whose required state the engine reports
    invalid outside any transfer (its q_g of Eq. 6 is 0, e.g. the scheduler
    found an erroneous block in that group); no window fails for them.
    """
    faults = faults or {}
    C, G = layout.chunk_tokens, layout.n_groups
    offs = layout.group_offsets()
    slot_bytes = layout.slot_bytes
    windows = plan_windows(n_hit, W)
    n_slots = max(1, min(n_hit, W if W > 0 else n_hit))
    staging = np.zeros((n_slots, slot_bytes), dtype=np.uint8)   # the local restore pool

    # bind: the advertised blocks hold no valid state until commit
    set_request_valid(layout, n_hit, block_tables, valid, 0)

    fail, first_failed, q = FAIL_NONE, NO_CHUNK, [1] * G
    for g in invalid_groups:
        q[g] = 0
    live = peak = h2d = installed = 0
    trace = [0]
    n_windows = 0
    for win in windows:
        n_windows += 1
        staged = []
        for i in win:                                  # fetch + stage, plan order
            if i in faults:
                fail, first_failed = faults[i], i
                q = [0] * G
                break
            missing = [g for g in range(G) if not store.has(keys[i], g)]
            if missing:
                fail, first_failed = FAIL_MISSING, i
                for g in missing:
                    q[g] = 0
                break
            slot = staging[i % n_slots]
            bad = []
            for g in range(G):
                data, tag = store.get(keys[i], g)
                slot[offs[g]:offs[g] + data.size] = data
                if entry_tag(slot[offs[g]:offs[g] + data.size]) != tag:
                    bad.append(g)
            live += slot_bytes
            peak = max(peak, live)
            trace.append(live)
            h2d += slot_bytes
            if bad:
                fail, first_failed = FAIL_CORRUPT, i
                for g in bad:
                    q[g] = 0
                break
            staged.append(i)
        for i in staged:                                # install the window
            install_chunk(layout, i, staging[i % n_slots], block_tables, pools)
            installed += layout.chunk_payload_bytes
        live = 0                                        # sync + release
        trace.append(live)
        if fail == FAIL_NONE and abort_after_windows is not None and n_windows >= abort_after_windows:
            fail = FAIL_ABORT
        if fail != FAIL_NONE:
            break

    # commit (Eq. 6, one rank): all groups valid and no window failed
    Q = fail == FAIL_NONE and all(q)
    if Q:
        set_request_valid(layout, n_hit, block_tables, valid, 1)
        exposed, fallback = n_hit * C, 0
    else:
        set_request_valid(layout, n_hit, block_tables, valid, 0)
        exposed, fallback = 0, 1
    return RestoreResult(exposed, fallback, fail, first_failed, q, n_windows, peak, h2d,
                         installed, trace)


# --------------------------------------------------------------------------
# one destination block after a successful restore (for sampled checks)
# --------------------------------------------------------------------------
def expected_block(layout: OracleLayout, store: OracleStore, keys: Sequence[int], n_hit: int,
                   block_table: np.ndarray, g: int, t: int, b: int,
                   before: np.ndarray) -> np.ndarray:
    """Bytes of physical block ``b`` of tensor ``t`` in group ``g`` after a
    successful restore of ``n_hit`` chunks, given its bytes ``before``.

    This is the whole-plan definition: every prefix token of the block takes
    its record from the stored entry of its chunk; everything else keeps its
    previous bytes.
    """
    gr = layout.groups[g]
    C, B = layout.chunk_tokens, gr.block_tokens
    blk = np.array(before, dtype=np.uint8, copy=True)
    hits = np.nonzero(np.asarray(block_table[:request_blocks(n_hit, C, B)]) == b)[0]
    for k in hits:
        for o in range(B):
            tau = int(k) * B + o
            if tau >= n_hit * C:
                break
            i, qq = divmod(tau, C)
            data, _ = store.get(keys[i], g)
            rec = data.reshape(gr.n_tensors, C, gr.record_bytes)[t, qq]
            _place(layout, g, blk, o, rec[None, :])
    return blk


# --------------------------------------------------------------------------
# request-side runtime: force-local markers across admissions
# --------------------------------------------------------------------------
class Runtime:
    """One rank's restore runtime: a store, a window W and force-local markers."""

    def __init__(self, layout: OracleLayout, store: OracleStore, W: int):
        self.layout, self.store, self.W = layout, store, W
        self.force_local: set = set()

    def probe(self, request_id: int, tokens: np.ndarray, salt: int):
        return probe(self.store, tokens, self.layout.chunk_tokens, salt,
                     force_local=request_id in self.force_local)

    def restore(self, request_id: int, keys, n_hit, block_tables, pools, valid, **kw):
        res = windowed_restore(self.layout, self.store, keys, n_hit, self.W, block_tables,
                               pools, valid, **kw)
        if res.fallback:
            self.force_local.add(request_id)
        return res

    def request_running(self, request_id: int) -> None:
        self.force_local.discard(request_id)

    def request_end(self, request_id: int) -> None:
        self.force_local.discard(request_id)
