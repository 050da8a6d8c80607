"""CPU oracle for Bounded-State Restoration (BSR) -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously correct CPU statement of what BSR's restore path
computes: the probe-only prefix lookup, the windowed restore through a
W-slot staging pool, and the request-level commit with whole-prefix
invalidation.  It follows the paper's §2 (restore plan, RWS, Eqs. 1-5,
Propositions 1-2), §3 (probe / install / commit, Eq. 6, force-local
recovery) and §4 (the windowed retrieve routine and failed-block / HMA-aware
invalidation).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never imports, calls or links anything here, and this
package shares no code with it.

Parity status of each part (what pins it, other than itself):
  * FNV-1a-64 primitive: the FNV specification's published constants and
    test vectors, plus the derivation of the offset basis (pinned).
  * chunk-key chain, chunk format, in-block layouts, tag: the paper fixes none
    of these (it keeps LMCache's representation unchanged); they are this
    build's stated readings.  Pinned by invariants (prefix sensitivity,
    brute force on tiny inputs, gather round-trips, library special cases),
    not by paper values: "parity unpinned" by the paper itself.
  * probe prefix, windowed restore image, staging accounting, commit rule:
    pinned by the paper's closed forms and printed numbers (Eq. 5 law,
    whole-plan peaks, Prop. 1, Prop. 2, Theta(|S|) installed bytes).
  * tier choice (remote store, then a lower reusable tier): pinned by the
    outcome table of §6.4 (full reuse from the lower tier when the remote is
    unavailable, zero when both are absent).
  * global admission budget B (§7): pinned by closed forms (B = 0 is the
    one-at-a-time lock; with a bounded window the number admitted together
    is floor(B / (W c)) whatever the plan lengths, Prop. 1) and by brute
    force over short event sequences (the aggregate never exceeds B, and
    every refusal is forced by B or by the slot count).
"""

from .fnv import fnv1a64, fnv0_64, FNV64_OFFSET_BASIS, FNV64_PRIME  # noqa: F401
from .keys import chunk_digest, chain_keys  # noqa: F401
from .layout import OracleLayout  # noqa: F401
from .tag import entry_tag  # noqa: F401
from .store import OracleStore  # noqa: F401
from .tiers import Tier, probe_tiers, PlannedStore, NO_TIER  # noqa: F401
from . import admission  # noqa: F401
from .restore import (  # noqa: F401
    FAIL_NONE, FAIL_MISSING, FAIL_CORRUPT, FAIL_TIMEOUT, FAIL_TRANSFER, FAIL_ABORT,
    Runtime, RestoreResult, probe, plan_windows, live_trace, peak_live_staging,
    windowed_restore, expected_block, request_blocks, set_request_valid, install_chunk,
)
