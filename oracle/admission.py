"""Global admission budget B over concurrently bound restores -- TEST INFRASTRUCTURE.

§7 "Current concurrency is conservative": the prototype admits one bounded
restore at a time (the bounded-retrieve lock of §3 "Install locally" and the
§4 component table), so the configured staging budget is never multiplied.
The extension the paper names is a global budget B: several requests'
windows may be live together as long as their aggregate restore working set
stays within B.

Plain definition used here (this build's reading of that sentence):

* a request's restore working set is the ring it binds, ``plan_staging``:
  W * c with a bounded window (Eq. 5), n * c in whole-plan mode (Eq. 2);
* B = 0 keeps the lock: a bind is admitted iff no request is bound;
* B > 0: a bind is refused as "too_large" when its own ring exceeds B (it
  could never run), refused as "busy" when the rings already bound plus its
  own would exceed B or every session slot (at most ``max_bound``) is in
  use, and admitted otherwise;
* "end" releases the request's ring (commit or teardown).

The replay returns each bind's outcome and the peak aggregate; nothing else
is modelled (no fairness, no queueing: a refused bind is simply retried
later by its caller).
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Sequence, Tuple

OK = "ok"
BUSY = "busy"
TOO_LARGE = "too_large"


def plan_staging(W: int, n_hit: int, slot_bytes: int) -> int:
    """Ring bytes of one request: W*c (Eq. 5) or, with W = 0, n*c (Eq. 2, at least one slot)."""
    return (W if W else max(1, n_hit)) * slot_bytes


@dataclass
class AdmissionTrace:
    outcomes: List[str] = field(default_factory=list)   # one per "bind" event, in order
    peak_bound_bytes: int = 0
    peak_bound: int = 0
    refused_busy: int = 0


def replay(budget: int, max_bound: int, W: int, slot_bytes: int,
           events: Sequence[Tuple]) -> AdmissionTrace:
    """events: ("bind", request_id, n_hit) or ("end", request_id), in order."""
    bound: Dict[int, int] = {}          # request id -> ring bytes
    tr = AdmissionTrace()
    for ev in events:
        if ev[0] == "end":
            bound.pop(ev[1], None)
            continue
        _, rid, n_hit = ev
        need = plan_staging(W, n_hit, slot_bytes)
        if budget == 0:
            out = OK if not bound else BUSY
        elif need > budget:
            out = TOO_LARGE
        elif sum(bound.values()) + need > budget or len(bound) >= max_bound:
            out = BUSY
        else:
            out = OK
        if out == OK:
            bound[rid] = need
            tr.peak_bound_bytes = max(tr.peak_bound_bytes, sum(bound.values()))
            tr.peak_bound = max(tr.peak_bound, len(bound))
        elif out == BUSY:
            tr.refused_busy += 1
        tr.outcomes.append(out)
    return tr
