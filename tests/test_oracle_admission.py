"""Pins of the oracle's global admission budget B (§7 "Current concurrency is
conservative") -- CPU.

What pins it, other than itself:
  * B = 0 is the bounded-retrieve lock: replayed against a real
    ``threading.Lock`` taken with a non-blocking acquire;
  * closed form with a bounded window (Prop. 1: a request's working set is
    W c whatever its plan length): binding k requests admits exactly
    min(M, floor(B / (W c))) of them, for any plan lengths;
  * whole-plan mode: equal plans of n chunks admit floor(B / (n c));
  * brute force over every short event sequence: the aggregate never exceeds
    B, and each outcome is forced (a refusal only when B, the slot count or
    the lock leaves no room; an admission only when there is room).
"""

import itertools
import threading

import pytest

from oracle import admission as adm

C5 = 16_404_480   # slot bytes of the 512K multi-group layout


def test_budget_zero_is_a_lock():
    rng = __import__("random").Random(5)
    for _ in range(200):
        events, live = [], set()
        for _ in range(12):
            rid = rng.randrange(4)
            if rid in live and rng.random() < 0.6:
                events.append(("end", rid))
                live.discard(rid)
            elif rid not in live:
                events.append(("bind", rid, rng.randrange(1, 50)))
                live.add(rid)
        lock = threading.Lock()
        holder = None
        want = []
        for ev in events:
            if ev[0] == "bind":
                if lock.acquire(blocking=False):
                    holder = ev[1]
                    want.append(adm.OK)
                else:
                    want.append(adm.BUSY)
            elif ev[1] == holder:
                lock.release()
                holder = None
        got = adm.replay(0, 1, 32, C5, events).outcomes
        assert got == want


@pytest.mark.parametrize("W", [1, 8, 32, 64])
@pytest.mark.parametrize("k_fit", [1, 2, 3, 5])
def test_bounded_window_admits_floor_b_over_wc(W, k_fit):
    B = k_fit * W * C5 + (W * C5) // 2            # room for k_fit rings and a half
    plans = [1, 2048, 7, 512, 3, 2048, 900, 64]   # plan length does not matter (Prop. 1)
    tr = adm.replay(B, 16, W, C5, [("bind", r, n) for r, n in enumerate(plans)])
    k = min(16, B // (W * C5))
    assert k == k_fit
    assert tr.outcomes == [adm.OK] * k + [adm.BUSY] * (len(plans) - k)
    assert tr.peak_bound_bytes == k * W * C5 <= B
    # the slot count binds first when it is smaller
    tr = adm.replay(B, 1, W, C5, [("bind", r, n) for r, n in enumerate(plans)])
    assert tr.outcomes.count(adm.OK) == 1


def test_exact_fit_and_release():
    W = 4
    B = 2 * W * C5
    ev = [("bind", 1, 9), ("bind", 2, 9), ("bind", 3, 9), ("end", 1), ("bind", 3, 9), ("bind", 4, 9)]
    tr = adm.replay(B, 8, W, C5, ev)
    assert tr.outcomes == [adm.OK, adm.OK, adm.BUSY, adm.OK, adm.BUSY]
    assert tr.peak_bound_bytes == B and tr.peak_bound == 2 and tr.refused_busy == 2


@pytest.mark.parametrize("n,k", [(1, 6), (3, 2), (6, 1), (7, 0)])
def test_whole_plan_equal_plans(n, k):
    B = 6 * C5
    tr = adm.replay(B, 16, 0, C5, [("bind", r, n) for r in range(8)])
    assert tr.outcomes.count(adm.OK) == k == B // (n * C5)
    if k == 0:
        assert set(tr.outcomes) == {adm.TOO_LARGE}


def test_paper_scale_contrast():
    """512K tokens = 2048 chunks: a 2 GiB budget holds four bounded W=32
    restores together, and cannot hold one whole-plan restore (Eq. 2 vs Eq. 5)."""
    B = 2 << 30
    assert adm.plan_staging(32, 2048, C5) == 524_943_360
    tr = adm.replay(B, 16, 32, C5, [("bind", r, 2048) for r in range(6)])
    assert tr.outcomes == [adm.OK] * 4 + [adm.BUSY] * 2
    assert adm.replay(B, 16, 0, C5, [("bind", 0, 2048)]).outcomes == [adm.TOO_LARGE]
    assert adm.plan_staging(0, 2048, C5) == 33_596_375_040


def _sequences(n_ids, length):
    acts = [("bind", r, n) for r in range(n_ids) for n in (1, 2, 3)] + [("end", r) for r in range(n_ids)]
    return itertools.product(acts, repeat=length)


@pytest.mark.parametrize("W", [0, 2])
def test_brute_force_outcomes_are_forced(W):
    c = 5
    for B in (0, c, 2 * c, 3 * c, 4 * c, 6 * c):
        for M in (1, 2, 3):
            if B == 0 and M != 1:
                continue
            for length in (1, 2, 3, 4):
                for seq in _sequences(2, length):
                    tr = adm.replay(B, M, W, c, seq)
                    bound = {}
                    outs = iter(tr.outcomes)
                    for ev in seq:
                        if ev[0] == "end":
                            bound.pop(ev[1], None)
                            continue
                        out = next(outs)
                        need = (W or ev[2]) * c
                        room = (not bound) if B == 0 else (sum(bound.values()) + need <= B and len(bound) < M)
                        if out == adm.OK:
                            assert room
                            bound[ev[1]] = need
                        elif out == adm.TOO_LARGE:
                            assert B and need > B
                        else:
                            assert not room and not (B and need > B)
                        if B:
                            assert sum(bound.values()) <= B
                        assert len(bound) <= (1 if B == 0 else M)
