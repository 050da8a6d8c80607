"""Random call sequences against the request state machine (GPU).

A seeded sequence of ABI calls (probe, bind, windows in and out of order,
invalidate, mark a group invalid, commit, teardown, RUNNING admission) on a
few requests of one context with a budget for two rings.  A small Python
model of the protocol (the order rules and admission of include/bsr.h)
predicts each call's status; after every commit the request is either fully
exposed with a pool image equal to the oracle's restore, or exposed not at
all with its advertised blocks invalid (Prop. 2).
"""

import random

import numpy as np
import pytest
import torch

import oracle
from gpu_side import GpuCase, say
from oracle_side import build_case
from paper_2608_17826_amd import bsr
from paper_2608_17826_amd.session import RestoreSession
from workloads import generate, get_config

pytestmark = pytest.mark.gpu

W = 4


class Req:
    def __init__(self, rid, gc):
        self.rid = rid
        self.state = "new"          # new / probed / bound / failed / done
        self.next = 0
        self.n = 0
        self.sess = RestoreSession(gc.ctx)
        self.marked = False
        self.force_local = False


@pytest.mark.parametrize("seed", [1, 2, 3, 4])
def test_random_call_sequences(seed):
    rng = random.Random(seed)
    wi = generate(get_config(1))               # 16 chunks of 64 tokens, one group
    w = wi.workload
    case = build_case(wi)
    n_full, _, keys = oracle.probe(case.store, wi.tokens, w.chunk_tokens, wi.salt)
    ref = oracle.windowed_restore(case.layout, case.store, keys, n_full, W, wi.block_tables,
                                  case.pools, case.valid)
    slot = case.layout.slot_bytes
    gc = GpuCase(wi, W=W)
    bsr.bsr_ctx_destroy(gc.ctx)                 # same store contents, but a context with a budget
    gc.ctx = bsr.bsr_ctx_create(gc.layout, W, hip_device=0, staging_budget_bytes=2 * W * slot)
    stride = (slot + 4095) // 4096 * 4096
    bsr.bsr_store_reserve(gc.ctx, stride * (w.held_chunks + 2))
    bsr.bsr_store_put_chunks(gc.ctx, keys[:w.held_chunks], [wi.payloads(i) for i in range(w.held_chunks)])
    say(f"case: random call sequence seed={seed}")
    reqs = {r: Req(r, gc) for r in (101, 102, 103)}
    bound = set()
    seen = {"exposed": 0, "fallback": 0, "refused": 0}
    # the three requests share the destination pools, so only one may hold
    # an exposed image at a time: keep one request at a time past bind
    try:
        for step in range(400):
            # mostly act on the bound request, so that restores do run to the end
            pick = sorted(bound) if bound and rng.random() < 0.7 else sorted(reqs)
            r = reqs[rng.choice(pick)]
            op = rng.choices(["probe", "bind", "window", "bad_window", "invalidate", "mark", "commit", "end",
                              "running"], weights=[3, 3, 12, 1, 0.5, 0.5, 3, 1, 3])[0]

            def expect(code, fn):
                try:
                    fn()
                    got = bsr.BSR_OK
                except bsr.BsrError as e:
                    got = e.code
                assert got == code, f"step {step} {op} on {r.rid} (state {r.state}): {got} != {code}"
                if got != bsr.BSR_OK:
                    seen["refused"] += 1
                return got == bsr.BSR_OK

            if op == "probe":
                if r.state in ("bound", "failed"):
                    expect(bsr.BSR_E_STATE, lambda: gc.probe(r.rid))
                else:
                    n = gc.probe(r.rid)[0]
                    assert n == (0 if r.force_local else n_full)
                    r.n, r.state, r.next, r.marked = n, "probed", 0, False
            elif op == "bind":
                if r.state in ("bound", "failed"):
                    expect(bsr.BSR_E_STATE, lambda: r.sess.bind(r.rid, r.n, gc.dsts()))
                elif r.state != "probed":
                    expect(bsr.BSR_E_STATE, lambda: r.sess.bind(r.rid, r.n, gc.dsts()))
                elif bound:
                    # one request at a time owns the shared pools in this test: the
                    # budget would admit a second ring, so the refusal is ours
                    continue
                else:
                    torch.cuda.synchronize()
                    expect(bsr.BSR_OK, lambda: r.sess.bind(r.rid, r.n, gc.dsts()))
                    r.state = "bound"
                    bound.add(r.rid)
            elif op in ("window", "bad_window"):
                first = r.next if op == "window" else r.next + rng.choice([1, W, -1])
                cnt = min(W, max(1, r.n - first)) if op == "window" else rng.randint(1, W)
                if r.state == "failed":
                    expect(bsr.BSR_E_STATE, lambda: bsr.bsr_restore_window(gc.ctx, r.rid, max(0, first), cnt))
                elif r.state != "bound":
                    expect(bsr.BSR_E_STATE, lambda: bsr.bsr_restore_window(gc.ctx, r.rid, max(0, first), cnt))
                elif op == "window" and r.next < r.n:
                    expect(bsr.BSR_OK, lambda: bsr.bsr_restore_window(gc.ctx, r.rid, first, cnt))
                    r.next += cnt
                elif op == "window":
                    # the whole prefix is restored already: any further window lies beyond it
                    expect(bsr.BSR_E_ARG, lambda: bsr.bsr_restore_window(gc.ctx, r.rid, r.next, 1))
                else:
                    f = max(0, first)
                    code = bsr.BSR_E_STATE if f != r.next else bsr.BSR_E_ARG
                    if f == r.next and f + cnt <= r.n:
                        continue   # that would be a valid window after all
                    expect(code, lambda: bsr.bsr_restore_window(gc.ctx, r.rid, f, cnt))
            elif op == "invalidate":
                if r.state in ("bound", "failed"):
                    expect(bsr.BSR_OK, lambda: bsr.bsr_invalidate(gc.ctx, r.rid, bsr.BSR_FAIL_ABORT))
                    r.state = "failed"
                else:
                    expect(bsr.BSR_E_STATE, lambda: bsr.bsr_invalidate(gc.ctx, r.rid, bsr.BSR_FAIL_ABORT))
            elif op == "mark":
                if r.state in ("bound", "failed"):
                    expect(bsr.BSR_OK, lambda: bsr.bsr_mark_group_invalid(gc.ctx, r.rid, 0))
                    r.marked = True
                else:
                    expect(bsr.BSR_E_STATE, lambda: bsr.bsr_mark_group_invalid(gc.ctx, r.rid, 0))
            elif op == "commit":
                if r.state not in ("bound", "failed"):
                    expect(bsr.BSR_E_STATE, lambda: bsr.bsr_commit(gc.ctx, r.rid))
                    continue
                out = r.sess.commit(r.rid)
                complete = r.state == "bound" and r.next == r.n and not r.marked
                if complete and r.n:
                    assert out.exposed_tokens == r.n * w.chunk_tokens and out.fallback == 0
                    np.testing.assert_array_equal(gc.pool_host(0), case.pools[0])
                    np.testing.assert_array_equal(gc.valid_host(0), case.valid[0])
                    assert ref.exposed_tokens == r.n * w.chunk_tokens
                elif r.n:
                    assert out.exposed_tokens == 0 and out.fallback == 1
                    adv = wi.block_tables[0][:oracle.request_blocks(r.n, w.chunk_tokens, 16)]
                    assert not gc.valid_host(0)[adv].any()
                else:
                    assert out.exposed_tokens == 0
                    assert out.fallback == (0 if complete else 1)
                if out.fallback:
                    r.force_local = True      # a fallback sets the marker; success keeps it as it was
                if out.fallback:
                    seen["fallback"] += 1
                elif out.exposed_tokens:
                    seen["exposed"] += 1
                r.state = "done"
                bound.discard(r.rid)
            elif op == "end":
                expect(bsr.BSR_OK, lambda: bsr.bsr_request_end(gc.ctx, r.rid))
                if r.state in ("bound", "failed") and r.n:
                    adv = wi.block_tables[0][:oracle.request_blocks(r.n, w.chunk_tokens, 16)]
                    assert not gc.valid_host(0)[adv].any()      # torn down unexposed
                r.state, r.force_local = "new", False
                bound.discard(r.rid)
            elif op == "running":
                expect(bsr.BSR_OK, lambda: bsr.bsr_request_running(gc.ctx, r.rid))
                r.force_local = False
            a = bsr.bsr_admission_get(gc.ctx)
            assert a["n_bound"] == len(bound) and a["bound_staging_bytes"] == len(bound) * W * slot
        for r in reqs.values():
            bsr.bsr_request_end(gc.ctx, r.rid)
        assert bsr.bsr_admission_get(gc.ctx)["n_bound"] == 0
        say(f"outcomes: {seen}")
        assert seen["exposed"] >= 1 and seen["fallback"] >= 1 and seen["refused"] >= 1, seen
    finally:
        gc.close()
