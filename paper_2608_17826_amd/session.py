"""Restore-session helper over the C ABI, with torch as the memory plumbing.

Allocates the W-slot staging ring (exactly ``bsr_staging_bytes`` bytes) and
the device status block with torch, creates two default-priority streams
(copy, compute), and drives one request at a time through bind ->
restore_window x K -> commit.  Requests bound together under a context's
admission budget each use a session of their own (their own ring, status
block and streams).  All restore work runs inside libbsr.so.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np
import torch

from . import bsr


@dataclass
class Outcome:
    exposed_tokens: int
    fallback: int
    window_errors: List[Tuple[int, int]] = field(default_factory=list)  # (first_chunk, code)
    stats: dict = field(default_factory=dict)
    status: dict = field(default_factory=dict)


def group_dsts(block_tables: Sequence[torch.Tensor], tensor_bases: Sequence[torch.Tensor],
               valid: Sequence[torch.Tensor], pool_blocks: Sequence[int]) -> List[bsr.bsr_group_dst]:
    return [bsr.group_dst(bt.data_ptr(), tb.data_ptr(), v.data_ptr(), bt.numel(), pb)
            for bt, tb, v, pb in zip(block_tables, tensor_bases, valid, pool_blocks)]


def status_dict(raw: torch.Tensor) -> dict:
    h = raw.cpu().numpy()
    s = bsr.bsr_dev_status.from_buffer_copy(h.tobytes())
    return {"fail": s.fail, "first_failed_chunk": s.first_failed_chunk, "q": list(s.q),
            "exposed_tokens": s.exposed_tokens, "fallback": s.fallback, "phase": s.phase}


class RestoreSession:
    """One ring (exactly the plan's staging bytes), one status block, two streams.

    With a bounded window the ring is W x chunk bytes and allocated once; in
    whole-plan mode (W = 0) it is sized per request, n_hit x chunk bytes.
    """

    def __init__(self, ctx: bsr.Ctx, device: str = "cuda:0"):
        self.ctx = ctx
        self.device = torch.device(device)
        self.staging = None
        self.staging_bytes = 0
        if ctx.window_chunks:
            self._ring(bsr.bsr_plan_staging_bytes(ctx, 0))
        self.status = torch.zeros(64, dtype=torch.uint8, device=self.device)
        self.copy_stream = torch.cuda.Stream(device=self.device)
        self.compute_stream = torch.cuda.Stream(device=self.device)

    def release_ring(self) -> None:
        """Drop the ring; the next bind allocates it again."""
        self.staging = None
        self.staging_bytes = 0

    def _ring(self, nbytes: int) -> None:
        if self.staging is None or self.staging.numel() != nbytes:
            self.staging = None
            self.staging = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
        self.staging_bytes = nbytes

    def bind(self, request_id: int, n_hit: int, dsts: Sequence[bsr.bsr_group_dst]) -> None:
        self._ring(bsr.bsr_plan_staging_bytes(self.ctx, n_hit))
        bsr.bsr_request_bind(self.ctx, request_id, n_hit, dsts, self.staging.data_ptr(),
                             self.staging_bytes, self.status.data_ptr(),
                             self.copy_stream.cuda_stream, self.compute_stream.cuda_stream)

    def commit(self, request_id: int, window_errors=None) -> Outcome:
        exposed, fallback = bsr.bsr_commit(self.ctx, request_id)
        return Outcome(exposed, fallback, list(window_errors or []), bsr.bsr_request_stats(self.ctx, request_id),
                       status_dict(self.status))

    def windows(self, n_hit: int) -> List[Tuple[int, int]]:
        """The plan of a request not bound yet (the library's own plan, once
        bound, comes from ``next_windows``)."""
        W = self.ctx.window_chunks or max(1, n_hit)
        return [(s, min(W, n_hit - s)) for s in range(0, n_hit, W)]

    def next_windows(self, request_id: int):
        """The bound request's remaining windows, as the library plans them:
        each is asked for after the one before has been restored."""
        while True:
            first, n = bsr.bsr_next_window(self.ctx, request_id)
            if n == 0:
                return
            yield first, n

    def restore(self, request_id: int, n_hit: int, dsts: Sequence[bsr.bsr_group_dst],
                plan: Optional[Sequence[Tuple[int, int]]] = None, abort_after_windows: Optional[int] = None,
                before_commit=None, after_window=None, after_bind=None) -> Outcome:
        """bind, every window of the plan, then commit (or invalidate + commit).

        ``after_bind()`` and ``after_window(j)`` (once window j has been
        enqueued) are the caller's hooks, e.g. a measurement, or an engine
        reporting a group invalid mid-restore.
        """
        torch.cuda.current_stream(self.device).synchronize()  # inputs written by torch are ready
        self.bind(request_id, n_hit, dsts)
        if after_bind is not None:
            after_bind()
        errors = []
        for j, (first, n) in enumerate(plan if plan is not None else self.next_windows(request_id)):
            try:
                bsr.bsr_restore_window(self.ctx, request_id, first, n)
            except bsr.BsrError as e:
                errors.append((first, e.code))
                break
            if after_window is not None:
                after_window(j)
            if abort_after_windows is not None and j + 1 >= abort_after_windows:
                bsr.bsr_invalidate(self.ctx, request_id, bsr.BSR_FAIL_ABORT)
                break
        if before_commit is not None:
            before_commit()
        return self.commit(request_id, errors)
