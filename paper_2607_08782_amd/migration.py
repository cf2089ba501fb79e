"""Computation-overlapped expert migration on one GPU (Sec. V-B).

When the placement changes, the experts that become local must be copied in
while the layer keeps serving.  The paper schedules those transfers only in
the computation phase of a step (the expert FFNs), never across the
all-to-all exchanges, and sizes them from the predicted length of that phase
so they finish before the next exchange.  This module does the one-GPU part:

* ``ExpertStore``: every expert's weights in pinned host memory, standing in
  for the peer GPUs a migrated expert comes from (on a node the copy would be
  a peer transfer over xGMI; here it is a host-to-device copy on the DMA
  engines, which use no compute units).
* ``Migrator``: double-buffered slots.  The experts of the current placement
  stay in their device buffers while the incoming ones are copied into spare
  buffers on a second stream (default priority), chunk by chunk, only inside
  the FFN window of a step: the migration stream waits for an event recorded
  where the window opens, gets at most the bytes the window is predicted to
  hide, and the compute stream waits for the chunks' completion event where
  the window closes (the point the all-to-all of the combine would start).
  When every chunk has landed, ``switch`` re-points the layer's weight table.
* The bytes a window can hide are predicted from the last window: the copies
  compete with the FFN for memory bandwidth (the FFN slows down and the copy
  rate drops while both run), so the next window gets the bytes the last
  window's copy rate moves in the window's target length, times a margin.
  The target is the computation's length without copies (``window_ms``, set
  by the caller from f_comp or a measurement): a window sized from the FFN
  time with copies would grow with the slowdown it causes.  The first window
  starts from the caller's estimate (f_comp of the step's load at the
  uncontended copy rate).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from . import moe


class ExpertStore:
    """All experts' (w13, w2) in pinned host memory."""

    def __init__(self, w13: Sequence[torch.Tensor], w2: Sequence[torch.Tensor]):
        self.w13 = [t.detach().to("cpu").pin_memory() for t in w13]
        self.w2 = [t.detach().to("cpu").pin_memory() for t in w2]

    def nbytes(self, e: int) -> int:
        return self.w13[e].numel() * self.w13[e].element_size() + self.w2[e].numel() * self.w2[e].element_size()


@dataclass
class _Chunk:
    expert: int
    which: int          # 0: w13, 1: w2
    start: int          # first row
    stop: int
    nbytes: int


@dataclass
class MigrationStats:
    windows: int = 0
    bytes: int = 0
    stall_ms: List[float] = field(default_factory=list)
    budgets: List[int] = field(default_factory=list)


# share of the last window's FFN time the next window's copies are sized to fill
WINDOW_MARGIN = 0.85


class Migrator:
    """Double-buffered expert slots of one GPU and the chunked copy schedule."""

    def __init__(self, store: ExpertStore, placement: np.ndarray, dev: int, spare: int,
                 device="cuda", chunk_bytes: int = 8 << 20):
        self.store = store
        self.dev = dev
        self.device = device
        self.chunk_bytes = int(chunk_bytes)
        self.placement = np.ascontiguousarray(placement, dtype=np.uint8)
        local = [int(e) for e in np.nonzero(self.placement[:, dev])[0]]
        n_buf = len(local) + spare
        e0 = local[0] if local else 0
        self.buf13 = [torch.empty_like(store.w13[e0], device=device) for _ in range(n_buf)]
        self.buf2 = [torch.empty_like(store.w2[e0], device=device) for _ in range(n_buf)]
        self.holds: Dict[int, int] = {}              # expert -> buffer
        for b, e in enumerate(local):
            self.buf13[b].copy_(store.w13[e])
            self.buf2[b].copy_(store.w2[e])
            self.holds[e] = b
        torch.cuda.synchronize()
        self.stream = torch.cuda.Stream(device=device)
        self.pending: List[_Chunk] = []
        self.target: Optional[np.ndarray] = None
        self.incoming: Dict[int, int] = {}
        self.stats = MigrationStats()
        self.budget_bytes = self.chunk_bytes     # bytes the next window may take
        self.window_ms: Optional[float] = None   # the computation's length without copies
        self._sent = 0

    # -- current weights -------------------------------------------------------
    def weights(self, placement: Optional[np.ndarray] = None):
        """(w13 list, w2 list) of the local slots of `placement` (ascending expert id)."""
        pl = self.placement if placement is None else placement
        local = [int(e) for e in np.nonzero(pl[:, self.dev])[0]]
        hold = dict(self.holds)
        hold.update(self.incoming)
        return [self.buf13[hold[e]] for e in local], [self.buf2[hold[e]] for e in local]

    # -- planning -----------------------------------------------------------------
    def plan(self, new_placement: np.ndarray) -> int:
        """Queue the copies that make `new_placement` local here; returns bytes to move."""
        new_placement = np.ascontiguousarray(new_placement, dtype=np.uint8)
        want = [int(e) for e in np.nonzero(new_placement[:, self.dev])[0]]
        keep = set(e for e in want if e in self.holds)
        free = [b for b in range(len(self.buf13)) if b not in self.holds.values()]
        need = [e for e in want if e not in keep]
        if len(need) > len(free):
            raise ValueError("%d experts to bring in but only %d spare buffers" % (len(need), len(free)))
        self.target = new_placement
        self.incoming = {}
        self.pending = []
        total = 0
        for e, b in zip(need, free):
            self.incoming[e] = b
            for which, src in ((0, self.store.w13[e]), (1, self.store.w2[e])):
                row_bytes = src[0].numel() * src.element_size()
                rows = max(1, self.chunk_bytes // row_bytes)
                for r0 in range(0, src.shape[0], rows):
                    r1 = min(src.shape[0], r0 + rows)
                    self.pending.append(_Chunk(e, which, r0, r1, (r1 - r0) * row_bytes))
                    total += (r1 - r0) * row_bytes
        return total

    # -- one computation window -----------------------------------------------------
    def window(self, opened: torch.cuda.Event, budget_bytes: int) -> Optional[torch.cuda.Event]:
        """Issue up to `budget_bytes` of pending chunks after `opened`; returns the
        event the compute stream must wait for where the window closes."""
        if not self.pending:
            return None
        self.stream.wait_event(opened)
        sent = 0
        self.stats.budgets.append(int(budget_bytes))
        with torch.cuda.stream(self.stream):
            while self.pending and (sent == 0 or sent + self.pending[0].nbytes <= budget_bytes):
                c = self.pending.pop(0)
                b = self.incoming[c.expert]
                dst = (self.buf13 if c.which == 0 else self.buf2)[b]
                src = (self.store.w13 if c.which == 0 else self.store.w2)[c.expert]
                dst[c.start:c.stop].copy_(src[c.start:c.stop], non_blocking=True)
                sent += c.nbytes
        done = torch.cuda.Event(enable_timing=True)
        done.record(self.stream)
        self.stats.windows += 1
        self.stats.bytes += sent
        self._sent = sent
        return done

    def empty_window(self, opened: torch.cuda.Event) -> torch.cuda.Event:
        """The window's stream join with no copy in it: what a window costs the compute
        stream by itself (an event on the migration stream after `opened`)."""
        self.stream.wait_event(opened)
        done = torch.cuda.Event(enable_timing=True)
        done.record(self.stream)
        return done

    def observe(self, ffn_ms: float, copy_ms: float):
        """Size the next window from the last one: its copies moved `_sent` bytes in
        `copy_ms` while the FFN took `ffn_ms`; the next window gets what that rate
        moves in the window's target length (`window_ms`, else `ffn_ms`)."""
        if self._sent <= 0 or copy_ms <= 0:
            return
        rate = self._sent / copy_ms                          # bytes per ms under contention
        target = self.window_ms if self.window_ms else ffn_ms
        self.budget_bytes = max(self.chunk_bytes, int(WINDOW_MARGIN * rate * target))

    @property
    def finished(self) -> bool:
        return self.target is not None and not self.pending

    def switch(self):
        """Adopt the target placement (every chunk must have been issued; the caller's
        stream has already waited for the last window's event)."""
        if not self.finished:
            raise RuntimeError("migration still has pending chunks")
        want = set(int(e) for e in np.nonzero(self.target[:, self.dev])[0])
        holds = {e: b for e, b in self.holds.items() if e in want}
        holds.update(self.incoming)
        self.holds = holds
        self.incoming = {}
        self.placement = self.target
        self.target = None
        return self.weights()


def measure_h2d_rate(nbytes: int = 64 << 20, device="cuda") -> float:
    """Bytes per microsecond of a pinned host-to-device copy on a side stream."""
    src = torch.empty(nbytes, dtype=torch.uint8).pin_memory()
    dst = torch.empty(nbytes, dtype=torch.uint8, device=device)
    s = torch.cuda.Stream(device=device)
    with torch.cuda.stream(s):
        dst.copy_(src, non_blocking=True)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(s)
        dst.copy_(src, non_blocking=True)
        b.record(s)
    b.synchronize()
    return nbytes / (a.elapsed_time(b) * 1e3)


def run_step(share, mig: Optional[Migrator], budget_bytes: Optional[int] = None,
             timing: Optional[dict] = None, empty: bool = False):
    """One layer step with the FFN window open to migration; returns the time (ms) the
    compute stream waited at the window's close for the copies (None if no copy).
    The window takes `budget_bytes`, or the migrator's own prediction from the last
    window (which this step then updates).  With `timing`, the FFN window's own
    duration (ms) is appended to timing["ffn"] and the copies' to timing["copy"].
    empty=True opens and closes the window with no copy (the join's own cost)."""
    cur = torch.cuda.current_stream()
    share.route()
    moe.moe_expert_histogram(share.topk_idx, share.E, counts=share.counts, coact=share.coact)
    share.package()
    opened = torch.cuda.Event(enable_timing=True)
    opened.record(cur)
    # the window's computation is enqueued first: the copies only wait for `opened`
    # on the device, and issuing them (one host call per chunk) must not hold back
    # the launch of the computation they hide behind
    share.routed_ffn(fused=False)
    share._shared_ffn()          # nothing when the shared experts share the routed call
    stall = None
    ffn_end = torch.cuda.Event(enable_timing=True)
    ffn_end.record(cur)
    adaptive = budget_bytes is None and not empty
    if mig is not None and adaptive:
        budget_bytes = mig.budget_bytes
    if mig is not None and empty:
        done = mig.empty_window(opened)
    else:
        done = mig.window(opened, budget_bytes) if mig is not None else None
    if done is not None:
        cur.wait_event(done)                 # the exchange after the FFN must not overlap copies
        after = torch.cuda.Event(enable_timing=True)
        after.record(cur)
        after.synchronize()
        stall = ffn_end.elapsed_time(after)
        copy_ms = opened.elapsed_time(done)
        if adaptive:
            mig.observe(opened.elapsed_time(ffn_end), copy_ms)
        if timing is not None:
            timing.setdefault("copy", []).append(copy_ms)
    if timing is not None:
        ffn_end.synchronize()
        timing.setdefault("ffn", []).append(opened.elapsed_time(ffn_end))
    share.combine()
    return stall
