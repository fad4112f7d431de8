"""Independent pure-Python model of the pool / block-table / ring index map.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).  The library's host
planner is compared with this model bit-exactly: block tables, the physical
(block, offset) of every planned token, evicted ranges, error codes and pool
counters.

What it follows (Metronome, arXiv 2607.02640):

* App. A "Sink half": a windowed session pins its first ceil(S / block)
  blocks, which are never freed while the session lives, and the admission
  cap counts them, so pool sizing stays exact.
* App. A "Window half": blocks wholly behind the window are not resident.
  Here a windowed session owns a fixed ring of R slots (R a multiple of the
  block size) after its sink blocks; a new position p >= S lands in ring slot
  (p - S) mod R and overwrites a position that has already left the window.
  The bound the paper states (sinks plus the last W tokens) is the same; the
  blocks are recycled inside the session instead of going back to the pool.
* §3.1 Eq. 1: under the unbounded policy the pool fills linearly in time; the
  tests compare the exhaustion frame of this model with the equation.

Reading: during a chunk of C tokens the query at the
first new position still needs W - 1 older window tokens while the chunk's C
tokens are being written, so the ring holds R = roundup(W + C_max - 1, block)
slots.  Positions S .. block-1 of the last sink block are never written (the
pinned blocks hold sink positions only).

Block assignment is lazy and lowest-free-first, in plan order (sequences in
the order given, positions increasing), the first time a logical block is
written.  Session ids are handed out lowest-free-first.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple
import heapq

# Status codes, identical in meaning to the C-ABI's.
OK = 0
ERR_INVALID_ARG = -1
ERR_BAD_SESSION = -2
ERR_CHUNK_TOO_LARGE = -3
ERR_NO_SESSION_SLOT = -4
ERR_POOL_EXHAUSTED = -5
ERR_SESSION_FULL = -6
ERR_BAD_STATE = -8


class IndexError_(Exception):
    def __init__(self, code: int, msg: str = ""):
        super().__init__(f"{code}: {msg}")
        self.code = code


def ceil_div(a: int, b: int) -> int:
    return -(-a // b)


def round_up(a: int, b: int) -> int:
    return ceil_div(a, b) * b


@dataclass
class _Session:
    length: int
    row: List[int]


@dataclass
class PlannedToken:
    sid: int
    pos: int
    block: int   # physical block id
    offset: int  # slot inside the block


class IndexModel:
    def __init__(self, n_blocks: int, block_size: int, n_sink: int,
                 window: Optional[int], max_chunk: int, max_sessions: int,
                 max_len: Optional[int] = None):
        self.n_blocks = n_blocks
        self.bs = block_size
        self.window = window
        self.max_chunk = max_chunk
        self.max_sessions = max_sessions
        if window is None:                      # unbounded (vanilla) policy
            if max_len is None:
                raise ValueError("unbounded policy needs max_len")
            self.n_sink = 0
            self.n_sink_blocks = 0
            self.ring = round_up(max_len, block_size)
            self.max_len = max_len
        else:
            self.n_sink = n_sink
            self.n_sink_blocks = ceil_div(n_sink, block_size)
            self.ring = round_up(window + max_chunk - 1, block_size)
            self.max_len = None
        self.row_len = self.n_sink_blocks + self.ring // block_size
        self.free: List[int] = list(range(n_blocks))  # min-heap
        heapq.heapify(self.free)
        self.sessions: Dict[int, _Session] = {}
        self.reserved = 0
        self.plan: Optional[List[Tuple[int, int]]] = None
        self.plan_tokens: List[PlannedToken] = []
        self.plan_evicted: List[Tuple[int, int]] = []
        self.plan_fresh: List[Tuple[int, int]] = []   # (sid, logical block) the plan assigned

    # -- slot map ----------------------------------------------------------
    def logical_slot(self, pos: int) -> Tuple[int, int]:
        """(logical block index in the session's row, offset) of a position."""
        if pos < self.n_sink:
            return pos // self.bs, pos % self.bs
        sigma = (pos - self.n_sink) % self.ring
        return self.n_sink_blocks + sigma // self.bs, sigma % self.bs

    # -- sessions ----------------------------------------------------------
    def open(self) -> int:
        sid = next((i for i in range(self.max_sessions)
                    if i not in self.sessions), None)
        if sid is None:
            raise IndexError_(ERR_NO_SESSION_SLOT, "no free session slot")
        if self.window is not None:
            if self.reserved + self.row_len > self.n_blocks:
                raise IndexError_(ERR_POOL_EXHAUSTED, "reservation exceeds pool")
            self.reserved += self.row_len
        self.sessions[sid] = _Session(0, [-1] * self.row_len)
        return sid

    def close(self, sid: int) -> None:
        if self.plan is not None:
            raise IndexError_(ERR_BAD_STATE, "plan open")
        s = self.sessions.get(sid)
        if s is None:
            raise IndexError_(ERR_BAD_SESSION, "not open")
        for b in s.row:
            if b >= 0:
                heapq.heappush(self.free, b)
        if self.window is not None:
            self.reserved -= self.row_len
        del self.sessions[sid]

    # -- planning ----------------------------------------------------------
    def plan_begin(self, sids: Sequence[int], n_tok: Sequence[int]) -> None:
        if self.plan is not None:
            raise IndexError_(ERR_BAD_STATE, "plan already open")
        if len(sids) < 1 or len(sids) != len(n_tok) or len(sids) > self.max_sessions:
            raise IndexError_(ERR_INVALID_ARG, "bad sequence count")
        seen = set()
        for sid, n in zip(sids, n_tok):
            if sid not in self.sessions:
                raise IndexError_(ERR_BAD_SESSION, f"sid {sid}")
            if sid in seen:
                raise IndexError_(ERR_INVALID_ARG, "duplicate sid")
            seen.add(sid)
            if n < 1:
                raise IndexError_(ERR_INVALID_ARG, "n_tok < 1")
            if n > self.max_chunk:
                raise IndexError_(ERR_CHUNK_TOO_LARGE, "n_tok > max_chunk")
            if self.max_len is not None and self.sessions[sid].length + n > self.max_len:
                raise IndexError_(ERR_SESSION_FULL, "past max_len")
        # Count the blocks this plan needs first, so that a failure changes
        # nothing; then assign them lowest-free-first in plan order.
        need = 0
        for sid, n in zip(sids, n_tok):
            L = self.sessions[sid].length
            row = self.sessions[sid].row
            fresh = {self.logical_slot(p)[0] for p in range(L, L + n)}
            need += sum(1 for lb in fresh if row[lb] < 0)
        if need > len(self.free):
            raise IndexError_(ERR_POOL_EXHAUSTED, "pool exhausted")
        toks: List[PlannedToken] = []
        fresh: List[Tuple[int, int]] = []
        for sid, n in zip(sids, n_tok):
            L = self.sessions[sid].length
            row = self.sessions[sid].row
            for p in range(L, L + n):
                lb, off = self.logical_slot(p)
                if row[lb] < 0:
                    row[lb] = heapq.heappop(self.free)
                    fresh.append((sid, lb))
                toks.append(PlannedToken(sid, p, row[lb], off))
        self.plan_fresh = fresh
        self.plan = list(zip(sids, n_tok))
        self.plan_tokens = toks
        ev = []
        for sid, n in self.plan:
            L = self.sessions[sid].length
            if self.window is None:
                ev.append((0, 0))
            else:
                lo = max(self.n_sink, L - self.window)
                ev.append((lo, max(lo, L + n - self.window)))
        self.plan_evicted = ev

    def plan_commit(self) -> None:
        if self.plan is None:
            raise IndexError_(ERR_BAD_STATE, "no plan")
        for sid, n in self.plan:
            self.sessions[sid].length += n
        self.plan = None
        self.plan_fresh = []

    def plan_abort(self) -> None:
        """Abandon the open plan: the blocks it assigned go back to the free
        set, so the pool (and every later lowest-free choice) is as if the
        plan had never begun; lengths do not move."""
        if self.plan is None:
            raise IndexError_(ERR_BAD_STATE, "no plan")
        for sid, lb in reversed(self.plan_fresh):
            row = self.sessions[sid].row
            heapq.heappush(self.free, row[lb])
            row[lb] = -1
        self.plan = None
        self.plan_fresh = []

    # -- observability -----------------------------------------------------
    def assigned(self) -> int:
        return sum(1 for s in self.sessions.values() for b in s.row if b >= 0)

    def reserved_blocks(self) -> int:
        return self.reserved if self.window is not None else self.assigned()

    def block_table(self, sid: int) -> List[int]:
        return list(self.sessions[sid].row)

    def resident_slots(self, sid: int) -> Dict[int, Tuple[int, int]]:
        """Physical (block, offset) of every retained position of a session."""
        s = self.sessions[sid]
        L = s.length
        out = {}
        for p in range(L):
            if self.window is None or p < self.n_sink or p >= L - self.window:
                lb, off = self.logical_slot(p)
                out[p] = (s.row[lb], off)
        return out
