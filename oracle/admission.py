"""Deadline-aware admission: an AIMD loop on the per-frame latency.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).  The library's
``mtn_admission_*`` controller is compared with this model call by call,
bit-exactly (cap, admitted count, counters, every admit/reject decision).

What it follows (Metronome, arXiv 2607.02640, §4.2): beyond the schedulable
concurrency N*, one more session degrades every session, so the controller
admits up to N* and sheds the rest.  N* is not set by hand; an online,
model-free AIMD loop discovers it from the measured per-frame latency: the
admission cap is lowered multiplicatively when latency nears a target
fraction of the frame budget, raised additively to probe when there is
headroom, and an arrival beyond the cap gets a clean overload rejection.
§5 ("Admission converges only with bounded state") states the claim the
pins check: with bounded KV the latency is a monotone signal of the load and
the loop settles near N*; when the signal stays flat while resident state
grows (unbounded KV), the same loop admits every arrival.

Readings, since the paper gives the rule but not its
constants or edge cases:

* "nears the target": the tick's latency is at or above ``target_ms``;
  the caller chooses the target as a fraction of the frame budget.
* The cut is relative to the load that produced the latency:
  cap <- max(min_cap, min(cap, floor(backoff * admitted))).  It never raises
  the cap and never evicts an admitted session.
* After a cut, ``hold_ticks`` observations pass without a decision, so the
  next decision sees the effect of the last one.
* The additive probe (cap <- min(max_cap, cap + increase)) happens only when
  demand pressed against the cap since the previous observation (an offer
  was rejected, or the admitted count reached the cap); an idle cap does not
  grow without bound.

Parity status: pinned (tests/test_admission.py) by closed forms -- linear
growth under headroom, a single cut's value, the hold -- and by the paper's
two claims as properties of latency models: convergence into [N*, N* + step)
on a monotone signal, and admission of every arrival on a flat one.
"""
from __future__ import annotations

import math
from dataclasses import dataclass


@dataclass
class AimdAdmission:
    target_ms: float
    backoff: float
    increase: int
    initial_cap: int
    min_cap: int
    max_cap: int
    hold_ticks: int

    def __post_init__(self):
        if not (self.target_ms > 0 and math.isfinite(self.target_ms)):
            raise ValueError("target_ms")
        if not (0.0 < self.backoff < 1.0):
            raise ValueError("backoff")
        if (self.increase < 1 or self.min_cap < 1 or self.initial_cap < self.min_cap
                or self.max_cap < self.initial_cap or self.hold_ticks < 0):
            raise ValueError("caps / steps")
        self.cap = self.initial_cap
        self.admitted = 0
        self.hold = 0
        self.offered = 0
        self.rejected = 0
        self.ticks = 0
        self.decreases = 0
        self.increases = 0
        self._demand_at_cap = False

    # an arriving session: admitted while under the cap, else rejected
    def offer(self) -> bool:
        self.offered += 1
        if self.admitted < self.cap:
            self.admitted += 1
            if self.admitted == self.cap:
                self._demand_at_cap = True
            return True
        self.rejected += 1
        self._demand_at_cap = True
        return False

    def release(self) -> None:
        if self.admitted == 0:
            raise RuntimeError("no admitted session to release")
        self.admitted -= 1

    # one tick's measured latency
    def observe(self, tick_ms: float) -> None:
        if not (tick_ms >= 0 and math.isfinite(tick_ms)):
            raise ValueError("tick_ms")
        self.ticks += 1
        demand = self._demand_at_cap
        self._demand_at_cap = False
        if self.hold > 0:
            self.hold -= 1
            return
        if tick_ms >= self.target_ms:
            # multiplicative decrease near the target
            self.cap = max(self.min_cap, min(self.cap, math.floor(self.backoff * self.admitted)))
            self.hold = self.hold_ticks
            self.decreases += 1
        elif demand:
            # additive increase: probe for headroom
            self.cap = min(self.max_cap, self.cap + self.increase)
            self.increases += 1

    def state(self) -> dict:
        return dict(cap=self.cap, admitted=self.admitted, hold=self.hold, offered=self.offered,
                    rejected=self.rejected, ticks=self.ticks, decreases=self.decreases,
                    increases=self.increases)
