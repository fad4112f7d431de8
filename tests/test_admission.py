"""Deadline-aware admission (§4.2): pins of the AIMD oracle, and bit-exact
parity of the library's host-only controller (mtn_admission_*) with it."""
import math
import random

import pytest
from hypothesis import given, settings, strategies as st

from oracle.admission import AimdAdmission

CFG = dict(target_ms=450.0, backoff=0.8, increase=8, initial_cap=16, min_cap=1, max_cap=1024,
           hold_ticks=2)


def _ramp(ctrl, latency_of, arrivals_per_tick, ticks, offered_total=10 ** 9):
    """Open-system ramp: each tick, offer the tick's arrivals, then observe
    the latency the admitted load produces.  Returns the admitted series."""
    offered = 0
    series = []
    for _ in range(ticks):
        for _ in range(arrivals_per_tick):
            if offered < offered_total:
                ctrl.offer()
                offered += 1
        ctrl.observe(latency_of(ctrl.admitted))
        series.append(ctrl.admitted)
    return series


# ---- closed forms --------------------------------------------------------

@pytest.mark.parametrize("c0,a,cmax,k", [(16, 8, 1024, 10), (5, 1, 9, 7), (1, 3, 1000, 50)])
def test_additive_growth_under_headroom(c0, a, cmax, k):
    """Demand pressing every tick, latency always below target: the cap grows
    by exactly `increase` per tick up to max_cap."""
    c = AimdAdmission(**{**CFG, "initial_cap": c0, "increase": a, "max_cap": cmax})
    for i in range(1, k + 1):
        while c.offer():
            pass
        c.observe(0.0)
        assert c.cap == min(cmax, c0 + i * a)


@pytest.mark.parametrize("n,beta,cap,mn,expect", [(100, 0.8, 120, 1, 80), (100, 0.5, 40, 1, 40),
                                                  (3, 0.3, 3, 2, 2), (7, 0.75, 7, 1, 5)])
def test_single_cut(n, beta, cap, mn, expect):
    """Latency at the target with N admitted: cap = max(min_cap, min(cap,
    floor(beta * N))) -- never raised, never below min_cap."""
    c = AimdAdmission(**{**CFG, "backoff": beta, "initial_cap": max(cap, n), "min_cap": mn})
    for _ in range(n):
        assert c.offer()
    c.cap = cap  # the cap may already sit below the admitted count
    c.observe(CFG["target_ms"])
    assert c.cap == expect == max(mn, min(cap, math.floor(beta * n)))
    assert c.admitted == n  # nothing evicted


def test_hold_after_cut():
    c = AimdAdmission(**{**CFG, "hold_ticks": 3, "initial_cap": 50})
    for _ in range(50):
        c.offer()
    c.observe(1e9)
    cap = c.cap
    for lat in (1e9, 0.0, 1e9):   # neither a second cut nor a probe
        c.offer()
        c.observe(lat)
        assert c.cap == cap
    c.offer()
    c.observe(0.0)                 # the hold is over: the probe resumes
    assert c.cap == cap + CFG["increase"]


def test_idle_cap_does_not_grow():
    c = AimdAdmission(**CFG)
    for _ in range(3):
        c.offer()
    for _ in range(20):
        c.observe(0.0)
    assert c.cap == CFG["initial_cap"] and c.increases == 0


@settings(max_examples=60, deadline=None)
@given(st.lists(st.tuples(st.sampled_from("oro"), st.floats(0, 900)), max_size=300))
def test_admission_invariants(ops):
    c = AimdAdmission(**CFG)
    admits = 0
    for op, lat in ops:
        if op == "o":
            before = (c.admitted, c.cap)
            if c.offer():
                admits += 1
                assert before[0] < before[1]
            else:
                assert before[0] >= before[1]
        elif op == "r" and c.admitted:
            c.release()
        else:
            c.observe(lat)
        assert c.min_cap <= c.cap <= c.max_cap
    assert c.offered == admits + c.rejected


# ---- the paper's two claims as properties of latency models --------------

@pytest.mark.parametrize("a0,b,step,rate", [(20.0, 1.21, 8, 12), (5.0, 0.7, 4, 4), (100.0, 3.3, 1, 2)])
def test_converges_on_a_monotone_signal(a0, b, step, rate):
    """Bounded KV: the tick grows with the admitted load, L(N) = a0 + b N.
    N* = the smallest N with L(N) >= target.  The cap probes in steps of
    `increase` until the first tick at or over the target, then admission
    stops: the admitted count settles in [N*, N* + increase)."""
    T = CFG["target_ms"]
    n_star = math.ceil((T - a0) / b)
    assert a0 + b * n_star >= T > a0 + b * (n_star - 1)
    c = AimdAdmission(**{**CFG, "increase": step})
    series = _ramp(c, lambda n: a0 + b * n, rate, ticks=400)
    assert n_star <= series[-1] < n_star + step
    assert series[-1] == series[-60]          # settled, no further admission
    assert c.rejected > 0                     # the surplus is shed


def test_over_admits_on_a_flat_signal():
    """Unbounded KV: the per-tick latency stays flat (below target) while the
    resident state grows, so the identical loop reads pure headroom and
    admits every arrival -- far past the N* a monotone signal gives."""
    T = CFG["target_ms"]
    c = AimdAdmission(**CFG)
    _ramp(c, lambda n: 0.5 * T, 12, ticks=400)
    n_star_bounded = math.ceil((T - 20.0) / 1.21)       # the monotone case's N*
    assert c.admitted == CFG["max_cap"] > 2 * n_star_bounded
    assert c.decreases == 0


def test_churn_keeps_the_load_near_n_star():
    """Closed population with departures: the admitted load oscillates
    between a cut (about backoff * N*) and the probe back to N*."""
    T, a0, b = CFG["target_ms"], 20.0, 1.21
    n_star = math.ceil((T - a0) / b)
    rnd = random.Random(3)
    c = AimdAdmission(**CFG)
    loads = []
    for t in range(3000):
        for _ in range(12):
            c.offer()
        for _ in range(c.admitted):
            if rnd.random() < 0.02:
                c.release()
        c.observe(a0 + b * c.admitted)
        loads.append(c.admitted)
    tail = loads[1000:]
    assert max(tail) < n_star + CFG["increase"] + 12
    assert min(tail) >= math.floor(CFG["backoff"] * n_star) - 12
    assert 0.8 * n_star < sum(tail) / len(tail) <= n_star + CFG["increase"]


# ---- planted mistakes: each fails a pin above ------------------------------

class _AdditiveDecrease(AimdAdmission):
    def observe(self, tick_ms):
        if self.hold == 0 and tick_ms >= self.target_ms:
            self.ticks += 1
            self._demand_at_cap = False
            self.cap = max(self.min_cap, self.cap - self.increase)
            self.hold = self.hold_ticks
            self.decreases += 1
            return
        super().observe(tick_ms)


class _NoHold(AimdAdmission):
    def observe(self, tick_ms):
        self.hold = 0
        super().observe(tick_ms)


def test_planted_mistakes_fail():
    with pytest.raises(AssertionError):
        c = _AdditiveDecrease(**{**CFG, "initial_cap": 120})
        for _ in range(100):
            c.offer()
        c.observe(CFG["target_ms"])
        assert c.cap == 80
    with pytest.raises(AssertionError):
        c = _NoHold(**{**CFG, "hold_ticks": 3, "initial_cap": 50})
        for _ in range(50):
            c.offer()
        c.observe(1e9)
        cap = c.cap
        c.offer()
        c.observe(0.0)
        assert c.cap == cap


# ---- the library's controller, call by call --------------------------------

def _lib_ctrl(**cfg):
    mtn = pytest.importorskip("paper_2607_02640_amd")
    return mtn.Admission(**cfg)


@settings(max_examples=40, deadline=None)
@given(st.lists(st.tuples(st.sampled_from("ooorx"), st.floats(0, 1000, allow_nan=False)),
                max_size=400),
       st.sampled_from([0.5, 0.8, 0.9, 0.999]), st.integers(1, 9), st.integers(0, 4))
def test_library_matches_oracle_bit_exactly(ops, beta, step, hold):
    cfg = dict(target_ms=450.0, backoff=beta, increase=step, initial_cap=5, min_cap=2,
               max_cap=300, hold_ticks=hold)
    lib, orc = _lib_ctrl(**cfg), AimdAdmission(**cfg)
    for op, lat in ops:
        if op == "o":
            assert lib.offer() == orc.offer()
        elif op == "r":
            if orc.admitted:
                orc.release()
                lib.release()
        else:
            # latencies straddling the target, exact ties included
            lat = 450.0 if op == "x" else lat
            lib.observe(lat)
            orc.observe(lat)
        assert lib.state() == orc.state()


def test_library_rejects_bad_input():
    mtn = pytest.importorskip("paper_2607_02640_amd")
    for bad in (dict(target_ms=0.0), dict(target_ms=float("nan")), dict(backoff=1.0),
                dict(backoff=0.0), dict(increase=0), dict(min_cap=0), dict(initial_cap=0),
                dict(max_cap=10, initial_cap=16), dict(hold_ticks=-1)):
        with pytest.raises(mtn.MtnError) as e:
            mtn.Admission(**{**CFG, **bad})
        assert e.value.code == mtn.MTN_ERR_INVALID_ARG
    a = mtn.Admission(**CFG)
    with pytest.raises(mtn.MtnError) as e:
        a.release()
    assert e.value.code == mtn.MTN_ERR_BAD_STATE
    for lat in (float("nan"), -1.0, float("inf")):
        with pytest.raises(mtn.MtnError) as e:
            a.observe(lat)
        assert e.value.code == mtn.MTN_ERR_INVALID_ARG
    assert a.state()["ticks"] == 0
