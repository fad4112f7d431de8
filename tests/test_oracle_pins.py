"""Pins of the float64 oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: every expected value comes from
a closed form, a library routine (torch SDPA on the CPU in float64), a
full-history computation that never prunes, a hand-enumerated fixture under
tests/golden/, or a textbook identity.  The planted-mistake tests at the end
show that plausible bugs in the oracle fail at least one pin.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

from oracle import windowed_attention as wa

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _rope_complex(x, pos, theta):
    """RoPE from its complex-exponential definition: pair (x_i, x_{i+D/2}) is
    the complex number x_i + j x_{i+D/2}, multiplied by exp(j pos theta^(-2i/D))."""
    x = np.asarray(x, np.float64)
    d = x.shape[-1]
    h = d // 2
    z = x[..., :h] + 1j * x[..., h:]
    w = np.exp(1j * pos * theta ** (-2.0 * np.arange(h) / d))
    zr = z * w
    return np.concatenate([zr.real, zr.imag], axis=-1)


def _run_session(sess, q, k, v, schedule):
    """Feed positions 0..T-1 through the session in the given chunk sizes."""
    outs, lses, t0 = [], [], 0
    for c in schedule:
        o, l = sess.step(q[t0:t0 + c], k[t0:t0 + c], v[t0:t0 + c])
        outs.append(o)
        lses.append(l)
        t0 += c
    return np.concatenate(outs), np.concatenate(lses)


def _schedule(rng, total, cmax):
    s, t = [], 0
    while t < total:
        c = int(min(rng.integers(1, cmax + 1), total - t))
        s.append(c)
        t += c
    return s


# ---------------------------------------------------------------------------
# Visibility: hand-enumerated fixture and closed-form counts
# ---------------------------------------------------------------------------

def check_visible_golden(visible_fn):
    with open(os.path.join(GOLDEN, "visible_sets.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        assert visible_fn(c["t"], c["S"], c["W"], False) == c["default"], c
        assert visible_fn(c["t"], c["S"], c["W"], True) == c["literal"], c


def test_visible_sets_match_hand_enumeration():
    check_visible_golden(wa.visible_positions)


@settings(max_examples=200, deadline=None)
@given(S=st.integers(0, 6), W=st.integers(1, 12), t=st.integers(0, 60))
def test_visible_count_closed_form(S, W, t):
    vis = wa.visible_positions(t, S, W)
    # all causal keys are visible until the window detaches from the sinks
    assert len(vis) == min(t + 1, S + W)
    assert vis[-1] == t
    tail = [p for p in vis if p >= S]
    assert tail == list(range(tail[0], t + 1)) if tail else True


def test_unbounded_sees_everything():
    assert wa.visible_positions(9, 3, None) == list(range(10))


# ---------------------------------------------------------------------------
# RoPE: the complex-exponential definition and its invariants
# ---------------------------------------------------------------------------

def check_rope(rope_fn):
    rng = _rng(1)
    for d in (8, 64, 128):
        x = rng.standard_normal((3, d))
        for pos in (0, 1, 17, 4099, 12345):
            got = rope_fn(x, pos, 10000.0)
            np.testing.assert_allclose(got, _rope_complex(x, pos, 10000.0),
                                       rtol=0, atol=1e-12)
            np.testing.assert_allclose(np.linalg.norm(got, axis=-1),
                                       np.linalg.norm(x, axis=-1), rtol=1e-13)
        np.testing.assert_array_equal(rope_fn(x, 0, 10000.0), x)
        q, k = rng.standard_normal(d), rng.standard_normal(d)
        a = rope_fn(q, 300, 1e4) @ rope_fn(k, 41, 1e4)
        b = rope_fn(q, 300 + 977, 1e4) @ rope_fn(k, 41 + 977, 1e4)
        assert abs(a - b) < 1e-10


def test_rope_definition_and_invariants():
    check_rope(wa.rope_rotate)


# ---------------------------------------------------------------------------
# Degenerate windows reduce to textbook attention
# ---------------------------------------------------------------------------

def _sdpa_reference(q, k, v, theta):
    """Full causal GQA attention via torch SDPA (float64, CPU) on inputs
    rotated with the complex-exponential RoPE."""
    t_len, hq, d = q.shape
    hkv = k.shape[1]
    qr = np.stack([_rope_complex(q[t], t, theta) for t in range(t_len)])
    kr = np.stack([_rope_complex(k[t], t, theta) for t in range(t_len)])
    Q = torch.from_numpy(qr).permute(1, 0, 2)            # [Hq, T, D]
    K = torch.from_numpy(kr).permute(1, 0, 2).repeat_interleave(hq // hkv, 0)
    V = torch.from_numpy(np.asarray(v, np.float64)).permute(1, 0, 2).repeat_interleave(hq // hkv, 0)
    o = torch.nn.functional.scaled_dot_product_attention(
        Q.unsqueeze(0), K.unsqueeze(0), V.unsqueeze(0), is_causal=True)
    return o[0].permute(1, 0, 2).numpy()


def check_full_causal(session_cls, seed=0):
    rng = _rng(seed)
    for (hq, hkv, d, S, W) in [(4, 2, 16, 3, 64), (8, 2, 8, 0, 40), (2, 2, 8, 5, None),
                               (6, 3, 8, 2, 33)]:
        T = 31
        q, k, v = (rng.standard_normal((T, h, d)) for h in (hq, hkv, hkv))
        sess = session_cls(hq, hkv, d, S, W, theta=500.0)
        out, _ = _run_session(sess, q, k, v, _schedule(rng, T, 6))
        ref = _sdpa_reference(q, k, v, 500.0)
        np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)


def test_window_covering_session_is_full_causal_attention():
    check_full_causal(wa.OracleSession)


def test_sinkless_unit_window_returns_own_value():
    rng = _rng(3)
    q, k, v = (rng.standard_normal((20, 2, 8)) for _ in range(3))
    sess = wa.OracleSession(2, 2, 8, 0, 1)
    out, lse = _run_session(sess, q, k, v, [3, 1, 5, 1, 1, 4, 5])
    np.testing.assert_allclose(out, v, rtol=0, atol=1e-14)
    # lse of a single key is its scaled score: <R(q,t), R(k,t)> = <q, k>
    np.testing.assert_allclose(lse, np.einsum("thd,thd->th", q, k) / math.sqrt(8),
                               rtol=0, atol=1e-12)


def test_one_sink_unit_window_two_term_softmax():
    rng = _rng(4)
    T, d = 12, 8
    q, k, v = (rng.standard_normal((T, 1, d)) for _ in range(3))
    sess = wa.OracleSession(1, 1, d, 1, 1, theta=1e4)
    out, _ = _run_session(sess, q, k, v, [1] * T)
    for t in range(1, T):
        qr = _rope_complex(q[t, 0], t, 1e4)
        s0 = qr @ _rope_complex(k[0, 0], 0, 1e4) / math.sqrt(d)
        st_ = qr @ _rope_complex(k[t, 0], t, 1e4) / math.sqrt(d)
        w0 = 1.0 / (1.0 + math.exp(st_ - s0))
        np.testing.assert_allclose(out[t, 0], w0 * v[0, 0] + (1 - w0) * v[t, 0],
                                   rtol=0, atol=1e-13)


# ---------------------------------------------------------------------------
# The mask, revealed by closed forms
# ---------------------------------------------------------------------------

def check_one_hot_reveals_set(session_cls, literal=False):
    """q = 0 gives uniform weights, and V_p = e_p makes out[t] the indicator
    of vis(t) divided by its size: the output spells out the visible set."""
    with open(os.path.join(GOLDEN, "visible_sets.json")) as f:
        cases = json.load(f)["cases"]
    for c in cases:
        S, W, t_max = c["S"], c["W"], c["t"]
        T = t_max + 1
        d = max(8, T + (T % 2))
        q = np.zeros((T, 1, d))
        k = _rng(5).standard_normal((T, 1, d))
        v = np.zeros((T, 1, d))
        v[np.arange(T), 0, np.arange(T)] = 1.0
        sess = session_cls(1, 1, d, S, W, literal_window=literal)
        out, _ = _run_session(sess, q, k, v, [1] * T)
        row = out[t_max, 0]
        expect = c["literal" if literal else "default"]
        support = [int(i) for i in np.nonzero(row > 0)[0]]
        assert support == expect, (c, support)
        np.testing.assert_allclose(row[expect], 1.0 / len(expect), rtol=0, atol=1e-15)


def test_one_hot_values_reveal_visible_set():
    check_one_hot_reveals_set(wa.OracleSession)
    check_one_hot_reveals_set(wa.OracleSession, literal=True)


# ---------------------------------------------------------------------------
# Pruning never drops a needed key: pruned state machine == full history
# ---------------------------------------------------------------------------

@settings(max_examples=40, deadline=None)
@given(S=st.integers(0, 5), W=st.integers(1, 9), cmax=st.integers(1, 12),
       G=st.sampled_from([1, 2, 3]), seed=st.integers(0, 10_000))
def test_pruned_oracle_equals_dense_full_history(S, W, cmax, G, seed):
    rng = _rng(seed)
    T, hkv, d = 40, 2, 8
    hq = G * hkv
    q = rng.standard_normal((T, hq, d))
    k = rng.standard_normal((T, hkv, d))
    v = rng.standard_normal((T, hkv, d))
    sess = wa.OracleSession(hq, hkv, d, S, W, theta=777.0)
    out, lse = _run_session(sess, q, k, v, _schedule(rng, T, cmax))
    ref, ref_lse = wa.dense_mask_attention(q, k, v, S, W, 777.0)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, ref_lse, rtol=0, atol=1e-12)


def test_brute_force_enumeration_tiny():
    """Pure-Python loops over every (query, key) pair of a tiny history."""
    rng = _rng(7)
    T, hq, hkv, d, S, W = 9, 2, 1, 4, 2, 3
    q, k, v = (rng.standard_normal((T, h, d)) for h in (hq, hkv, hkv))
    sess = wa.OracleSession(hq, hkv, d, S, W, theta=100.0)
    out, _ = _run_session(sess, q, k, v, [2, 1, 3, 1, 2])
    for t in range(T):
        for h in range(hq):
            qr = _rope_complex(q[t, h], t, 100.0)
            scores, vals = [], []
            for key in range(T):
                if key <= t and (key < S or key > t - W):
                    kr = _rope_complex(k[key, 0], key, 100.0)
                    scores.append(sum(qr[i] * kr[i] for i in range(d)) / math.sqrt(d))
                    vals.append(v[key, 0])
            m = max(scores)
            w = [math.exp(s - m) for s in scores]
            z = sum(w)
            exp = sum(wi / z * vi for wi, vi in zip(w, vals))
            np.testing.assert_allclose(out[t, h], exp, rtol=0, atol=1e-13)


# ---------------------------------------------------------------------------
# Retention: Ret(L) after arbitrary schedules, eviction ranges partition
# ---------------------------------------------------------------------------

@settings(max_examples=80, deadline=None)
@given(S=st.integers(0, 5), W=st.integers(1, 9), cmax=st.integers(1, 12),
       seed=st.integers(0, 10_000))
def test_retained_set_and_evictions_after_any_schedule(S, W, cmax, seed):
    rng = _rng(seed)
    T, d = 50, 4
    sess = wa.OracleSession(1, 1, d, S, W, n_layers=2)
    evicted = []
    t = 0
    for c in _schedule(rng, T, cmax):
        sess.begin(c)
        for layer in range(2):
            sess.layer_step(layer, rng.standard_normal((c, 1, d)),
                            rng.standard_normal((c, 1, d)),
                            rng.standard_normal((c, 1, d)), attend=False)
        lo, hi = sess.commit()
        t += c
        evicted.extend(range(lo, hi))
        keep = {p for p in range(t) if p < S or p >= t - W}
        for layer in range(2):
            assert set(sess.state[layer]) == keep
        assert len(keep) == min(t, S + W)
    # every position that ever left was a non-sink outside the final window,
    # and each left exactly once
    assert sorted(evicted) == list(range(S, max(S, T - W)))


def test_softmax_rows_sum_to_one_with_extreme_scores():
    rng = _rng(8)
    q = 40.0 * rng.standard_normal((30, 2, 8))
    k = 40.0 * rng.standard_normal((30, 2, 8))
    v = rng.standard_normal((30, 2, 8))
    sess = wa.OracleSession(2, 2, 8, 2, 5)
    _run_session(sess, q, k, v, [4, 1, 1, 7, 1, 8, 8])  # asserts |sum P - 1| < 1e-12


# ---------------------------------------------------------------------------
# Planted mistakes: each plausible bug fails at least one pin
# ---------------------------------------------------------------------------

def _fails(fn, *a, **kw):
    try:
        fn(*a, **kw)
    except AssertionError:
        return True
    return False


def test_planted_off_by_one_window_is_caught():
    def vis_plus_one(t, S, W, literal=False):
        return wa.visible_positions(t, S, W, not literal)
    assert _fails(check_visible_golden, vis_plus_one)


def test_planted_dropped_sinks_are_caught():
    def vis_no_sinks(t, S, W, literal=False):
        return wa.visible_positions(t, 0, W, literal)
    assert _fails(check_visible_golden, vis_no_sinks)


def test_planted_rope_sign_flip_is_caught():
    def rope_flipped(x, pos, theta):
        return wa.rope_rotate(x, -pos, theta)
    assert _fails(check_rope, rope_flipped)


def test_planted_rope_interleaved_variant_is_caught():
    def rope_interleaved(x, pos, theta):
        x = np.asarray(x, np.float64)
        d = x.shape[-1]
        perm = np.concatenate([np.arange(0, d, 2), np.arange(1, d, 2)])
        inv = np.argsort(perm)
        return wa.rope_rotate(x[..., perm], pos, theta)[..., inv]
    assert _fails(check_rope, rope_interleaved)


class _WrongGqaSession(wa.OracleSession):
    def __init__(self, *a, **kw):
        super().__init__(*a, **kw)
        hkv = self.hkv
        # interleaved grouping h % Hkv instead of contiguous floor(h / G)
        self.g = 1 if hkv == 1 else None
        self._hkv = hkv

    def layer_step(self, layer, q, k, v, attend=True):
        if self.g is None:
            q = np.asarray(q, np.float64).reshape(-1, self.hq, self.d)
            idx = np.array([(h % self._hkv) * (self.hq // self._hkv) + h // self._hkv
                            for h in range(self.hq)])
            inv = np.argsort(idx)
            self.g = self.hq // self._hkv
            res = super().layer_step(layer, q[:, idx], k, v, attend)
            self.g = None
            if res is None:
                return None
            return res[0][:, inv], res[1][:, inv]
        return super().layer_step(layer, q, k, v, attend)


def test_planted_wrong_gqa_grouping_is_caught():
    assert _fails(check_full_causal, _WrongGqaSession)


class _StaleChunkSession(wa.OracleSession):
    """Attends each chunk query before inserting the chunk (no intra-chunk
    causality) -- a plausible ordering mistake."""

    def layer_step(self, layer, q, k, v, attend=True):
        c = self._pending
        if c == 1 or not attend:
            return super().layer_step(layer, q, k, v, attend)
        outs, lses = [], []
        base = self.length
        for i in range(c):
            # give each query only the keys up to the chunk start plus itself
            st_ = self.state[layer]
            saved = dict(st_)
            self.state[layer] = {p: kv for p, kv in saved.items() if p < base}
            self._pending = 1
            self.length = base + i
            o, l = super().layer_step(layer, q[i:i + 1], k[i:i + 1], v[i:i + 1])
            self.state[layer] = saved
            self.state[layer][base + i] = (wa.rope_rotate(np.asarray(k[i], np.float64),
                                                          base + i, self.theta),
                                           np.asarray(v[i], np.float64))
            outs.append(o)
            lses.append(l)
        self.length = base
        self._pending = c
        return np.concatenate(outs), np.concatenate(lses)


def test_planted_chunk_causality_mistake_is_caught():
    assert _fails(check_full_causal, _StaleChunkSession)


class _LiteralWindowSession(wa.OracleSession):
    def __init__(self, *a, **kw):
        kw["literal_window"] = not kw.get("literal_window", False)
        super().__init__(*a, **kw)


def test_planted_window_reading_swap_is_caught_by_one_hot():
    assert _fails(check_one_hot_reveals_set, _LiteralWindowSession)
