"""Pins of the independent index model (oracle/index_model.py) against the
paper's block arithmetic and against brute-force invariants."""
import json
import os

import pytest
from hypothesis import given, settings, strategies as st

from oracle import index_model as im
from oracle import windowed_attention as wa

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden():
    with open(os.path.join(GOLDEN, "pool_arithmetic.json")) as f:
        return json.load(f)


def test_sink_blocks_pinned_per_session():
    # App. A: ceil(S / block) pinned blocks; S = 16 is one block, S = 32 two
    for S, nsb in [(0, 0), (4, 1), (16, 1), (17, 2), (32, 2)]:
        m = im.IndexModel(1000, 16, S, 64, 8, 4)
        assert m.n_sink_blocks == nsb
        assert m.row_len == nsb + im.round_up(64 + 7, 16) // 16


def test_eq1_exhaustion_frame_unbounded():
    g = _golden()["eq1_case"]
    n, C, tau, bs, nb = g["n_sessions"], g["chunk"], g["n_decode"], g["block_size"], g["n_blocks"]
    t_sat = nb / (n * (C + tau) / bs)
    assert abs(t_sat - g["t_sat_frames"]) < 1e-9
    m = im.IndexModel(nb, bs, 4, None, C, n, max_len=1 << 20)
    sids = [m.open() for _ in range(n)]
    frame = 0
    failed_at = None
    while failed_at is None:
        frame += 1
        for n_tok in [C] + [1] * tau:
            try:
                m.plan_begin(sids, [n_tok] * n)
            except im.IndexError_ as e:
                assert e.code == im.ERR_POOL_EXHAUSTED
                failed_at = frame
                break
            m.plan_commit()
    assert failed_at == g["exhaust_frame_1based"] == int(-(-t_sat // 1))


def test_windowed_plateau_matches_closed_form():
    g = _golden()
    p = g["plateau_case"]
    nb = g["eq1_case"]["n_blocks"]
    m = im.IndexModel(nb, 16, 4, 4096, 25, 128)
    assert m.row_len == p["blocks_per_session"]
    sids = [m.open() for _ in range(128)]
    assert m.reserved_blocks() == p["plateau_blocks"]
    assert abs(m.reserved_blocks() / nb - p["plateau_frac"]) < 1e-9
    # Drive one session far past a full ring lap: its assignment plateaus at
    # exactly its reservation and never exceeds it.
    for f in range(260):
        for n_tok in [25] + [1] * 16:
            m.plan_begin([sids[0]], [n_tok])
            m.plan_commit()
    row = m.block_table(sids[0])
    assert all(b >= 0 for b in row) and len(row) == p["blocks_per_session"]
    assert m.assigned() == p["blocks_per_session"]


def test_sinksweep_plateau_scales_with_window():
    g = _golden()["sinksweep_ratios"]
    a = im.IndexModel(10**6, 16, 0, 1024, 16, 32).row_len
    b = im.IndexModel(10**6, 16, 0, 2048, 16, 32).row_len
    assert abs((b / a) / g["w2048_over_w1024_s0"] - 1) < g["tolerance"]


@settings(max_examples=60, deadline=None)
@given(S=st.integers(0, 20), W=st.integers(1, 40), cmax=st.integers(1, 20),
       seed=st.integers(0, 10_000))
def test_ring_never_overwrites_a_needed_key(S, W, cmax, seed):
    """Brute force: for every plan, the slots of all keys any of its queries
    may read are distinct from each other and from nothing else written, so
    the ring capacity R = roundup(W + C_max - 1, block) suffices."""
    import random
    rnd = random.Random(seed)
    m = im.IndexModel(200, 16, S, W, cmax, 1)
    sid = m.open()
    for _ in range(25):
        c = rnd.randint(1, cmax)
        L = m.sessions[sid].length
        m.plan_begin([sid], [c])
        needed = set()
        for t in range(L, L + c):
            needed.update(wa.visible_positions(t, S, W))
        slots = {}
        row = m.block_table(sid)
        for p in needed:
            lb, off = m.logical_slot(p)
            key = (row[lb], off)
            assert key not in slots, (p, slots.get(key))
            slots[key] = p
        for tok in m.plan_tokens:
            assert slots.get((tok.block, tok.offset)) == tok.pos
        m.plan_commit()
        res = m.resident_slots(sid)
        assert len(set(res.values())) == len(res)
        assert set(res) == wa.retained_positions(m.sessions[sid].length, S, W)


def test_lowest_free_reuse_after_churn_hand_case():
    # S = 4 -> 1 sink block; W = 32, C_max = 1 -> R = 32 -> 2 ring blocks:
    # 3 blocks per session, pool of 10 blocks.
    m = im.IndexModel(10, 16, 4, 32, 1, 3)
    assert m.row_len == 3
    a, b, c = m.open(), m.open(), m.open()
    assert (a, b, c) == (0, 1, 2)
    # a takes positions 0..20: sink block, then ring block 0 and 1
    for _ in range(21):
        m.plan_begin([a], [1]); m.plan_commit()
    assert m.block_table(a) == [0, 1, 2]
    m.plan_begin([b, c], [1, 1]); m.plan_commit()
    assert m.block_table(b) == [3, -1, -1] and m.block_table(c) == [4, -1, -1]
    m.close(a)
    assert m.open() == 0            # lowest free session id is reused
    for _ in range(5):
        m.plan_begin([c, 0], [1, 1]); m.plan_commit()
    # plan 1: the new session's sink takes freed block 0; plan 4: c reaches
    # position 4 (its first ring block) and takes 1; plan 5: the new session
    # reaches position 4 and takes 2.
    assert m.block_table(c) == [4, 1, -1]
    assert m.block_table(0) == [0, 2, -1]


def test_errors_are_atomic():
    m = im.IndexModel(5, 16, 0, None, 16, 4, max_len=64)
    s0, s1 = m.open(), m.open()
    m.plan_begin([s0, s1], [16, 16]); m.plan_commit()
    m.plan_begin([s0, s1], [16, 16]); m.plan_commit()
    before = (m.block_table(s0), m.block_table(s1), list(m.free))
    with pytest.raises(im.IndexError_) as e:
        m.plan_begin([s0, s1], [16, 16])
    assert e.value.code == im.ERR_POOL_EXHAUSTED
    assert (m.block_table(s0), m.block_table(s1), list(m.free)) == before
    with pytest.raises(im.IndexError_) as e:
        m.plan_begin([s0], [17])
    assert e.value.code == im.ERR_CHUNK_TOO_LARGE
    m.close(s1)
    m.plan_begin([s0], [16]); m.plan_commit()
    m.plan_begin([s0], [16]); m.plan_commit()
    with pytest.raises(im.IndexError_) as e:
        m.plan_begin([s0], [1])
    assert e.value.code == im.ERR_SESSION_FULL
