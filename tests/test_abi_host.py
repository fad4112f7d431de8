"""CPU tests of the C ABI: the library loads, exports every declared symbol,
and its host planner (block tables, ring-slot map, evicted ranges, pool
counters, error codes) matches the independent index model bit-exactly.
No GPU: pools are created with MTN_POOL_HOST_ONLY."""
import os
import random
import re

import pytest

import paper_2607_02640_amd as mtn
from oracle import index_model as im

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_symbol():
    lib = mtn.load()
    with open(os.path.join(ROOT, "include", "mtn.h")) as f:
        hdr = f.read()
    declared = set(re.findall(r"\b(mtn_[a-z_]+)\s*\(", hdr))
    assert declared == set(mtn.EXPORTS), declared ^ set(mtn.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def _pair(n_blocks, S, W, cmax, max_sessions, max_len=None):
    pool = mtn.Pool(n_layers=2, n_q_heads=4, n_kv_heads=2, head_dim=64, n_sink=S, window=W,
                    max_chunk=cmax, max_sessions=max_sessions, n_blocks=n_blocks, dtype="f32",
                    max_len=max_len or 0, host_only=True)
    model = im.IndexModel(n_blocks, 16, S, W, cmax, max_sessions, max_len=max_len)
    return pool, model


def _code(fn, *a):
    try:
        r = fn(*a)
        return 0, r
    except mtn.MtnError as e:
        return e.code, None
    except im.IndexError_ as e:
        return e.code, None


def _compare(pool, model):
    st = pool.stats()
    assert st["assigned"] == model.assigned()
    assert st["reserved"] == model.reserved_blocks()
    assert st["blocks_per_session"] == model.row_len
    assert st["ring_tokens"] == model.ring
    assert st["sink_blocks"] == model.n_sink_blocks
    for sid, s in model.sessions.items():
        assert pool.block_table(sid) == model.block_table(sid)
        ln, na = pool.session_info(sid)
        assert ln == s.length
        assert na == sum(1 for b in s.row if b >= 0)


@pytest.mark.parametrize("policy", ["windowed", "unbounded"])
@pytest.mark.parametrize("seed", range(6))
def test_host_planner_matches_index_model(policy, seed):
    rnd = random.Random(seed)
    S = rnd.choice([0, 1, 4, 16, 20])
    W = None if policy == "unbounded" else rnd.choice([1, 5, 16, 33, 64])
    cmax = rnd.choice([1, 3, 8, 25])
    max_sessions = rnd.choice([2, 5])
    n_blocks = rnd.choice([8, 20, 60])
    max_len = rnd.choice([40, 100]) if W is None else None
    pool, model = _pair(n_blocks, S, W, cmax, max_sessions, max_len)
    for _ in range(250):
        op = rnd.random()
        if op < 0.12:
            a, ra = _code(pool.session_open)
            b, rb = _code(model.open)
            assert a == b and ra == rb
        elif op < 0.2 and model.sessions:
            sid = rnd.choice(list(model.sessions) + [max_sessions + 1])
            a, _ = _code(pool.session_close, sid)
            b, _ = _code(model.close, sid)
            assert a == b
        elif model.sessions:
            k = rnd.randint(1, len(model.sessions))
            sids = rnd.sample(sorted(model.sessions), k)
            if rnd.random() < 0.05:
                sids.append(sids[0])   # duplicate -> invalid
            n_tok = [rnd.randint(0 if rnd.random() < 0.03 else 1,
                                 cmax + (1 if rnd.random() < 0.05 else 0)) for _ in sids]
            a, _ = _code(pool.plan_begin, sids, n_tok)
            b, _ = _code(model.plan_begin, sids, n_tok)
            assert a == b, (a, b, sids, n_tok)
            if a == 0:
                pos, blk, off, lo, hi = pool.plan_info(len(sids))
                assert pos == [t.pos for t in model.plan_tokens]
                assert blk == [t.block for t in model.plan_tokens]
                assert off == [t.offset for t in model.plan_tokens]
                assert list(zip(lo, hi)) == model.plan_evicted
                # a second plan cannot open over this one
                c, _ = _code(pool.plan_begin, sids[:1], [1])
                assert c == mtn.MTN_ERR_BAD_STATE
                if rnd.random() < 0.1:   # closing during a plan is refused
                    c, _ = _code(pool.session_close, sids[0])
                    assert c == mtn.MTN_ERR_BAD_STATE
                if rnd.random() < 0.15:  # abandon the plan instead
                    pool.plan_abort()
                    model.plan_abort()
                else:
                    pool.plan_commit()
                    model.plan_commit()
        _compare(pool, model)


def test_device_calls_refused_on_host_only_pool():
    pool, _ = _pair(10, 4, 16, 4, 2)
    sid = pool.session_open()
    pool.plan_begin([sid], [2])
    lib = pool.lib
    assert lib.mtn_frame_append_kv(pool.h, 0, None, None, None) == mtn.MTN_ERR_BAD_STATE
    assert lib.mtn_attend_decode(pool.h, 0, None, None, None, 0, None) == mtn.MTN_ERR_BAD_STATE
    pool.plan_commit()
    assert pool.session_info(sid) == (2, 1)


def test_config_validation():
    bad = dict(n_layers=1, n_q_heads=8, n_kv_heads=3, head_dim=64, n_sink=4, window=16,
               max_chunk=4, max_sessions=2, n_blocks=10, dtype="f32", host_only=True)
    with pytest.raises(mtn.MtnError) as e:
        mtn.Pool(**bad)
    assert e.value.code == mtn.MTN_ERR_INVALID_ARG
    with pytest.raises(mtn.MtnError) as e:
        mtn.Pool(**{**bad, "n_kv_heads": 2, "head_dim": 96})
    assert e.value.code == mtn.MTN_ERR_UNSUPPORTED
    with pytest.raises(mtn.MtnError) as e:
        mtn.Pool(**{**bad, "n_kv_heads": 2, "block_size": 32})
    assert e.value.code == mtn.MTN_ERR_UNSUPPORTED
    with pytest.raises(mtn.MtnError) as e:
        mtn.Pool(**{**bad, "n_kv_heads": 2, "window": 0})
    assert e.value.code == mtn.MTN_ERR_INVALID_ARG


def test_required_bytes_layout():
    # [layer][block][kv_head]{K [16][D], V^T [D][16]}
    n = mtn.Pool.required(n_layers=48, n_q_heads=32, n_kv_heads=4, head_dim=128, n_sink=4,
                          window=4096, max_chunk=25, max_sessions=128, n_blocks=33152,
                          dtype="bf16")
    assert n == 48 * 33152 * 4 * 2 * 16 * 128 * 2


def test_fp8_pool_config_and_bytes():
    # E4M3 cache: 4224-byte (block, head) regions (2 KiB K codes, 2 KiB V codes,
    # 32 exponent bytes, padding to 128), bf16 io, head_dim 128 only
    kw = dict(n_layers=48, n_q_heads=32, n_kv_heads=4, head_dim=128, n_sink=4, window=4096,
              max_chunk=25, max_sessions=128, n_blocks=33152)
    assert mtn.Pool.required(**kw, dtype="fp8") == 48 * 33152 * 4 * 4224
    assert mtn.Pool.required(**kw, dtype="fp8") < 0.52 * mtn.Pool.required(**kw, dtype="bf16")
    pool = mtn.Pool(**kw, dtype="fp8", host_only=True)
    assert pool.stats()["blocks_per_session"] == 1 + 4128 // 16
    with pytest.raises(mtn.MtnError) as e:
        mtn.Pool(**{**kw, "head_dim": 64}, dtype="fp8", host_only=True)
    assert e.value.code == mtn.MTN_ERR_UNSUPPORTED
    from paper_2607_02640_amd import _lib
    cfg = _lib.PoolConfig(1, 8, 2, 128, 16, 4, 16, 4, 2, 0, 10, _lib.MTN_FP8_E4M3,
                          _lib.MTN_FP8_E4M3, 1e4, 0.0, _lib.MTN_POOL_HOST_ONLY)
    n = _lib.C.c_size_t()
    assert pool.lib.mtn_pool_required_bytes(_lib.C.byref(cfg), _lib.C.byref(n)) == \
        mtn.MTN_ERR_UNSUPPORTED   # fp8 io is refused: queries and outputs stay bf16


def test_windowed_admission_counts_pinned_blocks():
    # 3 blocks per session (1 sink + 2 ring); pool of 7 admits two sessions
    pool, model = _pair(7, 4, 32, 1, 4)
    assert pool.session_open() == 0 and pool.session_open() == 1
    with pytest.raises(mtn.MtnError) as e:
        pool.session_open()
    assert e.value.code == mtn.MTN_ERR_POOL_EXHAUSTED
    pool.session_close(0)
    assert pool.session_open() == 0


def test_prefill_pass_rows_setting():
    """The tuning hook takes 0 (per plan), 128 or 256 and refuses the rest
    without changing the pool."""
    pool = mtn.Pool(n_layers=1, n_q_heads=8, n_kv_heads=2, head_dim=128, n_sink=4, window=64,
                    max_chunk=8, max_sessions=2, n_blocks=12, dtype="bf16", host_only=True)
    for rows in (0, 128, 256, 0):
        pool.set_prefill_pass_rows(rows)
    for rows in (-1, 1, 64, 192, 512):
        with pytest.raises(mtn.MtnError) as e:
            pool.set_prefill_pass_rows(rows)
        assert e.value.code == mtn.MTN_ERR_INVALID_ARG


def test_table_index_width_and_status_strings():
    """Block-table entries are addressed with 32-bit indices: a configuration
    whose table would pass 2^31 entries is refused at validation; every status
    code has its own text."""
    lib = mtn.load()
    with pytest.raises(mtn.MtnError) as e:
        mtn.Pool(n_layers=1, n_q_heads=4, n_kv_heads=2, head_dim=64, n_sink=4, window=(1 << 21),
                 max_chunk=1, max_sessions=(1 << 14), n_blocks=10, dtype="f32", host_only=True)
    assert e.value.code == mtn.MTN_ERR_INVALID_ARG
    lib.mtn_status_string.restype = __import__("ctypes").c_char_p
    texts = {lib.mtn_status_string(c) for c in range(-10, 1)}
    assert len(texts) == 11 and b"unknown status" not in texts
    assert lib.mtn_status_string(mtn.MTN_ERR_HOST_MEMORY) == b"host allocation failed"


_OOM_CHILD = r"""
import resource, sys
sys.path.insert(0, sys.argv[1])
import paper_2607_02640_amd as mtn
mtn.load()
with open("/proc/self/statm") as f:
    vm = int(f.read().split()[0]) * resource.getpagesize()
lim = vm + (512 << 20)
resource.setrlimit(resource.RLIMIT_AS, (lim, lim))
try:
    # a 6 GiB host block table: far past the 512 MiB of headroom
    mtn.Pool(n_layers=1, n_q_heads=4, n_kv_heads=2, head_dim=64, n_sink=0, window=2032,
             max_chunk=1, max_sessions=(1 << 24), n_blocks=10, dtype="f32", host_only=True)
    print("created")
except mtn.MtnError as e:
    print("code", e.code)
"""


def test_host_allocation_failure_returns_a_status():
    """No C++ exception leaves the library: pool creation under an address
    space limit too small for its host block table returns
    MTN_ERR_HOST_MEMORY (the process survives)."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, "-c", _OOM_CHILD, ROOT], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 0, r.stderr[-2000:]
    assert r.stdout.strip() == f"code {mtn.MTN_ERR_HOST_MEMORY}", r.stdout + r.stderr[-2000:]


def _snapshot(pool, sids):
    return pool.stats(), {s: (pool.block_table(s), pool.session_info(s)) for s in sids}


@pytest.mark.parametrize("policy", ["windowed", "unbounded"])
def test_plan_abort_restores_the_pool(policy):
    """Failures inside a plan (a layer out of range, a null buffer: host-only
    pools refuse device calls too) leave the plan open; mtn_plan_abort then
    returns the pool to its state before mtn_plan_begin, bit for bit, and the
    next plan assigns exactly what it would have assigned without the abandoned
    one (failing cleanly instead of stalling, §3; App. B)."""
    W = None if policy == "unbounded" else 40
    nb = 60 if W is None else 30
    pool, model = _pair(nb, 4, W, 9, 3, max_len=200 if W is None else None)
    ref, ref_model = _pair(nb, 4, W, 9, 3, max_len=200 if W is None else None)
    sids = [pool.session_open() for _ in range(3)]
    for p_ in (model, ref, ref_model):
        [p_.session_open() if hasattr(p_, "session_open") else p_.open() for _ in range(3)]
    rnd = random.Random(7)
    lib = pool.lib
    for step in range(20 if W is None else 40):
        n_tok = [rnd.randint(1, 9) for _ in sids]
        before = _snapshot(pool, sids)
        pool.plan_begin(sids, n_tok)
        model.plan_begin(sids, n_tok)
        # per-layer calls that fail inside the plan
        assert lib.mtn_frame_append_kv(pool.h, 99, None, None, None) != mtn.MTN_OK
        assert lib.mtn_attend_chunk_prefill(pool.h, 0, None, None, None, None) != mtn.MTN_OK
        assert lib.mtn_plan_begin(pool.h, 1, mtn._lib._arr32(sids[:1]),
                                  mtn._lib._arr32([1]), None) == mtn.MTN_ERR_BAD_STATE
        if step % 3 == 0:
            pool.plan_abort()
            model.plan_abort()
            assert _snapshot(pool, sids) == before
            # the pool plans on as if the abandoned plan had never begun
            pool.plan_begin(sids, n_tok)
            model.plan_begin(sids, n_tok)
        ref.plan_begin(sids, n_tok)
        ref_model.plan_begin(sids, n_tok)
        assert pool.plan_info(len(sids)) == ref.plan_info(len(sids))
        for p_ in (pool, model, ref, ref_model):
            p_.plan_commit()
        _compare(pool, model)
        _compare(ref, ref_model)
        assert _snapshot(pool, sids) == _snapshot(ref, sids)
    with pytest.raises(mtn.MtnError) as e:
        pool.plan_abort()
    assert e.value.code == mtn.MTN_ERR_BAD_STATE


def _model_frame(model, sids, chunk, n_dec, n_layers, fail_at=None):
    """The frame as mtn_frame_step runs it -- the chunk plan, then one plan per
    decode round -- on the index model; with fail_at, the plan holding that
    launch point (chunk plans: one point per layer for one-token chunks, else
    two; decode rounds: one per layer) is abandoned and the frame stops."""
    per_chunk = n_layers * (1 if max(chunk) == 1 else 2)
    plans = [(list(sids), list(chunk), per_chunk)]
    for j in range(max(n_dec)):
        act = [s for s, d in zip(sids, n_dec) if d > j]
        plans.append((act, [1] * len(act), n_layers))
    k = fail_at
    for ps, nt, launches in plans:
        model.plan_begin(ps, nt)
        if k is not None and k < launches:
            model.plan_abort()
            return False
        if k is not None:
            k -= launches
        model.plan_commit()
    return True


@pytest.mark.parametrize("policy", ["windowed", "unbounded"])
def test_frame_step_plans_and_rolls_back_like_the_model(policy):
    """mtn_frame_step on a host-only pool plans every frame exactly as the index
    model's chunk plan + decode rounds; a launch failure injected anywhere in
    the frame abandons the plan it falls in, keeps the rounds already committed
    and leaves nothing open."""
    W = None if policy == "unbounded" else 48
    cmax, n_layers = 10, 3
    pool = mtn.Pool(n_layers=n_layers, n_q_heads=4, n_kv_heads=2, head_dim=64, n_sink=4,
                    window=W, max_chunk=cmax, max_sessions=4, n_blocks=80, dtype="f32",
                    max_len=400 if W is None else 0, host_only=True)
    model = im.IndexModel(80, 16, 4, W, cmax, 4, max_len=400 if W is None else None)
    sids = [pool.session_open() for _ in range(4)]
    for _ in range(4):
        model.open()
    rnd = random.Random(3)
    for frame in range(30):
        batch = rnd.sample(sids, rnd.randint(1, 4))
        chunk = [rnd.choice([1, rnd.randint(1, cmax)]) for _ in batch]
        n_dec = [rnd.randint(0, 4) for _ in batch]
        per_chunk = n_layers * (1 if max(chunk) == 1 else 2)
        total = per_chunk + n_layers * max(n_dec)
        fail_at = rnd.randrange(total) if rnd.random() < 0.4 else None
        if fail_at is not None:
            pool.inject_failure(fail_at)
        try:
            pool.frame_step(batch, chunk, n_dec, None, None, None, None)
            ok = True
        except mtn.MtnError as e:
            assert e.code == mtn.MTN_ERR_DEVICE and fail_at is not None
            ok = False
        assert ok == _model_frame(model, batch, chunk, n_dec, n_layers, fail_at)
        # nothing is left open: a plan can begin and be abandoned
        pool.plan_begin(batch[:1], [1])
        pool.plan_abort()
        _compare(pool, model)


def test_empty_plans_and_frames_are_refused_without_change():
    """An empty batch (no sequence) is an invalid argument for a plan and for a
    frame step, and leaves the pool as it was; so is a frame whose sessions all
    have zero tokens."""
    pool, model = _pair(20, 4, 16, 4, 3)
    sids = [pool.session_open() for _ in range(2)]
    for _ in sids:
        model.open()
    pool.plan_begin(sids, [3, 2])
    model.plan_begin(sids, [3, 2])
    pool.plan_commit()
    model.plan_commit()
    before = pool.stats()
    c, _ = _code(pool.plan_begin, [], [])
    assert c == mtn.MTN_ERR_INVALID_ARG
    c, _ = _code(pool.frame_step, [], [], [], None, None, None, None)
    assert c == mtn.MTN_ERR_INVALID_ARG
    c, _ = _code(pool.frame_step, sids, [0, 0], [0, 0], None, None, None, None)
    assert c == mtn.MTN_ERR_INVALID_ARG
    assert pool.stats() == before
    _compare(pool, model)
    # and the pool still plans normally afterwards
    pool.frame_step(sids, [1, 4], [2, 0], None, None, None, None)
    model.plan_begin(sids, [1, 4])
    model.plan_commit()
    model.plan_begin(sids[:1], [1])
    model.plan_commit()
    model.plan_begin(sids[:1], [1])
    model.plan_commit()
    _compare(pool, model)
