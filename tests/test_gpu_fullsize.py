"""Full-size parity at the Qwen3-Omni-shaped workload, in the launch
configuration the bench times: 128 sessions, 48 layers, GQA 32/4, D = 128,
bf16 (and the FP8 KV cache, against the oracle holding the same E4M3 round
trip), S = 4, W = 4096, 25-token chunks + 16 decodes, pool sized to the exact
windowed reservation.  Sessions are fast-forwarded to a full window by
append-only plans, then one whole frame runs through mtn_frame_step.
Sampled (session, layer) pairs are recomputed one by one by the float64
oracle from the same inputs (all 32 heads, every chunk and decode output).
Tolerance: max-abs 2e-2 (bf16 in, fp32 accumulate, bf16 out)."""
import numpy as np
import pytest
import torch

from oracle import windowed_attention as wa
from tests._gpu_util import make_pool, say
from workload import MINICPM_O, MOSHI, POOL_STRESS_UNBOUNDED, QWEN3_OMNI as W, device_bank

pytestmark = pytest.mark.gpu


def _f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


@pytest.mark.parametrize("dtype,n_split", [("bf16", 0), ("bf16", 2), ("fp8", 0)])
def test_qwen3_omni_shape_sampled_parity(dtype, n_split):
    N, Lyr, Hq, Hkv, D = W.n_sessions, W.n_layers, W.n_q_heads, W.n_kv_heads, W.head_dim
    C, tau = W.chunk[1], W.n_decode[1]
    R = -(-(W.window + C - 1) // 16) * 16
    n_blocks = N * (-(-W.n_sink // 16) + R // 16)
    say(f"full-size pool: {n_blocks} blocks, {dtype}, n_split={n_split}")
    pool = make_pool(n_layers=Lyr, hq=Hq, hkv=Hkv, d=D, S=W.n_sink, W=W.window, cmax=C,
                     max_sessions=N, n_blocks=n_blocks, dtype=dtype, theta=W.rope_theta)
    sids = [pool.session_open() for _ in range(N)]
    dev = torch.device("cuda")
    bf = torch.bfloat16
    ff_k = device_bank((Lyr, N * C, Hkv, D), bf, dev, 71)
    ff_v = device_bank((Lyr, N * C, Hkv, D), bf, dev, 72)
    n_ff = -(-(W.n_sink + W.window) // C)
    for _ in range(n_ff):
        pool.plan_begin(sids, [C] * N)
        for l in range(Lyr):
            pool.frame_append_kv(l, ff_k[l], ff_v[l])
        pool.plan_commit()
    qc = device_bank((Lyr, N * C, Hq, D), bf, dev, 73)
    kc = device_bank((Lyr, N * C, Hkv, D), bf, dev, 74)
    vc = device_bank((Lyr, N * C, Hkv, D), bf, dev, 75)
    qd = device_bank((tau, Lyr, N, Hq, D), bf, dev, 76)
    kd = device_bank((tau, Lyr, N, Hkv, D), bf, dev, 77)
    vd = device_bank((tau, Lyr, N, Hkv, D), bf, dev, 78)
    oc = torch.empty_like(qc)
    od = torch.empty_like(qd)
    pool.frame_step(sids, [C] * N, [tau] * N, qc, kc, vc, oc, qd, kd, vd, od, n_split=n_split)
    torch.cuda.synchronize()
    assert torch.isfinite(oc.float()).all() and torch.isfinite(od.float()).all()
    say("frame done; oracle samples")
    worst = 0.0
    for (i, l) in [(0, 0), (77, 23), (127, 47)]:
        o = wa.OracleSession(Hq, Hkv, D, W.n_sink, W.window, theta=W.rope_theta, n_layers=1,
                             kv_quant="fp8_e4m3" if dtype == "fp8" else None)
        k_rows = _f64(ff_k[l, i * C:(i + 1) * C])
        v_rows = _f64(ff_v[l, i * C:(i + 1) * C])
        for _ in range(n_ff):
            o.begin(C)
            o.layer_step(0, np.zeros((C, Hq, D)), k_rows, v_rows, attend=False)
            o.commit()
        o.begin(C)
        ref, _ = o.layer_step(0, _f64(qc[l, i * C:(i + 1) * C]), _f64(kc[l, i * C:(i + 1) * C]),
                              _f64(vc[l, i * C:(i + 1) * C]))
        o.commit()
        err = float(np.max(np.abs(_f64(oc[l, i * C:(i + 1) * C]) - ref)))
        for j in range(tau):
            o.begin(1)
            rd, _ = o.layer_step(0, _f64(qd[j, l, i:i + 1]), _f64(kd[j, l, i:i + 1]),
                                 _f64(vd[j, l, i:i + 1]))
            o.commit()
            err = max(err, float(np.max(np.abs(_f64(od[j, l, i:i + 1]) - rd))))
        say(f"session {i} layer {l}: max abs err {err:.3e}")
        worst = max(worst, err)
    assert worst <= 2e-2, worst
    pool.close()


def _ragged_fullsize(wl, dtype, lengths, chunk_len, n_dec, samples, seed):
    """Fast-forward every session of workload `wl` to its own length by
    append-only plans (only the sessions still short of their length take
    part, at most max_chunk tokens each), run one ragged frame through
    mtn_frame_step, and recompute the sampled (session, layer) pairs with the
    float64 oracle from the same rows.  Returns the worst max-abs error."""
    N, Lyr, Hq, Hkv, D = wl.n_sessions, wl.n_layers, wl.n_q_heads, wl.n_kv_heads, wl.head_dim
    cmax = wl.max_chunk
    R = -(-(wl.window + cmax - 1) // 16) * 16
    n_blocks = N * (-(-wl.n_sink // 16) + R // 16)
    say(f"{wl.name}: pool of {n_blocks} blocks, {dtype}")
    pool = make_pool(n_layers=Lyr, hq=Hq, hkv=Hkv, d=D, S=wl.n_sink, W=wl.window, cmax=cmax,
                     max_sessions=N, n_blocks=n_blocks, dtype=dtype, theta=wl.rope_theta)
    sids = [pool.session_open() for _ in range(N)]
    dev = torch.device("cuda")
    bf = torch.bfloat16
    sc = wl.act_scale
    ff_k = device_bank((Lyr, N * cmax, Hkv, D), bf, dev, seed + 1, sc)
    ff_v = device_bank((Lyr, N * cmax, Hkv, D), bf, dev, seed + 2, sc)
    have = [0] * N
    plans = []  # per plan: {session: (row offset, n_tok)}
    while True:
        idx = [i for i in range(N) if have[i] < lengths[i]]
        if not idx:
            break
        nt = [min(cmax, lengths[i] - have[i]) for i in idx]
        pool.plan_begin([sids[i] for i in idx], nt)
        for l in range(Lyr):
            pool.frame_append_kv(l, ff_k[l], ff_v[l])
        pool.plan_commit()
        rows, off = {}, 0
        for i, n in zip(idx, nt):
            rows[i] = (off, n)
            off += n
            have[i] += n
        plans.append(rows)
    say(f"fast-forward done: {len(plans)} plans")
    T = sum(chunk_len)
    tau = max(n_dec)
    qc = device_bank((Lyr, T, Hq, D), bf, dev, seed + 3, sc)
    kc = device_bank((Lyr, T, Hkv, D), bf, dev, seed + 4, sc)
    vc = device_bank((Lyr, T, Hkv, D), bf, dev, seed + 5, sc)
    qd = device_bank((tau, Lyr, N, Hq, D), bf, dev, seed + 6, sc)
    kd = device_bank((tau, Lyr, N, Hkv, D), bf, dev, seed + 7, sc)
    vd = device_bank((tau, Lyr, N, Hkv, D), bf, dev, seed + 8, sc)
    oc = torch.empty_like(qc)
    od = torch.zeros_like(qd)
    pool.frame_step(sids, chunk_len, n_dec, qc, kc, vc, oc, qd, kd, vd, od)
    torch.cuda.synchronize()
    assert torch.isfinite(oc.float()).all() and torch.isfinite(od.float()).all()
    say("frame done; oracle samples")
    c_off = np.concatenate([[0], np.cumsum(chunk_len)])
    worst = 0.0
    for (i, l) in samples:
        o = wa.OracleSession(Hq, Hkv, D, wl.n_sink, wl.window, theta=wl.rope_theta, n_layers=1,
                             kv_quant="fp8_e4m3" if dtype == "fp8" else None)
        for rows in plans:
            if i not in rows:
                continue
            off, n = rows[i]
            o.begin(n)
            o.layer_step(0, np.zeros((n, Hq, D)), _f64(ff_k[l, off:off + n]),
                         _f64(ff_v[l, off:off + n]), attend=False)
            o.commit()
        a, b = int(c_off[i]), int(c_off[i + 1])
        o.begin(b - a)
        ref, _ = o.layer_step(0, _f64(qc[l, a:b]), _f64(kc[l, a:b]), _f64(vc[l, a:b]))
        o.commit()
        err = float(np.max(np.abs(_f64(oc[l, a:b]) - ref)))
        for j in range(n_dec[i]):
            o.begin(1)
            rd, _ = o.layer_step(0, _f64(qd[j, l, i:i + 1]), _f64(kd[j, l, i:i + 1]),
                                 _f64(vd[j, l, i:i + 1]))
            o.commit()
            err = max(err, float(np.max(np.abs(_f64(od[j, l, i:i + 1]) - rd))))
        say(f"session {i} (length {lengths[i]}) layer {l}: max abs err {err:.3e}")
        worst = max(worst, err)
    pool.close()
    return worst


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_minicpm_shape_ragged_sampled_parity(dtype):
    """MiniCPM-o-shaped backbone at full size: 256 sessions, 36 layers, GQA
    32/8, S = 4, W = 2048, chunks U{10..40}, decodes U{8..24}; 30 % of the
    sessions still filling their window, 70 % wrapped once or twice."""
    wl = MINICPM_O
    rng = np.random.default_rng(2026)
    N = wl.n_sessions
    full = wl.n_sink + wl.window
    lengths = [int(rng.integers(1, full - 60)) if i % 10 < 3 else int(rng.integers(full, 2 * full))
               for i in range(N)]
    chunk_len = [int(x) for x in rng.integers(wl.chunk[0], wl.chunk[1] + 1, N)]
    n_dec = [int(x) for x in rng.integers(wl.n_decode[0], wl.n_decode[1] + 1, N)]
    samples = [(0, 0), (5, 17), (200, 35), (N - 1, 9)]
    worst = _ragged_fullsize(wl, dtype, lengths, chunk_len, n_dec, samples, seed=510)
    assert worst <= 2e-2, worst


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_moshi_shape_sampled_parity(dtype):
    """Moshi-shaped temporal transformer at full size: 64 sessions, 32 layers,
    MHA 32/32, S = 4, W = 2048, one appended token and one decode per frame;
    a quarter of the sessions still filling their window, the rest wrapped."""
    wl = MOSHI
    N = wl.n_sessions
    full = wl.n_sink + wl.window
    lengths = [300 + 7 * i if i % 4 == 0 else full + 3 + 11 * i for i in range(N)]
    samples = [(0, 0), (1, 15), (62, 31)]
    worst = _ragged_fullsize(wl, dtype, lengths, [1] * N, [1] * N, samples, seed=520)
    assert worst <= 2e-2, worst


@pytest.mark.parametrize("rows", [256, 128])
def test_recycle_reprefill_sampled_parity(rows):
    """The application-level recycling arm's re-prefill at the Qwen3-Omni
    shape (§4.1's alternative, measured in §5): a fresh session takes the
    sinks plus the last W tokens of an old one, S + W = 4100 tokens, as one
    chunk on an unbounded pool with max_chunk 4100 -- 32 800 query rows per KV
    head in 129 passes of 256 rows (257 of 128), each over the keys its own
    rows see.  A second session takes a 37-token chunk in the same plan, then
    both decode one token.  Sampled chunk tokens (all 32 heads) and every
    other output against the float64 oracle."""
    Hq, Hkv, D, C, C2 = W.n_q_heads, W.n_kv_heads, W.head_dim, W.n_sink + W.window, 37
    say(f"recycle re-prefill: chunk {C}, {rows}-row passes")
    n_blocks = 2 * (-(-(C + 8) // 16))
    pool = make_pool(n_layers=1, hq=Hq, hkv=Hkv, d=D, S=0, W=None, cmax=C, max_sessions=2,
                     n_blocks=n_blocks, dtype="bf16", theta=W.rope_theta, max_len=C + 8)
    pool.set_prefill_pass_rows(rows)
    sids = [pool.session_open(), pool.session_open()]
    dev, bf = torch.device("cuda"), torch.bfloat16
    q = device_bank((C + C2, Hq, D), bf, dev, 91)
    k = device_bank((C + C2, Hkv, D), bf, dev, 92)
    v = device_bank((C + C2, Hkv, D), bf, dev, 93)
    out = torch.empty_like(q)
    pool.plan_begin(sids, [C, C2])
    pool.frame_append_kv(0, k, v)
    pool.attend_chunk_prefill(0, q, out)
    pool.plan_commit()
    qd = device_bank((2, Hq, D), bf, dev, 94)
    kd = device_bank((2, Hkv, D), bf, dev, 95)
    vd = device_bank((2, Hkv, D), bf, dev, 96)
    od = torch.empty_like(qd)
    pool.plan_begin(sids, [1, 1])
    pool.frame_append_kv(0, kd, vd)
    pool.attend_decode(0, qd, od)
    pool.plan_commit()
    torch.cuda.synchronize()
    assert torch.isfinite(out.float()).all() and torch.isfinite(od.float()).all()
    qh, kh, vh, oh = _f64(q), _f64(k), _f64(v), _f64(out)
    worst = 0.0
    # session 0: the long chunk's state, then sampled queries attended one by
    # one over the positions they see (unbounded: every earlier position)
    o = wa.OracleSession(Hq, Hkv, D, 0, None, theta=W.rope_theta, n_layers=1)
    o.begin(C)
    o.layer_step(0, np.zeros((C, Hq, D)), kh[:C], vh[:C], attend=False)
    o.commit()
    st = o.state[0]
    g = Hq // Hkv
    for t in [0, 1, 15, 16, 31, 32, 33, 255, 256, 511, 1024, 2047, 2048, 3000, 4090, C - 1]:
        vis = wa.visible_positions(t, 0, None)
        kmat = np.stack([st[p][0] for p in vis])
        vmat = np.stack([st[p][1] for p in vis])
        qr = wa.rope_rotate(qh[t], t, W.rope_theta)
        for h in range(Hq):
            ref, _, _ = wa.attend_row(qr[h], kmat[:, h // g], vmat[:, h // g], o.scale)
            worst = max(worst, float(np.max(np.abs(oh[t, h] - ref))))
    o.begin(1)
    rd, _ = o.layer_step(0, _f64(qd[0:1]), _f64(kd[0:1]), _f64(vd[0:1]))
    o.commit()
    worst = max(worst, float(np.max(np.abs(_f64(od[0:1]) - rd))))
    # session 1: every output of its chunk and its decode
    o2 = wa.OracleSession(Hq, Hkv, D, 0, None, theta=W.rope_theta, n_layers=1)
    ref2, _ = o2.step(qh[C:], kh[C:], vh[C:])
    worst = max(worst, float(np.max(np.abs(oh[C:] - ref2))))
    rd2, _ = o2.step(_f64(qd[1:2]), _f64(kd[1:2]), _f64(vd[1:2]))
    worst = max(worst, float(np.max(np.abs(_f64(od[1:2]) - rd2))))
    say(f"max abs err {worst:.3e}")
    assert worst <= 2e-2, worst
    pool.close()


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_pool_stress_unbounded_sampled_parity(dtype):
    """The pool-stress workload's unbounded arm at its last frame: 128
    sessions at the Qwen3-Omni head shapes on an unbounded pool (no window,
    no eviction), fast-forwarded to 299 frames of 41 tokens (12 259 tokens
    each), then frame 300 -- a 25-token chunk and 16 decodes -- through
    mtn_frame_step: every query sees its whole history, up to 12 300 keys
    (770 blocks per unit, three times the windowed arm).  Two layers (the
    launch configuration of a layer does not depend on the layer count).
    Sampled (session, layer) pairs against the float64 oracle."""
    wl = POOL_STRESS_UNBOUNDED
    N, Lyr, Hq, Hkv, D = wl.n_sessions, 2, wl.n_q_heads, wl.n_kv_heads, wl.head_dim
    C, tau = wl.chunk[1], wl.n_decode[1]
    L0 = 299 * (C + tau)
    max_len = L0 + C + tau
    n_blocks = N * -(-max_len // 16)
    say(f"unbounded full-size pool: {n_blocks} blocks, {dtype}, sessions at {L0} tokens")
    pool = make_pool(n_layers=Lyr, hq=Hq, hkv=Hkv, d=D, S=0, W=None, cmax=C, max_sessions=N,
                     n_blocks=n_blocks, dtype=dtype, theta=wl.rope_theta, max_len=max_len)
    sids = [pool.session_open() for _ in range(N)]
    dev, bf = torch.device("cuda"), torch.bfloat16
    ff_k = device_bank((Lyr, N * C, Hkv, D), bf, dev, 171)
    ff_v = device_bank((Lyr, N * C, Hkv, D), bf, dev, 172)
    ff = [C] * (L0 // C) + ([L0 % C] if L0 % C else [])
    for n in ff:
        pool.plan_begin(sids, [n] * N)
        for l in range(Lyr):
            pool.frame_append_kv(l, ff_k[l], ff_v[l])
        pool.plan_commit()
    say(f"fast-forward done: {len(ff)} plans")
    qc = device_bank((Lyr, N * C, Hq, D), bf, dev, 173)
    kc = device_bank((Lyr, N * C, Hkv, D), bf, dev, 174)
    vc = device_bank((Lyr, N * C, Hkv, D), bf, dev, 175)
    qd = device_bank((tau, Lyr, N, Hq, D), bf, dev, 176)
    kd = device_bank((tau, Lyr, N, Hkv, D), bf, dev, 177)
    vd = device_bank((tau, Lyr, N, Hkv, D), bf, dev, 178)
    oc = torch.empty_like(qc)
    od = torch.empty_like(qd)
    pool.frame_step(sids, [C] * N, [tau] * N, qc, kc, vc, oc, qd, kd, vd, od)
    torch.cuda.synchronize()
    assert torch.isfinite(oc.float()).all() and torch.isfinite(od.float()).all()
    say("frame done; oracle samples")
    worst = 0.0
    for (i, l) in [(0, 0), (77, 1), (127, 1)]:
        o = wa.OracleSession(Hq, Hkv, D, 0, None, theta=wl.rope_theta, n_layers=1,
                             kv_quant="fp8_e4m3" if dtype == "fp8" else None)
        for n in ff:
            # each fast-forward plan appended the session's first n rows of the bank
            o.begin(n)
            o.layer_step(0, np.zeros((n, Hq, D)), _f64(ff_k[l, i * n:(i + 1) * n]),
                         _f64(ff_v[l, i * n:(i + 1) * n]), attend=False)
            o.commit()
        o.begin(C)
        ref, _ = o.layer_step(0, _f64(qc[l, i * C:(i + 1) * C]), _f64(kc[l, i * C:(i + 1) * C]),
                              _f64(vc[l, i * C:(i + 1) * C]))
        o.commit()
        err = float(np.max(np.abs(_f64(oc[l, i * C:(i + 1) * C]) - ref)))
        for j in range(tau):
            o.begin(1)
            rd, _ = o.layer_step(0, _f64(qd[j, l, i:i + 1]), _f64(kd[j, l, i:i + 1]),
                                 _f64(vd[j, l, i:i + 1]))
            o.commit()
            err = max(err, float(np.max(np.abs(_f64(od[j, l, i:i + 1]) - rd))))
        say(f"session {i} layer {l}: max abs err {err:.3e}")
        worst = max(worst, err)
    assert worst <= 2e-2, worst
    pool.close()
