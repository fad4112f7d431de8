"""GPU parity: the HIP path through the C ABI against the float64 oracle on
identical seeded inputs.  Tolerances: max-abs 1e-5 for fp32 pools, 2e-2 for
bf16 pools (bf16 in, fp32 accumulate, bf16 out)."""
import random

import numpy as np
import pytest
import torch

from tests._gpu_util import Harness, f64, make_pool, say

pytestmark = pytest.mark.gpu


def _tiny(dtype="f32", d=64, hq=8, hkv=2, S=4, W=128, cmax=8, n=4, L=1, blocks=80):
    pool = make_pool(n_layers=L, hq=hq, hkv=hkv, d=d, S=S, W=W, cmax=cmax, max_sessions=n,
                     n_blocks=blocks, dtype=dtype)
    h = Harness(pool, n_sessions=n, n_layers=L, hq=hq, hkv=hkv, d=d, S=S, W=W, dtype=dtype)
    return pool, h


def test_tiny_config_every_output_40_frames():
    """4 sessions, GQA 8/2, D = 64, fp32, S = 4, W = 128, 8-token chunks and 4
    decodes for 40 frames: the window wraps several times."""
    say("tiny f32 40 frames")
    pool, h = _tiny()
    for f in range(40):
        h.frame([8] * 4, [4] * 4)
    say(f"max err {h.max_err:.2e} lse {h.max_lse_err:.2e}")
    assert pool.session_info(h.sids[0])[0] == 480


def test_per_layer_calls_match_oracle_ragged():
    say("per-layer ragged f32")
    pool, h = _tiny(S=3, W=37, cmax=11, n=5, L=2)
    rnd = random.Random(1)
    for f in range(30):
        h.frame([rnd.randint(1, 11) for _ in range(5)], [rnd.randint(0, 5) for _ in range(5)],
                use_frame_step=False)


@pytest.mark.parametrize("g", [1, 2, 4, 8])
def test_bf16_d128_gqa_groups(g):
    say(f"bf16 d128 G={g}")
    hkv = 2
    pool, h = _tiny(dtype="bf16", d=128, hq=hkv * g, hkv=hkv, S=4, W=70, cmax=25, n=3, L=2,
                    blocks=3 * 10)
    rnd = random.Random(g)
    for f in range(12):
        h.frame([rnd.randint(1, 25) for _ in range(3)], [rnd.randint(0, 6) for _ in range(3)])
    say(f"max err {h.max_err:.2e}")


def test_bf16_chunk_longer_than_window():
    """C > W: chunk tokens leave the window inside their own chunk."""
    say("bf16 C > W")
    pool, h = _tiny(dtype="bf16", d=128, hq=16, hkv=2, S=3, W=8, cmax=25, n=3, L=1, blocks=12)
    for f in range(8):
        h.frame([25, 9, 1], [2, 0, 3])


def test_bf16_multi_pass_rows():
    """C * G > 256 query rows per (sequence, kv head): several row passes."""
    say("bf16 multi-pass rows")
    pool, h = _tiny(dtype="bf16", d=128, hq=16, hkv=2, S=4, W=100, cmax=40, n=2, L=1, blocks=20)
    for f in range(5):
        h.frame([40, 33], [1, 2])


@pytest.mark.parametrize("dtype,d", [("f32", 128), ("bf16", 64)])
def test_other_head_dims(dtype, d):
    say(f"{dtype} d{d}")
    pool, h = _tiny(dtype=dtype, d=d, hq=8, hkv=4, S=5, W=40, cmax=9, n=3)
    rnd = random.Random(7)
    for f in range(15):
        h.frame([rnd.randint(1, 9) for _ in range(3)], [rnd.randint(0, 4) for _ in range(3)])


@pytest.mark.parametrize("n_split", [1, 2, 3, 7, 33, 64])
def test_decode_split_counts(n_split):
    """Forced splits run as asked (the library reports the split of its last
    decode launch): with 64 segments over a 94-key window most segments are
    empty, and the merge must ignore them."""
    say(f"split {n_split}")
    pool, h = _tiny(S=4, W=90, cmax=8, n=3)
    for f in range(14):
        h.frame([8] * 3, [3] * 3, n_split=n_split)
        assert pool.last_split() == n_split


def test_no_sinks_and_unit_window():
    say("S=0 W=1")
    pool, h = _tiny(S=0, W=1, cmax=4, n=2)
    for f in range(10):
        h.frame([4, 1], [2, 3])


def test_sinks_larger_than_a_block():
    say("S=20")
    pool, h = _tiny(S=20, W=24, cmax=6, n=2)
    for f in range(12):
        h.frame([6, 3], [2, 1])


def test_unbounded_policy():
    say("unbounded")
    pool = make_pool(n_layers=1, hq=8, hkv=2, d=64, S=0, W=None, cmax=8, max_sessions=3,
                     n_blocks=3 * 20, dtype="f32", max_len=300)
    h = Harness(pool, n_sessions=3, n_layers=1, hq=8, hkv=2, d=64, S=0, W=None, dtype="f32")
    for f in range(20):
        h.frame([8, 5, 1], [4, 2, 0])


def test_poisoned_dead_slots_are_never_read():
    """NaN in every unassigned block, every sink-block slot past S and every
    ring slot outside the retained set: the next frames stay finite and match."""
    say("poison")
    pool, h = _tiny(S=4, W=50, cmax=8, n=3, blocks=60)
    rnd = random.Random(3)
    for f in range(12):
        h.frame([rnd.randint(1, 8) for _ in range(3)], [rnd.randint(0, 4) for _ in range(3)])
        pool.poison_dead()
    say(f"max err {h.max_err:.2e}")


def test_session_churn_reuses_blocks():
    say("churn")
    pool, h = _tiny(S=4, W=40, cmax=8, n=3, blocks=3 * 8)
    for f in range(8):
        h.frame([8, 2, 5], [2, 2, 2])
    # close session 1 and reopen it fresh (new oracle state, new inputs)
    from oracle import windowed_attention as wa
    pool.session_close(h.sids[1])
    assert pool.session_open() == h.sids[1]
    h.orc[1] = wa.OracleSession(8, 2, 64, 4, 40, theta=1e4, n_layers=1)
    pool.poison_dead()
    for f in range(8):
        h.frame([8, 2, 5], [2, 2, 2])


@pytest.mark.parametrize("dtype,d,hq,hkv,S,W,cmax", [
    ("bf16", 128, 16, 2, 4, 70, 25),   # G = 8: two wave groups, the owner is the second
    ("bf16", 128, 4, 4, 3, 48, 1),     # G = 1, C_max = 1: ring R = W, so the window wraps
    ("f32", 64, 8, 2, 4, 37, 6),       # fp32 path, G = 4
])
def test_fused_decode_append_matches_oracle(dtype, d, hq, hkv, S, W, cmax):
    """mtn_attend_decode_append (one launch: the newest key from the inputs,
    the pool copy written for later calls) against the oracle, per-layer
    calls over ragged frames, dead slots NaN-poisoned between frames."""
    say(f"fused decode+append {dtype} d{d} {hq}/{hkv} S={S} W={W} cmax={cmax}")
    n = 3
    R = -(-(W + cmax - 1) // 16) * 16
    pool, h = _tiny(dtype=dtype, d=d, hq=hq, hkv=hkv, S=S, W=W, cmax=cmax, n=n, L=2,
                    blocks=n * (-(-S // 16) + R // 16))
    rnd = random.Random(11)
    for f in range(14):
        h.frame([rnd.randint(1, cmax) for _ in range(n)], [rnd.randint(0, 5) for _ in range(n)],
                use_frame_step=False, fused=True)
        pool.poison_dead()
    say(f"max err {h.max_err:.2e}")


def test_fused_and_separate_calls_store_identical_pools():
    """The fused call stores exactly what mtn_frame_append_kv stores: two
    pools, NaN-poisoned end to end, fed the same frames through the two call
    sequences, hold bit-identical bytes after every frame."""
    say("fused vs separate pool bytes")
    n, L = 3, 2
    cfg = dict(dtype="bf16", d=128, hq=16, hkv=2, S=4, W=40, cmax=9, n=n, L=L, blocks=n * 4)
    pa, ha = _tiny(**cfg)
    pb, hb = _tiny(**cfg)
    pa.poison_dead()
    pb.poison_dead()
    rnd = random.Random(5)
    for f in range(10):
        cl = [rnd.randint(1, 9) for _ in range(n)]
        nd = [rnd.randint(0, 4) for _ in range(n)]
        ha.frame(cl, nd, use_frame_step=False, fused=True)
        hb.frame(cl, nd, use_frame_step=False, fused=False)
        torch.cuda.synchronize()
        assert torch.equal(pa.kv, pb.kv), f"pool bytes differ after frame {f}"


@pytest.mark.parametrize("dtype,g", [("fp8", 8), ("fp8", 4), ("fp8", 1), ("bf16", 8)])
@pytest.mark.parametrize("rows", [0, 256])
def test_prefill_with_fused_append_stores_what_the_append_stores(dtype, g, rows):
    """mtn_frame_step folds the chunk append into the fp8 pool's chunk prefill
    when every sequence takes one row pass (the bf16 pool keeps the append
    launch, and the comparison then checks frame_step against the per-layer
    calls).  Two NaN-poisoned pools fed the same frames,
    one through mtn_frame_step and one through the separate per-layer calls,
    hold bit-identical bytes after every frame, and both match the oracle.
    Chunks of up to 40 tokens at G = 8 take one or two 256-row passes (two or
    three 128-row ones), so some plans fuse and some do not (at G = 1 every
    plan fuses, its waves storing up to seven tokens each in two batches); the sequences
    start empty (the chunk lies in the first stages a workgroup copies, so
    the copies wait behind the append) and grow past 18 blocks and through
    the window's wrap (the append then runs beside the first copies)."""
    say(f"prefill fused append vs separate pool bytes, {dtype}, G={g}, rows {rows}")
    n, L = 3, 2
    cfg = dict(dtype=dtype, d=128, hq=2 * g, hkv=2, S=4, W=300, cmax=40, n=n, L=L,
               blocks=n * (1 + 22) + 2)
    pa, ha = _tiny(**cfg)
    pb, hb = _tiny(**cfg)
    for p in (pa, pb):
        if rows:
            p.set_prefill_pass_rows(rows)
        p.kv.zero_()      # fp8 regions hold 96 padding bytes that no kernel writes
        p.poison_dead()
        p.set_timing(True)
        p.kernel_times()
    rnd = random.Random(11)
    n_chunk_plans = 0  # plans whose chunk prefill runs (not all one-token chunks)
    for f in range(16):
        cl = [rnd.randint(1, 40) for _ in range(n)]
        nd = [rnd.randint(0, 2) for _ in range(n)]
        n_chunk_plans += max(cl) > 1
        ha.frame(cl, nd, use_frame_step=True)
        hb.frame(cl, nd, use_frame_step=False, fused=False)
        torch.cuda.synchronize()
        assert torch.equal(pa.kv, pb.kv), f"pool bytes differ after frame {f}"
    ka, kb = pa.kernel_times(), pb.kernel_times()
    say(f"appends: frame_step {ka['append'][0]}, per-layer {kb['append'][0]}; "
        f"max err {ha.max_err:.2e} / {hb.max_err:.2e}")
    # frame_step launches an append only for chunk plans it does not fuse (its
    # decode rounds always fuse theirs)
    if dtype == "fp8":
        assert ka["append"][0] < n_chunk_plans * L, "no chunk plan took the fused prefill"
    else:
        assert ka["append"][0] == n_chunk_plans * L


@pytest.mark.parametrize("rows", [256, 128])
def test_bf16_long_chunks_split_into_row_passes(rows):
    """A re-prefill-sized chunk: 300 tokens x G = 8 is 2400 query rows, ten
    256-row (or nineteen 128-row) passes, each its own workgroup over the
    keys its rows can see; the window (130) is shorter than the chunk and the
    sinks (20) span two blocks, so passes differ in their sink, window and
    causal edges."""
    say(f"bf16 long chunks, {rows}-row passes")
    S, W, C = 20, 130, 300
    R = -(-(W + C - 1) // 16) * 16
    pool, h = _tiny(dtype="bf16", d=128, hq=16, hkv=2, S=S, W=W, cmax=C, n=2, L=1,
                    blocks=2 * (2 + R // 16))
    pool.set_prefill_pass_rows(rows)
    for cl in ([300, 137], [1, 300], [299, 5]):
        h.frame(cl, [2, 1])
    say(f"max err {h.max_err:.2e}")


@pytest.mark.parametrize("S,W,cmax,frames", [
    (4, 300, 40, 14),    # windows wrap; stages every row sees whole run the unmasked loop
    (20, 300, 33, 12),   # sinks span a whole block and part of the next
    (0, 200, 25, 12),    # no sinks
    (16, 1, 9, 6),       # sinks exactly one block, unit window
    (4, None, 30, 8),    # unbounded: every key stays visible
])
def test_bf16_mfma_prefill_edges(S, W, cmax, frames):
    """The MFMA chunk prefill (bf16, D = 128, G = 8) across the key-union
    shapes its stage loops split on: masked first and last stages around a run
    of unmasked ones, sink blocks whole or partial, no sinks, a unit window and
    the unbounded pool; first chunks of one token give one-stage passes."""
    say(f"bf16 mfma prefill S={S} W={W} cmax={cmax}")
    n, hkv, g = 3, 2, 8
    if W is None:
        pool = make_pool(n_layers=1, hq=hkv * g, hkv=hkv, d=128, S=S, W=None, cmax=cmax,
                         max_sessions=n, n_blocks=n * 40, dtype="bf16", max_len=600)
        h = Harness(pool, n_sessions=n, n_layers=1, hq=hkv * g, hkv=hkv, d=128, S=S, W=None,
                    dtype="bf16")
    else:
        R = -(-(W + cmax - 1) // 16) * 16
        pool, h = _tiny(dtype="bf16", d=128, hq=hkv * g, hkv=hkv, S=S, W=W, cmax=cmax, n=n,
                        L=1, blocks=n * (2 + -(-S // 16) + R // 16))
    rnd = random.Random(S * 1000 + cmax)
    h.frame([1, cmax, 2], [0, 1, 2])
    for f in range(frames - 1):
        h.frame([rnd.randint(1, cmax) for _ in range(n)], [rnd.randint(0, 3) for _ in range(n)])
    say(f"max err {h.max_err:.2e}")


def test_calls_on_a_side_stream():
    """Every launch and plan upload goes on the stream the caller passes: the
    harness's inputs, the library's work and the outputs all live on a side
    stream (torch's current stream inside the context)."""
    say("side stream")
    pool, h = _tiny(dtype="bf16", d=128, hq=16, hkv=2, S=4, W=60, cmax=12, n=3, L=2, blocks=3 * 7)
    s = torch.cuda.Stream()
    rnd = random.Random(11)
    with torch.cuda.stream(s):
        for f in range(8):
            h.frame([rnd.randint(1, 12) for _ in range(3)], [rnd.randint(0, 3) for _ in range(3)],
                    use_frame_step=(f % 2 == 0))
    say(f"max err {h.max_err:.2e}")


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("rows", [128, 256])
def test_prefill_pass_rows(dtype, rows):
    """Chunk prefill with 128- and with 256-row passes (G = 8: chunks of up
    to 40 tokens are up to 320 rows, so both sizes give one or more passes,
    some with waves whose second tile lies past the pass) against the
    oracle."""
    say(f"prefill pass rows {rows} {dtype}")
    S, W, C, n, hkv = 4, 120, 40, 3, 2
    R = -(-(W + C - 1) // 16) * 16
    pool = make_pool(n_layers=1, hq=8 * hkv, hkv=hkv, d=128, S=S, W=W, cmax=C, max_sessions=n,
                     n_blocks=n * (1 + R // 16), dtype=dtype)
    pool.set_prefill_pass_rows(rows)
    h = Harness(pool, n_sessions=n, n_layers=1, hq=8 * hkv, hkv=hkv, d=128, S=S, W=W, dtype=dtype)
    rnd = random.Random(rows)
    for f in range(8):
        h.frame([rnd.randint(1, C) for _ in range(n)], [rnd.randint(0, 2) for _ in range(n)])
    say(f"max err {h.max_err:.2e}")


@pytest.mark.parametrize("d,g", [(64, 1), (64, 8), (128, 1), (128, 8)])
def test_fp32_gqa_group_extremes(d, g):
    """fp32 pools at one query head per KV head and at the largest group the
    boundary accepts (the vector kernel's one-wave and two-wave-group shapes)."""
    say(f"f32 d{d} G={g}")
    hkv = 2
    pool, h = _tiny(dtype="f32", d=d, hq=hkv * g, hkv=hkv, S=4, W=45, cmax=7, n=3, L=2)
    rnd = random.Random(d + g)
    for f in range(12):
        h.frame([rnd.randint(1, 7) for _ in range(3)], [rnd.randint(0, 4) for _ in range(3)])
    say(f"max err {h.max_err:.2e}")


@pytest.mark.parametrize("g", [1, 4, 8])
def test_bf16_d64_gqa_groups(g):
    """bf16 at head_dim 64 (vector kernels for the chunk and the decode)."""
    say(f"bf16 d64 G={g}")
    hkv = 2
    pool, h = _tiny(dtype="bf16", d=64, hq=hkv * g, hkv=hkv, S=4, W=45, cmax=7, n=3, L=2)
    rnd = random.Random(64 + g)
    for f in range(12):
        h.frame([rnd.randint(1, 7) for _ in range(3)], [rnd.randint(0, 4) for _ in range(3)])
    say(f"max err {h.max_err:.2e}")


@pytest.mark.parametrize("kind,g", [(1, 8), (2, 1), (2, 2), (2, 4)])
def test_bf16_decode_kernel_forced(kind, g):
    """Each bf16 decode kernel on the shapes the automatic choice gives the
    other: the vector kernel at G = 8, the matrix-core kernel at G = 1, 2, 4
    (D = 128), with splits and the fused append."""
    say(f"bf16 decode kernel {kind} G={g}")
    hkv = 2
    pool, h = _tiny(dtype="bf16", d=128, hq=hkv * g, hkv=hkv, S=4, W=70, cmax=9, n=3, L=2,
                    blocks=3 * 6)
    pool.set_decode_kernel(kind)
    rnd = random.Random(10 * kind + g)
    for f in range(12):
        h.frame([rnd.randint(1, 9) for _ in range(3)], [rnd.randint(0, 4) for _ in range(3)],
                n_split=(0, 2, 5)[f % 3])
    say(f"max err {h.max_err:.2e}")


def test_plans_alternating_between_streams():
    """Consecutive plans on two streams with no host synchronisation in
    between: the library orders each plan's uploads after the previous plan's
    kernels (they share the metadata, RoPE table and split partials), so
    every frame still matches the oracle."""
    say("plans alternating between two streams")
    n, L, hq, hkv, d = 3, 2, 16, 2, 128
    pool, h = _tiny(dtype="bf16", d=d, hq=hq, hkv=hkv, S=4, W=60, cmax=12, n=n, L=L, blocks=3 * 7)
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    rnd = random.Random(17)
    frames = []
    for f in range(10):
        cl = [rnd.randint(1, 12) for _ in range(n)]
        nd = [rnd.randint(0, 3) for _ in range(n)]
        draws = [h._draw(i, cl[i]) for i in range(n)]
        dec = [[h._draw(i, 1) if nd[i] > j else None for i in range(n)] for j in range(max(nd))]
        frames.append((cl, nd, draws, dec))
    # inputs on the device before any plan runs
    dev = []
    for cl, nd, draws, dec in frames:
        qc, kc, vc = (torch.cat([dr[j] for dr in draws], dim=1).contiguous().cuda()
                      for j in range(3))
        md = max(nd)
        if md:
            def dstack(c, hh):
                out = torch.zeros((md, L, n, hh, d), dtype=torch.bfloat16)
                for j in range(md):
                    for i in range(n):
                        if dec[j][i] is not None:
                            out[j, :, i] = dec[j][i][c][:, 0]
                return out.cuda()
            qd, kd, vd = dstack(0, hq), dstack(1, hkv), dstack(2, hkv)
        else:
            qd = kd = vd = None
        dev.append((qc, kc, vc, torch.empty_like(qc), qd, kd, vd,
                    torch.zeros_like(qd) if md else None))
    torch.cuda.synchronize()
    for f, (cl, nd, _, _) in enumerate(frames):
        qc, kc, vc, oc, qd, kd, vd, od = dev[f]
        with torch.cuda.stream(streams[f % 2]):
            if f % 3 == 2:   # per-layer calls on this stream
                pool.plan_begin(h.sids, cl)
                for l in range(L):
                    pool.frame_append_kv(l, kc[l], vc[l])
                    if max(cl) == 1:
                        pool.attend_decode(l, qc[l], oc[l])
                    else:
                        pool.attend_chunk_prefill(l, qc[l], oc[l])
                pool.plan_commit()
                nd[:] = [0] * n   # decodes of this frame are not issued
            else:
                pool.frame_step(h.sids, cl, nd, qc, kc, vc, oc, qd, kd, vd, od, n_split=2)
    torch.cuda.synchronize()
    for f, (cl, nd, draws, dec) in enumerate(frames):
        qc, kc, vc, oc, qd, kd, vd, od = dev[f]
        off = 0
        for i in range(n):
            ref, _ = h._oracle_step(i, *draws[i])
            got = oc[:, off:off + cl[i]].cpu()
            assert float(np.max(np.abs(f64(got) - ref))) <= 2e-2, f"frame {f} chunk s{i}"
            off += cl[i]
        for j in range(max(nd) if nd else 0):
            for i in range(n):
                if nd[i] > j:
                    ref, _ = h._oracle_step(i, *dec[j][i])
                    got = od[j, :, i:i + 1].cpu()
                    assert float(np.max(np.abs(f64(got) - ref))) <= 2e-2, f"frame {f} dec{j} s{i}"


def test_misaligned_activation_buffers_are_rejected():
    """q/k/v/out move in 16-byte vectors: a buffer off by one element is an
    MTN_ERR_INVALID_ARG that changes nothing, and the plan then runs with
    aligned buffers and matches the oracle."""
    say("misaligned buffers")
    import paper_2607_02640_amd as mtn
    pool, h = _tiny(dtype="bf16", d=128, hq=8, hkv=2, S=4, W=64, cmax=8, n=2, L=1, blocks=16)
    h.frame([8, 5], [1, 0])
    T, hq, hkv, d = 4, 8, 2, 128
    pool.plan_begin(h.sids, [3, 1])
    flat = torch.zeros(T * hq * d + 8, dtype=torch.bfloat16, device="cuda")
    kflat = torch.zeros(T * hkv * d + 8, dtype=torch.bfloat16, device="cuda")
    k_bad = kflat[1:1 + T * hkv * d].view(T, hkv, d)
    q_bad = flat[1:1 + T * hq * d].view(T, hq, d)
    k_ok = torch.zeros(T, hkv, d, dtype=torch.bfloat16, device="cuda")
    q_ok = torch.zeros(T, hq, d, dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(q_ok)
    with pytest.raises(mtn.MtnError) as e:
        pool.frame_append_kv(0, k_bad, k_ok)
    assert e.value.code == mtn.MTN_ERR_INVALID_ARG
    pool.frame_append_kv(0, k_ok, k_ok)
    with pytest.raises(mtn.MtnError) as e:
        pool.attend_chunk_prefill(0, q_bad, out)
    assert e.value.code == mtn.MTN_ERR_INVALID_ARG
    with pytest.raises(mtn.MtnError) as e:
        pool.attend_chunk_prefill(0, q_ok, flat[1:1 + T * hq * d].view(T, hq, d))
    assert e.value.code == mtn.MTN_ERR_INVALID_ARG
    pool.plan_abort()
    torch.cuda.synchronize()
    # the sessions are where they were: the harness continues against the oracle
    assert [pool.session_info(s)[0] for s in h.sids] == [9, 5]
    h.frame([4, 7], [2, 1])
