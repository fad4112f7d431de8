"""GPU parity of the FP8 (E4M3) KV cache through the C ABI: the stored codes
and scale exponents against the oracle's codec, and attention outputs against
the float64 oracle that holds the same E4M3 round trip of every stored row
(bf16 io, max-abs 2e-2)."""
import random

import numpy as np
import pytest
import torch

from oracle.fp8_kv import E4M3_MAX, e4m3_decode, quantize_heads, scale_exponent
from oracle.windowed_attention import rope_rotate
from tests._gpu_util import Harness, f64, make_pool, say

pytestmark = pytest.mark.gpu

REGION = 4224  # bytes per (layer, block, kv head)
DEC = np.array([e4m3_decode(c) for c in range(256)])


def _pool(hq=16, hkv=2, S=4, W=70, cmax=8, n=3, L=1, blocks=None, max_len=0):
    R = -(-(W + cmax - 1) // 16) * 16 if W is not None else -(-max_len // 16) * 16
    if blocks is None:
        blocks = n * (-(-S // 16) + R // 16)
    pool = make_pool(n_layers=L, hq=hq, hkv=hkv, d=128, S=S, W=W, cmax=cmax, max_sessions=n,
                     n_blocks=blocks, dtype="fp8", max_len=max_len)
    h = Harness(pool, n_sessions=n, n_layers=L, hq=hq, hkv=hkv, d=128, S=S, W=W, dtype="fp8")
    return pool, h, blocks


def _region(kvb, layer, block, head, n_blocks, hkv):
    o = ((layer * n_blocks + block) * hkv + head) * REGION
    r = kvb[o:o + REGION]
    kc = r[:2048].reshape(16, 128)
    vc = r[2048:4096].reshape(4, 128, 4).transpose(0, 2, 1).reshape(16, 128)  # [key][d]
    return kc, vc, r[4096:4112], r[4112:4128]


def _k_codes_ok(got, got_eb, kr64):
    """The rotated key is computed in float32 on the device and in float64
    here: a code may differ only where the scaled value sits within float32
    rounding of a rounding midpoint (then it must still be a nearest code up
    to that error), and the exponent only where the row max sits that close
    to 448 * 2^e."""
    exp_codes, exp_eb = quantize_heads(kr64[None], as_float32=True)
    exp_codes, exp_eb = exp_codes[0], int(exp_eb[0])
    amax = float(np.max(np.abs(kr64)))
    e = int(got_eb) - 127
    if int(got_eb) != exp_eb:
        e_lo = scale_exponent(amax * (1 - 2.0 ** -20))
        e_hi = scale_exponent(amax * (1 + 2.0 ** -20))
        assert e_lo <= e <= e_hi, (got_eb, exp_eb, amax)
        return 0
    bad = np.nonzero(got != exp_codes)[0]
    for i in bad:
        y = kr64[i] * 2.0 ** -e
        dg, de = DEC[got[i]], DEC[exp_codes[i]]
        assert abs(dg - y) <= abs(de - y) + abs(y) * 2.0 ** -20 + 2.0 ** -40, (i, y, dg, de)
    return len(bad)


def test_append_stores_oracle_codes():
    """mtn_frame_append_kv on an fp8 pool: V codes and both exponent rows
    bit-exact against the oracle codec, K codes equal up to the float32
    rotation's rounding at midpoints; ragged chunks over several blocks."""
    say("fp8 append codes")
    hq, hkv, n = 8, 2, 3
    pool, h, nb = _pool(hq=hq, hkv=hkv, S=4, W=60, cmax=20, n=n)
    rng = np.random.default_rng(4)
    n_k_diff = n_total = 0
    for frame in range(4):
        chunk = [int(x) for x in rng.integers(1, 21, n)]
        T = sum(chunk)
        k = torch.from_numpy(rng.standard_normal((T, hkv, 128)).astype(np.float32)).to(torch.bfloat16)
        v = torch.from_numpy(rng.standard_normal((T, hkv, 128)).astype(np.float32) * 0.05).to(torch.bfloat16)
        if frame == 3:
            v[0, 0] = 0   # an all-zero row: exponent byte 127, zero codes
            k[1, 1] *= 1e-30
        pool.plan_begin(h.sids, chunk)
        pos, blk, off, _, _ = pool.plan_info(n)
        pool.frame_append_kv(0, k.cuda(), v.cuda())
        pool.plan_commit()
        torch.cuda.synchronize()
        kvb = pool.kv.cpu().numpy()
        for t in range(T):
            for hh in range(hkv):
                kc, vc, ke, ve = _region(kvb, 0, blk[t], hh, nb, hkv)
                k64, v64 = f64(k[t, hh]), f64(v[t, hh])
                cv, ev = quantize_heads(v64[None], as_float32=True)
                assert np.array_equal(vc[off[t]], cv[0]), (frame, t, hh)
                assert ve[off[t]] == ev[0]
                kr = rope_rotate(k64, pos[t], 1e4)
                n_k_diff += _k_codes_ok(kc[off[t]], ke[off[t]], kr)
                n_total += 128
    say(f"K codes differing at float32 midpoints: {n_k_diff} of {n_total}")
    assert n_k_diff <= n_total * 1e-3


@pytest.mark.parametrize("g", [1, 2, 4, 8])
def test_fp8_decode_gqa_groups(g):
    """Single-token frames through mtn_frame_step (every round is the fused
    decode + append) against the quantized oracle; the window wraps."""
    say(f"fp8 G={g}")
    hkv = 2
    pool, h, _ = _pool(hq=hkv * g, hkv=hkv, S=4, W=40, cmax=1, n=3, L=2)
    rnd = random.Random(g)
    for f in range(30):
        h.frame([1, 1, 1], [rnd.randint(0, 3) for _ in range(3)])
    say(f"max err {h.max_err:.2e} lse {h.max_lse_err:.2e}")


@pytest.mark.parametrize("fused", [False, True])
def test_fp8_per_layer_calls(fused):
    """mtn_frame_append_kv + mtn_attend_decode, or mtn_attend_decode_append,
    per layer; dead slots NaN-poisoned (NaN codes, infinite scales) between
    frames."""
    say(f"fp8 per-layer fused={fused}")
    pool, h, _ = _pool(hq=16, hkv=2, S=20, W=50, cmax=1, n=3, L=2)
    rnd = random.Random(7)
    for f in range(40):
        h.frame([1, 1, 1], [rnd.randint(0, 4) for _ in range(3)], use_frame_step=False,
                fused=fused)
        pool.poison_dead()
    say(f"max err {h.max_err:.2e}")


@pytest.mark.parametrize("n_split", [1, 2, 3, 7, 33, 64])
def test_fp8_decode_split_counts(n_split):
    say(f"fp8 split {n_split}")
    pool, h, _ = _pool(hq=8, hkv=2, S=4, W=150, cmax=1, n=3)
    for f in range(12):
        h.frame([1, 1, 1], [12, 5, 9], n_split=n_split)
        assert pool.last_split() == n_split


def test_fp8_fused_and_separate_store_identical_pools():
    """The fused decode quantizes the newest token exactly as the append
    kernel does: two pools fed the same frames through the two call
    sequences hold bit-identical bytes after every frame."""
    say("fp8 fused vs separate pool bytes")
    cfg = dict(hq=16, hkv=2, S=4, W=40, cmax=1, n=3, L=2)
    pa, ha, _ = _pool(**cfg)
    pb, hb, _ = _pool(**cfg)
    for p in (pa, pb):
        p.kv.zero_()      # the 96 padding bytes of each region are never written
        p.poison_dead()
    rnd = random.Random(5)
    for f in range(24):
        nd = [rnd.randint(0, 4) for _ in range(3)]
        ha.frame([1, 1, 1], nd, use_frame_step=False, fused=True)
        hb.frame([1, 1, 1], nd, use_frame_step=False, fused=False)
        torch.cuda.synchronize()
        assert torch.equal(pa.kv, pb.kv), f"pool bytes differ after frame {f}"


def test_fp8_unbounded_and_no_sinks():
    say("fp8 unbounded")
    pool, h, _ = _pool(hq=8, hkv=2, S=0, W=None, cmax=1, n=2, max_len=200,
                       blocks=2 * 13)
    for f in range(20):
        h.frame([1, 1], [5, 2])
    pool2, h2, _ = _pool(hq=8, hkv=2, S=0, W=1, cmax=1, n=2)
    for f in range(10):
        h2.frame([1, 1], [2, 3])


def test_fp8_quantization_error_against_exact_attention():
    """Quality, not parity: the fp8 pool's outputs against the exact
    (unquantized) float64 oracle stay within the quantization bound's order
    (reported), and far outside the bf16 pool's error."""
    from oracle import windowed_attention as wa
    say("fp8 vs exact")
    pool, h, _ = _pool(hq=8, hkv=2, S=4, W=64, cmax=1, n=2)
    exact = [wa.OracleSession(8, 2, 128, 4, 64) for _ in range(2)]
    worst = 0.0
    gen = torch.Generator().manual_seed(20261)
    for f in range(20):
        q = torch.randn(1, 2, 8, 128, generator=gen).to(torch.bfloat16)
        k = torch.randn(1, 2, 2, 128, generator=gen).to(torch.bfloat16)
        v = (torch.randn(1, 2, 2, 128, generator=gen) * 0.3).to(torch.bfloat16)
        out = torch.empty_like(q).cuda()
        pool.frame_step(h.sids, [1, 1], [0, 0], q.cuda(), k.cuda(), v.cuda(), out)
        torch.cuda.synchronize()
        for i in range(2):
            ref, _ = exact[i].step(f64(q[0, i:i + 1]), f64(k[0, i:i + 1]), f64(v[0, i:i + 1]))
            worst = max(worst, float(np.max(np.abs(f64(out[0, i:i + 1]) - ref))))
    say(f"fp8 vs exact max abs {worst:.3e}")
    assert worst < 0.1


@pytest.mark.parametrize("g", [1, 8])
def test_fp8_chunk_prefill_ragged(g):
    """Ragged chunks (MFMA prefill over converted fp8 stages) and decodes
    through mtn_frame_step, against the quantized oracle."""
    say(f"fp8 prefill G={g}")
    hkv = 2
    pool, h, _ = _pool(hq=hkv * g, hkv=hkv, S=4, W=70, cmax=25, n=3, L=2)
    rnd = random.Random(10 + g)
    for f in range(12):
        h.frame([rnd.randint(1, 25) for _ in range(3)], [rnd.randint(0, 6) for _ in range(3)])
    say(f"max err {h.max_err:.2e} lse {h.max_lse_err:.2e}")


def test_fp8_chunk_longer_than_window_poisoned():
    """C > W, per-layer calls, dead slots NaN-poisoned between frames."""
    say("fp8 C > W poisoned")
    pool, h, _ = _pool(hq=16, hkv=2, S=3, W=8, cmax=25, n=3, L=1)
    for f in range(8):
        h.frame([25, 9, 1], [2, 0, 3], use_frame_step=False)
        pool.poison_dead()


@pytest.mark.parametrize("rows", [256, 128])
def test_fp8_long_chunks_split_into_row_passes(rows):
    """300-token chunks at G = 8: ten 256-row (or nineteen 128-row) passes
    over fp8 stages; sinks span two blocks and the window is shorter than
    the chunk."""
    say(f"fp8 long chunks, {rows}-row passes")
    pool, h, _ = _pool(hq=16, hkv=2, S=20, W=130, cmax=300, n=2, L=1)
    pool.set_prefill_pass_rows(rows)
    for cl in ([300, 137], [1, 300], [299, 5]):
        h.frame(cl, [2, 1])
    say(f"max err {h.max_err:.2e}")
