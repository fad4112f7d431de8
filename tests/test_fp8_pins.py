"""Pins of the FP8 (OCP E4M3) KV oracle: the codec against torch's
float8_e4m3fn conversion and the format's closed forms, the scale rule's
closed form, brute-force nearest-value search, and quantized attention
within its error bound of the exact float64 oracle."""
import math

import numpy as np
import pytest
import torch

from oracle import fp8_kv
from oracle.fp8_kv import (e4m3_decode, e4m3_decode_array, e4m3_encode, e4m3_encode_array,
                           quantize_row, scale_exponent)
from oracle.windowed_attention import OracleSession, rope_rotate

ALL = np.arange(256, dtype=np.uint8)
FINITE = [c for c in range(256) if (c & 0x7F) != 0x7F]


def torch_decode(codes):
    return torch.from_numpy(np.asarray(codes, np.uint8)).view(torch.float8_e4m3fn).float().numpy()


def torch_encode(x):
    t = torch.tensor(np.asarray(x, np.float32), dtype=torch.float32)
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy()


# ---- codec against the library routine -----------------------------------

def test_decode_matches_torch_on_every_code():
    mine = np.array([e4m3_decode(c) for c in ALL])
    ref = torch_decode(ALL).astype(np.float64)
    assert np.array_equal(np.isnan(mine), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(mine[ok], ref[ok])
    assert np.array_equal(np.signbit(mine[ok]), np.signbit(ref[ok]))
    assert sorted(c for c in range(256) if math.isnan(e4m3_decode(c))) == [0x7F, 0xFF]


def _midpoints():
    pos = sorted({e4m3_decode(c) for c in FINITE if e4m3_decode(c) >= 0})
    return [(a + b) / 2 for a, b in zip(pos, pos[1:])]


def test_encode_matches_torch_on_codes_midpoints_and_random():
    mids = _midpoints()
    vals = [e4m3_decode(c) for c in FINITE] + mids + [-m for m in mids]
    rng = np.random.default_rng(7)
    vals += list(rng.uniform(-448, 448, 4000).astype(np.float32))
    vals += list((rng.standard_normal(4000) * 2.0 ** rng.integers(-14, 8, 4000)).astype(np.float32))
    vals = [v for v in vals if abs(v) <= 448]
    x32 = np.asarray(vals, np.float32)
    assert np.array_equal(x32.astype(np.float64), np.asarray(vals, np.float64))  # all exact in fp32
    mine = np.array([e4m3_encode(v) for v in vals], np.uint8)
    assert np.array_equal(mine, torch_encode(x32))


def test_array_codec_equals_scalar_codec():
    """The vectorised encoder the oracle's rows use is the scalar definition
    element by element (and so torch's cast): every code, every midpoint,
    random and tiny values, signed zeros."""
    mids = _midpoints()
    rng = np.random.default_rng(17)
    vals = ([e4m3_decode(c) for c in FINITE] + mids + [-m for m in mids] + [0.0, -0.0]
            + list(rng.uniform(-448, 448, 3000)) + list(rng.standard_normal(3000) * 1e-3))
    x = np.array(vals)
    got = e4m3_encode_array(x)
    ref = np.array([e4m3_encode(v) for v in vals], np.uint8)
    assert np.array_equal(got, ref)
    dec = e4m3_decode_array(ALL)
    ok = ~np.isnan(dec)
    assert np.array_equal(dec[ok], np.array([e4m3_decode(c) for c in ALL])[ok])
    with pytest.raises(ValueError):
        e4m3_encode_array(np.array([1.0, 449.0]))


# ---- closed forms of the format ---------------------------------------------

@pytest.mark.parametrize("x,code", [
    (448.0, 0x7E), (-448.0, 0xFE), (1.0, 0x38), (-1.0, 0xB8), (2.0 ** -6, 0x08),
    (2.0 ** -9, 0x01), (7 * 2.0 ** -9, 0x07), (0.0, 0x00), (-0.0, 0x80),
    (1.0625, 0x38),          # tie between 1 and 1.125: even mantissa (000)
    (1.1875, 0x3A),          # tie between 1.125 and 1.25: even mantissa (010)
    (2.0 ** -10, 0x00),      # tie between 0 and the smallest subnormal
    (3 * 2.0 ** -10, 0x02),  # tie between 2^-9 and 2^-8: even (010)
    (-2.0 ** -11, 0x80),     # rounds to zero, keeps the sign
    (240.0, 0x77), (256.0, 0x78), (432.0, 0x7E), (415.99, 0x7D),
])
def test_closed_forms(x, code):
    assert e4m3_encode(x) == code


def test_encode_rejects_out_of_range():
    for bad in (448.5, -500.0, math.inf, math.nan):
        with pytest.raises(ValueError):
            e4m3_encode(bad)


def test_brute_force_nearest_with_ties_to_even():
    table = [(c, e4m3_decode(c)) for c in FINITE]
    rng = np.random.default_rng(11)
    xs = list(rng.uniform(-448, 448, 1500)) + list(rng.uniform(-0.05, 0.05, 1500)) + _midpoints()
    for x in xs:
        best = min(abs(v - x) for _, v in table)
        near = [c for c, v in table if abs(v - x) == best]
        got = e4m3_encode(x)
        if x == 0:
            continue
        # among equally near codes of x's sign, the even mantissa wins
        near = [c for c in near if (c & 0x80) == (0x80 if x < 0 else 0) or e4m3_decode(c) == 0]
        if len(near) > 1:
            near = [c for c in near if (c & 1) == 0]
        assert got in near, (x, got, near)


# ---- the scale rule ---------------------------------------------------------

def test_scale_exponent_closed_form():
    rng = np.random.default_rng(3)
    for amax in list(rng.lognormal(0, 6, 3000)) + [448.0 * 2.0 ** k for k in range(-20, 20)]:
        e = scale_exponent(amax)
        assert amax <= 448.0 * 2.0 ** e and amax > 448.0 * 2.0 ** (e - 1)
        assert 224.0 < amax * 2.0 ** -e <= 448.0
    for k in (-30, -3, 0, 5, 40):
        b = 448.0 * 2.0 ** k
        assert scale_exponent(b) == k                       # exactly at the limit
        assert scale_exponent(math.nextafter(b, math.inf)) == k + 1
        assert scale_exponent(math.nextafter(b, 0.0)) == k
    assert scale_exponent(0.0) == 0
    assert scale_exponent(2.0 ** -140) == -126              # clamped
    assert scale_exponent(1e38) == 118                      # 1e38 / 2^118 = 300.9
    assert scale_exponent(float(np.finfo(np.float32).max)) == 120


def test_quantize_row_codes_and_error():
    rng = np.random.default_rng(5)
    for scale in (1e-6, 0.088, 1.0, 3e4):
        x = rng.standard_normal(128) * scale
        codes, e = quantize_row(x)
        xh = fp8_kv.dequantize_row(codes, e)
        assert np.max(np.abs(xh)) <= 448 * 2.0 ** e
        # half a quantum of the binade, or of the subnormal range
        bound = np.maximum(np.abs(x) * 2.0 ** -4, 2.0 ** (e - 10))
        assert np.all(np.abs(xh - x) <= bound)
        # the row's largest element keeps 3 mantissa bits: relative 2^-4
        i = int(np.argmax(np.abs(x)))
        assert abs(xh[i] - x[i]) <= abs(x[i]) * 2.0 ** -4


# ---- planted mistakes: each fails a pin above --------------------------------

def _truncating(x):
    a = abs(x)
    if a == 0:
        return 0
    _, k = math.frexp(a)
    q = 2.0 ** (max(k - 1, -6) - 3)
    return e4m3_encode(math.copysign(math.floor(a / q) * q, x))


def _fnuz_decode(code):  # bias 8, the other 8-bit E4M3 family
    v = e4m3_decode(code)
    return v / 2 if not math.isnan(v) else v


def test_planted_mistakes_fail():
    with pytest.raises(AssertionError):
        assert _truncating(1.1875) == 0x3A
    ref = torch_decode(ALL).astype(np.float64)
    mine = np.array([_fnuz_decode(c) for c in ALL])
    ok = ~np.isnan(ref)
    assert not np.array_equal(mine[ok], ref[ok])
    with pytest.raises(AssertionError):     # amax * 2^e instead of 2^-e
        e = -scale_exponent(1000.0)
        assert 224.0 < 1000.0 * 2.0 ** -e <= 448.0


# ---- quantized attention within its error bound --------------------------------

def _bound(qr, K, V, scale):
    """Bound on |out_fp8 - out| for one query row: element errors
    |x^ - x| <= 2^-4 |x| + 2^(e - 10) per stored row, score errors
    delta_j <= scale * sum_d |q_d| |dk_jd|, probabilities within exp(+-2 delta)."""
    ek = np.array([scale_exponent(np.max(np.abs(k))) for k in K])
    ev = np.array([scale_exponent(np.max(np.abs(v))) for v in V])
    dk = np.abs(K) * 2.0 ** -4 + 2.0 ** (ek - 10)[:, None]
    dv = np.abs(V) * 2.0 ** -4 + 2.0 ** (ev - 10)[:, None]
    delta = np.max(scale * (dk @ np.abs(qr)))
    s = scale * (K @ qr)
    p = np.exp(s - s.max())
    p /= p.sum()
    return dv.max(axis=0) + (math.exp(2 * delta) - 1) * (p @ np.abs(V))


def test_quantized_attention_within_bound_of_exact():
    hq, hkv, d, S, W = 4, 2, 64, 4, 40
    g = hq // hkv
    exact = OracleSession(hq, hkv, d, S, W)
    quant = OracleSession(hq, hkv, d, S, W, kv_quant="fp8_e4m3")
    rng = np.random.default_rng(21)
    worst = 0.0
    for f in range(12):
        c = 5 if f % 3 == 0 else 1
        q = rng.standard_normal((c, hq, d))
        k = rng.standard_normal((c, hkv, d))
        v = rng.standard_normal((c, hkv, d))
        oe, _ = exact.step(q, k, v)
        oq, _ = quant.step(q, k, v)
        # the bound from the exact retained state (rotated keys, values)
        st = exact.state[0]
        for i in range(c):
            t = exact.length - c + i
            vis = [p for p in sorted(st) if p <= t]
            vis = [p for p in vis if p < S or p > t - W]
            qr = rope_rotate(q[i], t, exact.theta)
            for h in range(hq):
                K = np.stack([st[p][0][h // g] for p in vis])
                V = np.stack([st[p][1][h // g] for p in vis])
                b = _bound(qr[h], K, V, exact.scale)
                err = np.abs(oq[i, h] - oe[i, h])
                assert np.all(err <= b), (f, i, h, float(np.max(err - b)))
                worst = max(worst, float(np.max(err)))
    assert 0 < worst < 0.2  # quantization is visible, and small


def test_quantized_session_on_exactly_representable_values():
    """Rows that are already E4M3 values with amax in (224, 448] (e = 0)
    pass the codec unchanged: with values of that form, the quantized and
    exact sessions agree exactly at position 0 (RoPE angle 0 leaves the key
    unrotated)."""
    rng = np.random.default_rng(2)
    pos_codes = [c for c in FINITE if c < 0x7F]
    d = 16
    def row():
        r = np.array([e4m3_decode(c) for c in rng.choice(pos_codes, d)])
        r *= rng.choice([-1.0, 1.0], d)
        r[0] = 448.0
        return r
    q = rng.standard_normal((1, 2, d)) * 0.01
    k = np.stack([row(), row()])[None]
    v = np.stack([row(), row()])[None]
    a = OracleSession(2, 2, d, 0, 8).step(q, k, v)
    b = OracleSession(2, 2, d, 0, 8, kv_quant="fp8_e4m3").step(q, k, v)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
