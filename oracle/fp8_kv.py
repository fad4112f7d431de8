"""FP8 (OCP E4M3) KV cache: the codec and the per-token scale rule.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).  Nothing here is shared
with the library; its quantizer is compared with this one code by code.

What it follows (Metronome, arXiv 2607.02640): per-token KV reduction --
techniques that shrink what each resident token stores -- is orthogonal to the
window, which bounds which tokens stay resident, and the two compose (§4.1,
closing remark; §6, "Attention, long context, and KV reduction").  The paper
fixes no format, so everything below is a reading:

* Format: the OCP 8-bit floating-point E4M3 encoding -- sign, 4 exponent bits
  with bias 7, 3 mantissa bits; exponent field 0 holds subnormals
  (m * 2^-9); no infinities; S.1111.111 is NaN, so the largest finite
  magnitude is 1.75 * 2^8 = 448.  Rounding is to nearest, ties to the even
  mantissa; a value that rounds to zero keeps its sign (0x80 for negatives).
* Scale: one power of two per (token, KV head) and tensor (K or V):
  2^e with e the smallest integer such that amax <= 448 * 2^e, where amax is
  the largest magnitude of the row, clamped to [-126, 127]; e = 0 for an
  all-zero row.  The scaled row x * 2^-e is then exact and its largest
  magnitude lies in (224, 448], so no code overflows.  The pool stores the
  biased byte e + 127.
* What is quantized: the rotated key (the cache holds keys after RoPE, as
  the bf16 cache does) and the value, each in the precision the kernel has
  them in (float32: the rotation is rounded to float32 first, since the code
  is an integer decided by floating point); attention then reads the exact
  dequantized values code * 2^e.

Parity status: pinned (tests/test_fp8_pins.py) against torch's float8_e4m3fn
conversion (every code, every rounding midpoint, random values), the format's
closed forms (448, smallest normal / subnormal, ties to even), brute-force
nearest-value search, the scale rule's closed form, and the error bound of
quantized attention against the exact float64 oracle.  The rows are encoded
by ``e4m3_encode_array``, the same steps on arrays, pinned element by element
against the scalar ``e4m3_encode``.
"""
from __future__ import annotations

import math
from typing import Tuple

import numpy as np

E4M3_MAX = 448.0
E4M3_BIAS = 7
SCALE_BIAS = 127  # stored exponent byte = e + 127


def e4m3_decode(code: int) -> float:
    """Value of an E4M3 code (NaN for S.1111.111)."""
    code = int(code) & 0xFF
    sign = -1.0 if code & 0x80 else 1.0
    ex = (code >> 3) & 0xF
    man = code & 0x7
    if ex == 0xF and man == 0x7:
        return math.nan
    if ex == 0:
        return sign * man * 2.0 ** (1 - E4M3_BIAS - 3)       # subnormal: m * 2^-9
    return sign * (1.0 + man / 8.0) * 2.0 ** (ex - E4M3_BIAS)


def e4m3_encode(x: float) -> int:
    """Round a finite |x| <= 448 to the nearest E4M3 code, ties to even."""
    x = float(x)
    if not math.isfinite(x) or abs(x) > E4M3_MAX:
        raise ValueError("outside the finite E4M3 range")
    sign = 0x80 if math.copysign(1.0, x) < 0 else 0
    a = abs(x)
    if a == 0.0:
        return sign
    _, k = math.frexp(a)            # a = f * 2^k, f in [0.5, 1)
    ex = max(k - 1, 1 - E4M3_BIAS)  # binade exponent; subnormals share 2^-6's quantum
    quantum = 2.0 ** (ex - 3)
    n = round(a / quantum)          # exact ratio; Python rounds halves to even
    if n == 0:
        return sign
    mag = n * quantum
    # re-derive the fields from the rounded magnitude (n may have carried into
    # the next binade, n == 16)
    _, k2 = math.frexp(mag)
    ex2 = k2 - 1
    if ex2 < 1 - E4M3_BIAS:         # subnormal
        return sign | int(mag / 2.0 ** (1 - E4M3_BIAS - 3))
    man = int(mag / 2.0 ** (ex2 - 3)) - 8
    return sign | ((ex2 + E4M3_BIAS) << 3) | man


_DECODE_TABLE = None


def e4m3_decode_array(codes: np.ndarray) -> np.ndarray:
    """e4m3_decode of every code (a lookup in the 256 values it defines)."""
    global _DECODE_TABLE
    if _DECODE_TABLE is None:
        _DECODE_TABLE = np.array([e4m3_decode(c) for c in range(256)], dtype=np.float64)
    return _DECODE_TABLE[np.asarray(codes, dtype=np.uint8)]


def e4m3_encode_array(x: np.ndarray) -> np.ndarray:
    """e4m3_encode of every element, the same steps on arrays: the binade
    exponent from frexp, the quantum 2^(e - 3) (2^-9 below the normal range),
    the ratio rounded half to even (exact: a power-of-two division), then the
    fields of the rounded magnitude."""
    x = np.asarray(x, dtype=np.float64)
    if not np.all(np.isfinite(x)) or np.any(np.abs(x) > E4M3_MAX):
        raise ValueError("outside the finite E4M3 range")
    sign = np.where(np.signbit(x), 0x80, 0).astype(np.int64)
    a = np.abs(x)
    _, k = np.frexp(a)
    ex = np.maximum(k - 1, 1 - E4M3_BIAS)
    mag = np.rint(np.ldexp(a, -(ex - 3))) * np.ldexp(1.0, ex - 3)
    _, k2 = np.frexp(mag)
    ex2 = k2 - 1
    sub = mag < 2.0 ** (1 - E4M3_BIAS)
    sub_code = np.ldexp(mag, 9).astype(np.int64)
    norm_code = ((ex2 + E4M3_BIAS) << 3) + (np.ldexp(mag, -(ex2 - 3)).astype(np.int64) - 8)
    code = np.where(sub, sub_code, norm_code)
    return (sign | code).astype(np.uint8)


def scale_exponent(amax: float) -> int:
    """Smallest e with amax <= 448 * 2^e, clamped to [-126, 127]; 0 for 0."""
    amax = float(amax)
    if amax == 0.0:
        return 0
    if not math.isfinite(amax) or amax < 0:
        raise ValueError("amax must be finite and >= 0")
    # 448 * 2^e >= amax  <=>  e >= log2(amax / 448); search from frexp's guess
    _, k = math.frexp(amax / E4M3_MAX)
    e = k - 1
    while E4M3_MAX * 2.0 ** e < amax:
        e += 1
    while E4M3_MAX * 2.0 ** (e - 1) >= amax:
        e -= 1
    return min(max(e, -126), 127)


def quantize_row(x: np.ndarray) -> Tuple[np.ndarray, int]:
    """Codes (uint8[D]) and scale exponent e of one (token, head) row."""
    x = np.asarray(x, dtype=np.float64)
    e = scale_exponent(float(np.max(np.abs(x))) if x.size else 0.0)
    return e4m3_encode_array(np.ldexp(x, -e)), e


def dequantize_row(codes: np.ndarray, e: int) -> np.ndarray:
    return e4m3_decode_array(codes) * 2.0 ** e


def roundtrip_row(x: np.ndarray, as_float32: bool) -> np.ndarray:
    """What the cache returns for a stored row: quantize, then dequantize.
    ``as_float32`` first rounds the row to float32 (the kernel's precision for
    the rotated key; a no-op for bf16 / float32 inputs)."""
    x = np.asarray(x, dtype=np.float64)
    if as_float32:
        x = x.astype(np.float32).astype(np.float64)
    codes, e = quantize_row(x)
    return dequantize_row(codes, e)


def quantize_heads(x: np.ndarray, as_float32: bool) -> Tuple[np.ndarray, np.ndarray]:
    """Codes [H, D] and stored exponent bytes [H] (e + 127) of one token's
    rows x[H, D]."""
    x = np.asarray(x, dtype=np.float64)
    if as_float32:
        x = x.astype(np.float32).astype(np.float64)
    codes = np.zeros(x.shape, dtype=np.uint8)
    ebytes = np.zeros(x.shape[0], dtype=np.uint8)
    for h in range(x.shape[0]):
        c, e = quantize_row(x[h])
        codes[h] = c
        ebytes[h] = e + SCALE_BIAS
    return codes, ebytes
