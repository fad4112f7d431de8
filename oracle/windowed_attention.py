"""Float64 oracle of windowed-KV frame attention with pinned sinks.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

What it computes (Metronome, arXiv 2607.02640):

* §4.1 and App. A ("Window half", "Sink half"): a session keeps its first S
  tokens pinned plus its most recent W tokens; the attention mask of a query at
  absolute position t admits keys in [0, S) together with the window that ends
  at t, always under causality (k <= t).
* §4.1: positions are absolute; eviction removes old keys from memory but
  never renumbers the ones that remain.
* §2, "The task model": each frame appends (prefills) a chunk of new tokens and
  then decodes up to tau tokens, one at a time.
* App. A: visiting the sink keys first (or in any other order) is exact,
  because the softmax is order-invariant; each key counts once.

Readings where the paper is silent or ambiguous:

* Window endpoint.  The printed interval [t-W, t] holds W+1 positions.  The
  default reading admits exactly W window keys including t, i.e. (t-W, t], so
  that "retain the last W tokens" is exactly the set a decode step reads.  The
  literal W+1 reading is available with ``literal_window=True``.
* Chunk prefill: every chunk query has its own window (the mask is a function
  of t); the whole chunk is inserted before any of its queries attends.
* RoPE: rotate-half form with base theta, applied to k (at append) and q (at
  attention) at the token's absolute position.  The paper names no variant, so
  the choice is a reading; the implementation of the chosen variant is pinned
  against its complex-exponential definition in the tests.
* GQA: query head h reads KV head floor(h / G), G = Hq / Hkv (contiguous
  groups).  Softmax scale 1/sqrt(D) unless given.
* Unbounded policy (the paper's vanilla baseline): no window, no eviction;
  the sink count is irrelevant.

Nothing is rounded: inputs are widened to float64 exactly (bf16 and fp32 are
both exactly representable) and every step runs in float64.  The one
exception is opt-in: ``kv_quant="fp8_e4m3"`` stores every K/V row through the
E4M3 codec of ``fp8_kv`` (per-token KV reduction, §4.1 / §6), and attention
reads the exact dequantized values.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from .fp8_kv import roundtrip_row

UNBOUNDED = None  # window value that means "no window" (the vanilla policy)


# ---------------------------------------------------------------------------
# Visibility and retention (§4.1 mask; App. A sink pinning / window freeing)
# ---------------------------------------------------------------------------

def visible_positions(t: int, n_sink: int, window: Optional[int],
                      literal_window: bool = False) -> List[int]:
    """Sorted key positions a query at absolute position ``t`` may attend to.

    vis(t) = { k : 0 <= k <= t  and  (k < S  or  k in window(t)) }, where the
    window is (t-W, t] (default reading) or [t-W, t] (literal reading).  With
    no window every causal key is visible.
    """
    if t < 0:
        raise ValueError("position must be >= 0")
    out = []
    for k in range(t + 1):
        if window is None:
            out.append(k)
            continue
        lo = t - window if literal_window else t - window + 1
        if k < n_sink or k >= lo:
            out.append(k)
    return out


def retained_positions(length: int, n_sink: int, window: Optional[int]) -> set:
    """Ret(L): positions a session of length L keeps resident.

    The first S positions plus the last W positions (all positions when there
    is no window).
    """
    if window is None:
        return set(range(length))
    return {p for p in range(length) if p < n_sink or p >= length - window}


def evicted_range(old_len: int, new_len: int, n_sink: int,
                  window: Optional[int]) -> Tuple[int, int]:
    """Half-open range of positions that leave the retained set when a session
    grows from ``old_len`` to ``new_len`` tokens (empty when lo >= hi).

    A position p >= S is resident while p >= L - W, so growing the length
    evicts every p >= S with p < new_len - W that was resident before, i.e.
    p >= old_len - W.  Positions that were appended and evicted within the
    same growth step are included.
    """
    if window is None:
        return (0, 0)
    lo = max(n_sink, old_len - window)
    hi = max(lo, new_len - window)
    return (lo, hi)


# ---------------------------------------------------------------------------
# Rotary position embedding at absolute positions (§4.1 logical growth)
# ---------------------------------------------------------------------------

def rope_frequencies(head_dim: int, theta: float) -> np.ndarray:
    """omega_i = theta ** (-2 i / D) for i < D/2, in float64."""
    if head_dim % 2:
        raise ValueError("head_dim must be even")
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(np.float64(theta), -2.0 * i / head_dim)


def rope_rotate(x: np.ndarray, pos: int, theta: float) -> np.ndarray:
    """Rotate-half RoPE of ``x[..., D]`` at absolute position ``pos``.

    For i < D/2 with angle a = pos * omega_i:
        x'_i       = x_i cos a - x_{i+D/2} sin a
        x'_{i+D/2} = x_{i+D/2} cos a + x_i sin a
    """
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    h = d // 2
    ang = np.float64(pos) * rope_frequencies(d, theta)
    c, s = np.cos(ang), np.sin(ang)
    lo, hi = x[..., :h], x[..., h:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)


# ---------------------------------------------------------------------------
# One query row against an explicit key set
# ---------------------------------------------------------------------------

def attend_row(q_rot: np.ndarray, keys: np.ndarray, vals: np.ndarray,
               scale: float) -> Tuple[np.ndarray, float, float]:
    """Softmax attention of one rotated query row over explicit keys/values.

    Returns (output[D], log-sum-exp of the scaled scores, sum of the weights).
    """
    s = scale * (keys @ q_rot)
    m = np.max(s)
    e = np.exp(s - m)
    z = np.sum(e)
    p = e / z
    return p @ vals, float(m + math.log(z)), float(np.sum(p))


# ---------------------------------------------------------------------------
# Session state machine
# ---------------------------------------------------------------------------

class OracleSession:
    """One session's retained KV across ``n_layers`` layers.

    The state of each layer is a dict ``pos -> (K_rot[Hkv, D], V[Hkv, D])``
    holding exactly Ret(L).  Usage mirrors the per-frame structure: ``begin(C)``
    reserves the next C absolute positions, ``layer_step`` inserts that layer's
    K/V for them and attends every new query, ``commit()`` advances L and
    prunes every layer back to Ret(L).  ``step`` does all three for one layer.
    """

    def __init__(self, n_q_heads: int, n_kv_heads: int, head_dim: int,
                 n_sink: int, window: Optional[int], theta: float = 10000.0,
                 scale: Optional[float] = None, n_layers: int = 1,
                 literal_window: bool = False, check_psum: bool = True,
                 kv_quant: Optional[str] = None):
        if n_q_heads % n_kv_heads:
            raise ValueError("n_q_heads must be a multiple of n_kv_heads")
        self.hq, self.hkv, self.d = n_q_heads, n_kv_heads, head_dim
        self.g = n_q_heads // n_kv_heads
        self.n_sink = 0 if window is None else n_sink
        self.window = window
        self.theta = theta
        self.scale = 1.0 / math.sqrt(head_dim) if scale is None else scale
        self.n_layers = n_layers
        self.literal = literal_window
        self.check_psum = check_psum
        if kv_quant not in (None, "fp8_e4m3"):
            raise ValueError("kv_quant must be None or 'fp8_e4m3'")
        self.kv_quant = kv_quant
        self.length = 0
        self.state: List[Dict[int, Tuple[np.ndarray, np.ndarray]]] = [
            {} for _ in range(n_layers)]
        self._pending: Optional[int] = None
        self._done = set()
        self.last_evicted = (0, 0)

    # -- frame structure -------------------------------------------------
    def begin(self, n_tok: int) -> List[int]:
        if self._pending is not None:
            raise RuntimeError("a step is already open")
        if n_tok < 1:
            raise ValueError("n_tok must be >= 1")
        self._pending = n_tok
        self._done = set()
        return list(range(self.length, self.length + n_tok))

    def layer_step(self, layer: int, q: np.ndarray, k: np.ndarray,
                   v: np.ndarray, attend: bool = True):
        """Insert this layer's K/V for the open positions, then attend.

        q: [C, Hq, D], k and v: [C, Hkv, D].  Returns (out[C, Hq, D],
        lse[C, Hq]) or None when ``attend`` is False (append only).
        """
        c = self._pending
        if c is None:
            raise RuntimeError("no open step")
        q = np.asarray(q, dtype=np.float64).reshape(c, self.hq, self.d)
        k = np.asarray(k, dtype=np.float64).reshape(c, self.hkv, self.d)
        v = np.asarray(v, dtype=np.float64).reshape(c, self.hkv, self.d)
        st = self.state[layer]
        base = self.length
        # Insert every chunk token first: each query then sees the earlier
        # tokens of its own chunk (causal inside the chunk).
        for i in range(c):
            kr = rope_rotate(k[i], base + i, self.theta)
            vi = v[i].copy()
            if self.kv_quant == "fp8_e4m3":
                # the cache holds what the quantized pool returns: each
                # (token, head) row of the rotated key and of the value
                # through the E4M3 codec with its own power-of-two scale
                kr = np.stack([roundtrip_row(kr[h], True) for h in range(self.hkv)])
                vi = np.stack([roundtrip_row(vi[h], True) for h in range(self.hkv)])
            st[base + i] = (kr, vi)
        self._done.add(layer)
        if not attend:
            return None
        out = np.zeros((c, self.hq, self.d))
        lse = np.zeros((c, self.hq))
        for i in range(c):
            t = base + i
            vis = visible_positions(t, self.n_sink, self.window, self.literal)
            missing = [p for p in vis if p not in st]
            assert not missing, f"visible positions not resident: {missing[:5]}"
            kmat = np.stack([st[p][0] for p in vis])  # [n, Hkv, D]
            vmat = np.stack([st[p][1] for p in vis])
            qr = rope_rotate(q[i], t, self.theta)     # [Hq, D]
            for h in range(self.hq):
                kv = h // self.g
                o, l, psum = attend_row(qr[h], kmat[:, kv, :], vmat[:, kv, :],
                                        self.scale)
                if self.check_psum:
                    assert abs(psum - 1.0) < 1e-12, psum
                out[i, h] = o
                lse[i, h] = l
        return out, lse

    def commit(self) -> Tuple[int, int]:
        c = self._pending
        if c is None:
            raise RuntimeError("no open step")
        if self._done != set(range(self.n_layers)):
            raise RuntimeError("commit before every layer was appended")
        old = self.length
        self.length += c
        keep = retained_positions(self.length, self.n_sink, self.window)
        for st in self.state:
            for p in [p for p in st if p not in keep]:
                del st[p]
            assert set(st) == keep, "retained set differs from Ret(L)"
        self._pending = None
        self.last_evicted = evicted_range(old, self.length, self.n_sink,
                                          self.window)
        return self.last_evicted

    def step(self, q, k, v, layer: int = 0):
        """begin + layer_step + commit for a single-layer session."""
        if self.n_layers != 1:
            raise RuntimeError("step() is for single-layer sessions")
        self.begin(np.asarray(k).shape[0])
        res = self.layer_step(layer, q, k, v)
        self.commit()
        return res

    def frame(self, chunk, decodes: Sequence, layer: int = 0):
        """One frame of a single-layer session: a chunk prefill, then one step
        per decode entry.  ``chunk`` and each decode entry are (q, k, v)
        triples.  Returns (chunk_out, chunk_lse, [(dec_out, dec_lse), ...])."""
        co, cl = self.step(*chunk, layer=layer)
        dec = [self.step(*d, layer=layer) for d in decodes]
        return co, cl, dec


# ---------------------------------------------------------------------------
# Full-history dense-mask attention (no pruning) for the pruning pins
# ---------------------------------------------------------------------------

def dense_mask_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                         n_sink: int, window: Optional[int], theta: float,
                         scale: Optional[float] = None,
                         literal_window: bool = False) -> Tuple[np.ndarray, np.ndarray]:
    """Attention over a session's whole history with an explicit T x T mask.

    q: [T, Hq, D], k/v: [T, Hkv, D] for positions 0..T-1.  Nothing is evicted;
    the mask M[t, k] = (k <= t) and (k < S or k in window(t)) alone decides
    what each query sees.  Used to show that the pruned state machine never
    drops a key some query needs.
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    t_len, hq, d = q.shape
    hkv = k.shape[1]
    g = hq // hkv
    sc = 1.0 / math.sqrt(d) if scale is None else scale
    pos = np.arange(t_len)
    qr = np.stack([rope_rotate(q[t], t, theta) for t in range(t_len)])
    kr = np.stack([rope_rotate(k[t], t, theta) for t in range(t_len)])
    tt, kk = np.meshgrid(pos, pos, indexing="ij")
    mask = kk <= tt
    if window is not None:
        lo = tt - window if literal_window else tt - window + 1
        mask &= (kk < n_sink) | (kk >= lo)
    out = np.zeros_like(q)
    lse = np.zeros((t_len, hq))
    for h in range(hq):
        s = sc * qr[:, h, :] @ kr[:, h // g, :].T
        s = np.where(mask, s, -np.inf)
        m = s.max(axis=1, keepdims=True)
        e = np.exp(s - m)
        z = e.sum(axis=1, keepdims=True)
        out[:, h, :] = (e / z) @ v[:, h // g, :]
        lse[:, h] = (m + np.log(z))[:, 0]
    return out, lse
