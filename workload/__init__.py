"""Seeded synthetic workloads shared by the tests, the bench and the oracle's
callers.

This module holds shapes, seeds and random draws only -- none of the method's
arithmetic (no masks, no RoPE, no attention, no index maps).  Both the HIP
path and the float64 oracle consume exactly the tensors produced here.

Workload shapes stand in for the paper's real-audio sessions (Metronome,
arXiv 2607.02640, §5 setup: LibriSpeech / spoken-question clips streamed to
omni models); no dataset item is used.  Each workload is an attention-only
frame stream: per frame a chunk of C tokens is prefilled, then tau single-token
decode steps run (§2, "The task model").
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    n_sessions: int
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str                 # "f32" or "bf16" (KV cache and q/k/v/out)
    n_sink: int
    window: Optional[int]      # None = unbounded (vanilla) policy
    chunk: Tuple[int, int]     # inclusive range of chunk tokens per frame
    n_decode: Tuple[int, int]  # inclusive range of decode steps per frame
    frames: int
    frame_period_s: float
    act_scale: float = 1.0     # q/k/v ~ N(0, 1) * act_scale
    block_size: int = 16
    rope_theta: float = 1.0e6
    workload_id: int = 0

    @property
    def max_chunk(self) -> int:
        return self.chunk[1]

    @property
    def g(self) -> int:
        return self.n_q_heads // self.n_kv_heads


# Tiny single-layer parity check: 4 sessions, GQA 8/2, D = 64, fp32, S = 4,
# W = 128, 8-token chunks then 4 decodes, 40 frames (the window wraps).
TINY = Workload("tiny-gqa8x2-d64-f32", 4, 1, 8, 2, 64, "f32", 4, 128,
                (8, 8), (4, 4), 40, 0.08, 1.0, rope_theta=1.0e4, workload_id=1)

# Moshi-like temporal transformer: 32 layers, MHA 32/32, D = 128, bf16,
# 64 sessions, 80 ms frames of 1 appended token + 1 decode, S = 4, W = 2048,
# 3750 frames (5 min); activations scaled by 1/sqrt(D).
MOSHI = Workload("moshi-like-l32-h32-d128-bf16", 64, 32, 32, 32, 128, "bf16", 4, 2048,
                 (1, 1), (1, 1), 3750, 0.08, 1.0 / np.sqrt(128.0), rope_theta=1.0e4,
                 workload_id=2)

# Qwen3-Omni-30B-A3B-shaped attention: 48 layers, GQA 32/4, D = 128, bf16,
# 128 sessions, 1.5 s frames of a 25-token chunk + 16 decodes, S = 4,
# W = 4096, 200 frames.
QWEN3_OMNI = Workload("qwen3-omni-like-l48-h32x4-d128-bf16", 128, 48, 32, 4, 128, "bf16",
                      4, 4096, (25, 25), (16, 16), 200, 1.5, workload_id=3)

# Unbounded-vs-windowed pool stress at the Qwen3-Omni shapes: 128 sessions,
# 300 frames of 41 tokens; windowed arm S = 4, W = 4096.
POOL_STRESS_WINDOWED = Workload("pool-stress-windowed", 128, 48, 32, 4, 128, "bf16",
                                4, 4096, (25, 25), (16, 16), 300, 1.5, workload_id=4)
POOL_STRESS_UNBOUNDED = Workload("pool-stress-unbounded", 128, 48, 32, 4, 128, "bf16",
                                 0, None, (25, 25), (16, 16), 300, 1.5, workload_id=4)

# MiniCPM-o-4.5 backbone (Qwen3-8B-like): 36 layers, GQA 32/8, D = 128,
# bf16, 256 sessions, chunk ~ U{10..40}, decodes ~ U{8..24}, S = 4, W = 2048.
MINICPM_O = Workload("minicpm-o-like-l36-h32x8-d128-bf16", 256, 36, 32, 8, 128, "bf16",
                     4, 2048, (10, 40), (8, 24), 300, 1.0, workload_id=5)

ALL = {w.name: w for w in (TINY, MOSHI, QWEN3_OMNI, POOL_STRESS_WINDOWED,
                           POOL_STRESS_UNBOUNDED, MINICPM_O)}


def session_rng(workload_id: int, session_uid: int, stream: int = 0) -> np.random.Generator:
    """Independent PCG64 stream per (workload, session, stream)."""
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([workload_id, session_uid, stream])))


def draw_qkv(rng: np.random.Generator, n_layers: int, n_tok: int, hq: int, hkv: int,
             d: int, scale: float = 1.0):
    """q [n_layers, n_tok, hq, d], k and v [n_layers, n_tok, hkv, d], float32,
    i.i.d. N(0, 1) * scale."""
    q = (rng.standard_normal((n_layers, n_tok, hq, d)) * scale).astype(np.float32)
    k = (rng.standard_normal((n_layers, n_tok, hkv, d)) * scale).astype(np.float32)
    v = (rng.standard_normal((n_layers, n_tok, hkv, d)) * scale).astype(np.float32)
    return q, k, v


def frame_lengths(w: Workload, rng: np.random.Generator) -> Tuple[int, int]:
    """(chunk tokens, decode steps) of one session-frame."""
    c = int(rng.integers(w.chunk[0], w.chunk[1] + 1))
    t = int(rng.integers(w.n_decode[0], w.n_decode[1] + 1))
    return c, t


def device_bank(shape, dtype, device, seed: int, scale: float = 1.0):
    """A seeded N(0, 1) * scale bank drawn on the given torch device with
    torch's own generator (used for full-size runs; the oracle side copies the
    same tensor to the host)."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    t = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    if scale != 1.0:
        t.mul_(scale)
    return t.to(dtype)
