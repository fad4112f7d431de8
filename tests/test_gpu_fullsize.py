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
from workload import QWEN3_OMNI as W, device_bank

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
