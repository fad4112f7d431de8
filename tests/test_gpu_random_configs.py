"""GPU parity over seeded random configurations: pool element type, head dim,
GQA group, sinks, window, chunk limit, session count, prefill pass size and
decode kernel are drawn per case, and a few ragged frames from empty sessions
(so windows fill, wrap and sink blocks fill part way) are compared with the
float64 oracle on every output.  Each case prints its configuration first."""
import random

import pytest

from tests._gpu_util import Harness, make_pool, say

pytestmark = pytest.mark.gpu


def _config(seed):
    rnd = random.Random(1000 + seed)
    dtype = rnd.choice(["f32", "bf16", "bf16", "fp8"])
    d = 128 if dtype == "fp8" else rnd.choice([64, 128])
    hkv = rnd.choice([1, 2])
    g = rnd.choice([1, 2, 4, 8])
    S = rnd.choice([0, 1, 4, 17])
    W = rnd.choice([1, 7, 16, 33, 100, 300])
    cmax = rnd.choice([1, 5, 25, 40, 64])
    n = rnd.randint(1, 6)
    frames = rnd.randint(4, 7)
    rows = rnd.choice([0, 128, 256])
    kernel = rnd.choice([0, 0, 1, 2])
    return dict(dtype=dtype, d=d, hkv=hkv, g=g, S=S, W=W, cmax=cmax, n=n, frames=frames,
                rows=rows, kernel=kernel, seed=seed)


@pytest.mark.parametrize("seed", range(48))
def test_random_configuration_against_oracle(seed):
    c = _config(seed)
    say(f"random config {c}")
    R = -(-(c["W"] + c["cmax"] - 1) // 16) * 16
    blocks = c["n"] * (-(-c["S"] // 16) + R // 16) + 4
    pool = make_pool(n_layers=2, hq=c["hkv"] * c["g"], hkv=c["hkv"], d=c["d"], S=c["S"],
                     W=c["W"], cmax=c["cmax"], max_sessions=c["n"], n_blocks=blocks,
                     dtype=c["dtype"])
    if c["rows"]:
        pool.set_prefill_pass_rows(c["rows"])
    kernel = c["kernel"]
    if kernel == 1 and c["dtype"] == "fp8":
        kernel = 0   # the FP8 cache has no vector decode kernel
    if kernel == 2 and not (c["dtype"] in ("bf16", "fp8") and c["d"] == 128):
        kernel = 0   # the matrix decode kernel needs a bf16 / fp8 pool with D = 128
    if kernel:
        pool.set_decode_kernel(kernel)
    h = Harness(pool, n_sessions=c["n"], n_layers=2, hq=c["hkv"] * c["g"], hkv=c["hkv"],
                d=c["d"], S=c["S"], W=c["W"], dtype=c["dtype"], seed=seed)
    rnd = random.Random(seed)
    for f in range(c["frames"]):
        chunk = [rnd.randint(1, c["cmax"]) for _ in range(c["n"])]
        dec = [rnd.randint(0, 3) for _ in range(c["n"])]
        h.frame(chunk, dec, n_split=rnd.choice([0, 0, 1, 2, 5]),
                use_frame_step=rnd.random() < 0.7)
    say(f"max err {h.max_err:.2e}")
