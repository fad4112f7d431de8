"""The allocation-free decode entry point (mtn_attend_decode_noalloc): the
same kernels as mtn_attend_decode with the split partials in the library's
static device array instead of the pool's workspace.  Two calls in a row (the
second over a smaller batch) give bit-identical results to mtn_attend_decode
with the same split; a forced split past the array is refused."""
import numpy as np
import pytest
import torch

import paper_2607_02640_amd as mtn
from tests._gpu_util import Harness, make_pool, say

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,d,hq,hkv", [("bf16", 128, 16, 2), ("f32", 64, 8, 2),
                                            ("fp8", 128, 16, 2)])
def test_noalloc_decode_matches_decode(dtype, d, hq, hkv):
    say(f"noalloc decode {dtype} d{d} {hq}/{hkv}")
    n, L, S, W = 4, 2, 4, 90
    R = -(-(W + 7) // 16) * 16
    pool = make_pool(n_layers=L, hq=hq, hkv=hkv, d=d, S=S, W=W, cmax=8, max_sessions=n,
                     n_blocks=n * (1 + R // 16), dtype=dtype)
    h = Harness(pool, n_sessions=n, n_layers=L, hq=hq, hkv=hkv, d=d, S=S, W=W, dtype=dtype)
    for f in range(12):   # fill and wrap the windows
        h.frame([8] * n, [2] * n, check=False)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    gen = torch.Generator(device="cuda").manual_seed(5)
    for batch, n_split in ((list(range(n)), 5), ([2, 0], 3), ([1], 0), ([3, 1, 2], 64)):
        sids = [h.sids[i] for i in batch]
        m = len(sids)
        pool.plan_begin(sids, [1] * m)
        for l in range(L):
            k = torch.randn((m, hkv, d), generator=gen, device="cuda").to(tdt)
            v = torch.randn((m, hkv, d), generator=gen, device="cuda").to(tdt)
            q = torch.randn((m, hq, d), generator=gen, device="cuda").to(tdt)
            pool.frame_append_kv(l, k, v)
            o_ref, o_new = torch.empty_like(q), torch.empty_like(q)
            lse_ref = torch.empty((m, hq), dtype=torch.float32, device="cuda")
            lse_new = torch.empty_like(lse_ref)
            pool.attend_decode(l, q, o_ref, lse_ref, n_split=n_split)
            split_ref = pool.last_split()
            pool.attend_decode_noalloc(l, q, o_new, lse_new, n_split=split_ref)
            assert pool.last_split() == split_ref
            torch.cuda.synchronize()
            assert torch.equal(o_ref, o_new), (batch, n_split, l)
            assert torch.equal(lse_ref, lse_new), (batch, n_split, l)
        pool.plan_commit()
        say(f"batch {batch} split {n_split}: identical")
    # a forced split whose partials pass the static array (4 Mi floats) is refused
    big = make_pool(n_layers=1, hq=32, hkv=4, d=128, S=4, W=256, cmax=1, max_sessions=256,
                    n_blocks=256 * 17, dtype="bf16")
    sids = [big.session_open() for _ in range(256)]
    big.plan_begin(sids, [1] * 256)
    k = torch.zeros((256, 4, 128), dtype=torch.bfloat16, device="cuda")
    q = torch.zeros((256, 32, 128), dtype=torch.bfloat16, device="cuda")
    big.frame_append_kv(0, k, k)
    o = torch.empty_like(q)
    with pytest.raises(mtn.MtnError) as e:
        big.attend_decode_noalloc(0, q, o, n_split=64)   # 256*32*64*130 floats > 4 Mi
    assert e.value.code == mtn.MTN_ERR_INVALID_ARG
    big.attend_decode_noalloc(0, q, o, n_split=2)        # 2.1 Mi floats: fits
    torch.cuda.synchronize()
    big.plan_commit()
