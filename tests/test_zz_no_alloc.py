"""The allocation-free fused decode step (eva_append_decode_noalloc) against
the fused step with a caller workspace (eva_append_decode), through the C
ABI: two calls in a row, the second on a smaller cache, each on a pair of
identical caches.  Both shapes split their rows over several workgroups, so
the partials really go through the library's fixed device array; the second
call reads only slots it wrote itself, so any stale slot of the first call
would show."""
import numpy as np
import pytest
import torch

import oracle
from paper_2511_00576_amd import eva, inputs
from parity import assert_parity, to64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    eva._lib.load()


def _pair(B, H, Hkv, d, W, C, L0, seed):
    q, k, v = inputs.qkv(B, H, Hkv, L0 + 1, d, torch.bfloat16, seed=seed)
    caches = []
    for _ in range(2):
        c = eva.Cache(B, H, Hkv, d, W, C, max_tokens=L0 + 1, fill=float("nan"))
        eva.prefill(q[:, :, :L0].contiguous().cuda(), k[:, :, :L0].contiguous().cuda(),
                    v[:, :, :L0].contiguous().cuda(), W, C, cache=c)
        caches.append(c)
    new = tuple(t[:, :, L0].contiguous().cuda() for t in (q, k, v))
    return caches, new, (q, k, v)


@pytest.mark.parametrize("order", ["large_then_small"])
def test_noalloc_matches_workspace_call(order):
    shapes = [
        # B, H, Hkv, d, W, C, L0: (b, kv head) units 32 and 2, rows split 5 and 3 ways
        (4, 32, 8, 128, 512, 128, 2000, 81),
        (1, 8, 2, 64, 256, 64, 1000, 82),
    ]
    for B, H, Hkv, d, W, C, L0, seed in shapes:
        print(f"noalloc B{B} H{H}/{Hkv} d{d} W{W} C{C} L0={L0}", flush=True)
        (ca, cb), (qn, kn, vn), (q, k, v) = _pair(B, H, Hkv, d, W, C, L0, seed)
        assert ca.workspace() is not None, "shape must split its rows"
        o_ref = eva.append_decode(ca, qn, kn, vn)
        o = torch.full_like(qn, float("nan"))
        eva.append_decode_noalloc(cb, qn, kn, vn, out=o)
        torch.cuda.synchronize()
        assert cb.n_tok == ca.n_tok == L0 + 1
        assert torch.equal(o, o_ref), "allocation-free step differs from the workspace step"
        for name in ("k_ring", "vt_ring", "k_sum", "vt_sum"):
            a, b = getattr(ca, name), getattr(cb, name)
            assert torch.equal(torch.nan_to_num(a, nan=7.0), torch.nan_to_num(b, nan=7.0)), name
        # and both against the oracle's row L0
        k64, v64 = to64(k), to64(v)
        got = to64(o)
        for b in range(B):
            for h in (0, H - 1):
                g = h // (H // Hkv)
                Ks, Vs = oracle.summaries(k64[b, g], v64[b, g], C)
                ref = oracle.attend_rows(to64(q[b, h, L0])[None], np.array([L0]), k64[b, g], v64[b, g], Ks, Vs,
                                         W, C)
                assert_parity(got[b, h][None], ref, torch.bfloat16, f"b{b} h{h}")
