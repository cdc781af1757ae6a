"""GPU parity of the decode cache path: eva_prefill with a cache, then
eva_cache_append + eva_decode_step, against oracle rows of the same tokens.

Decode of position p must equal row p of a prefill over the whole history
(same window, same summaries); multi-step runs cross chunk boundaries and
wrap the ring several times.  Caches pre-filled with NaN prove that no stale
slot or unused summary row leaks into an output.
"""
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


def oracle_row(qrow, K, V, p, W, C, window=oracle.SLIDING):
    """Oracle output of the query at position p; K, V hold positions 0..p."""
    Ks, Vs = oracle.summaries(K[: p + 1], V[: p + 1], C)
    if window == oracle.SLIDING:
        return oracle.attend_rows(qrow[None], np.array([p]), K[: p + 1], V[: p + 1], Ks, Vs, W, C)[0]
    return oracle.attend_rows_variant(qrow[None], np.array([p]), K[: p + 1], V[: p + 1], Ks, Vs, W, C, window)[0]


def run_sequence(B, H, Hkv, d, W, C, L0, steps, seed, fill=None, use_ws=True, check_every=1, fused=False,
                 window=oracle.SLIDING, dtype=torch.bfloat16):
    """Prefill L0 tokens (if L0 > 0) into a cache, then append + decode `steps`
    tokens (two calls, or the fused call); compare every `check_every`-th
    decode output with the oracle."""
    print(f"decode B{B} H{H}/{Hkv} d{d} W{W} C{C} L0={L0} steps={steps} fill={fill} ws={use_ws} fused={fused} "
          f"{dtype}", flush=True)
    total = L0 + steps
    q, k, v = inputs.qkv(B, H, Hkv, total, d, dtype, seed=seed)
    cache = eva.Cache(B, H, Hkv, d, W, C, max_tokens=total, dtype=dtype, fill=fill, window=window)
    if L0 > 0:
        eva.prefill(q[:, :, :L0].contiguous().cuda(), k[:, :, :L0].contiguous().cuda(),
                    v[:, :, :L0].contiguous().cuda(), W, C, cache=cache, window=window)
        assert cache.n_tok == L0
    k64, v64 = to64(k), to64(v)
    worst = 0.0
    for t in range(steps):
        p = L0 + t
        kn, vn, qn = (t[:, :, p].contiguous().cuda() for t in (k, v, q))
        if fused:
            o = eva.append_decode(cache, qn, kn, vn, use_workspace=use_ws)
        else:
            eva.cache_append(cache, kn, vn)
            o = eva.decode_step(cache, qn, use_workspace=use_ws)
        assert cache.n_tok == p + 1
        if t % check_every and t != steps - 1:
            continue
        torch.cuda.synchronize()
        got = to64(o)
        for b in range(B):
            for h in range(H):
                g = h // (H // Hkv)
                ref = oracle_row(to64(q[b, h, p]), k64[b, g], v64[b, g], p, W, C, window)
                worst = max(worst, assert_parity(got[b, h][None], ref[None], dtype, f"p={p} b{b} h{h}"))
    return cache


def test_decode_after_prefill_matches_next_row():
    run_sequence(2, 8, 2, 128, 64, 16, L0=300, steps=1, seed=21)


@pytest.mark.parametrize("fused", [False, True])
def test_decode_many_steps_cross_chunks_and_ring_wraps(fused):
    # R = 96 slots for W = 64, C = 16: 260 steps wrap the ring ~3 times and
    # complete 16 chunks (and make 16 summaries visible) during decode.
    run_sequence(1, 4, 2, 128, 64, 16, L0=100, steps=260, seed=22, check_every=7, fused=fused)


@pytest.mark.parametrize("fused", [False, True])
def test_decode_from_empty_cache(fused):
    run_sequence(1, 4, 1, 64, 24, 8, L0=0, steps=120, seed=23, check_every=5, fused=fused)


@pytest.mark.parametrize("fused", [False, True])
def test_decode_nan_filled_cache(fused):
    run_sequence(2, 4, 2, 128, 40, 8, L0=77, steps=60, seed=24, fill=float("nan"), check_every=3, fused=fused)


@pytest.mark.parametrize("fused", [False, True])
def test_decode_window_of_one(fused):
    # W = 1: a chunk becomes visible one step after its last token
    run_sequence(1, 4, 2, 128, 1, 8, L0=30, steps=40, seed=28, check_every=1, fused=fused)


@pytest.mark.parametrize("H,Hkv", [(2, 2), (32, 2), (48, 1)])
def test_decode_head_groupings(H, Hkv):
    # G = 1, G = 16 (one full column block), G = 48 (three head groups)
    run_sequence(1, H, Hkv, 128, 48, 16, L0=200, steps=20, seed=25, check_every=6)
    run_sequence(1, H, Hkv, 128, 48, 16, L0=200, steps=20, seed=25, check_every=6, fused=True)


@pytest.mark.parametrize("use_ws", [True, False])
@pytest.mark.parametrize("fused", [False, True])
def test_decode_split_and_unsplit(use_ws, fused):
    # B * Hkv = 2 units: with a workspace the rows are split over many workgroups
    run_sequence(1, 8, 2, 128, 512, 64, L0=3000, steps=3, seed=26, use_ws=use_ws, fused=fused)


@pytest.mark.parametrize("window", [oracle.CHUNK_ALIGNED, oracle.BLOCKED])
@pytest.mark.parametrize("fused", [False, True])
def test_decode_window_variants(window, fused):
    # window / summary sets of the causal variants across chunk completions,
    # block starts and ring wraps (R = 96 for W = 64, C = 16)
    run_sequence(1, 8, 2, 128, 64, 16, L0=150, steps=140, seed=32, check_every=3, fused=fused, window=window)


def test_fused_step_equals_two_calls():
    # same kernels, same arithmetic order: bit-identical outputs and caches
    B, H, Hkv, d, W, C, L0, steps = 2, 8, 2, 128, 64, 16, 150, 70
    q, k, v = inputs.qkv(B, H, Hkv, L0 + steps, d, torch.bfloat16, seed=29)
    caches = []
    outs = []
    for fused in (False, True):
        cache = eva.Cache(B, H, Hkv, d, W, C, max_tokens=L0 + steps, fill=0.0)
        eva.prefill(q[:, :, :L0].contiguous().cuda(), k[:, :, :L0].contiguous().cuda(),
                    v[:, :, :L0].contiguous().cuda(), W, C, cache=cache)
        o = []
        for t in range(steps):
            p = L0 + t
            kn, vn, qn = (x[:, :, p].contiguous().cuda() for x in (k, v, q))
            if fused:
                o.append(eva.append_decode(cache, qn, kn, vn))
            else:
                eva.cache_append(cache, kn, vn)
                o.append(eva.decode_step(cache, qn))
        caches.append(cache)
        outs.append(torch.stack(o))
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])
    n_sum = (L0 + steps) // C
    for name in ("k_ring", "vt_ring"):
        assert torch.equal(getattr(caches[0], name), getattr(caches[1], name)), name
    assert torch.equal(caches[0].k_sum[:, :, :n_sum], caches[1].k_sum[:, :, :n_sum])
    assert torch.equal(caches[0].vt_sum, caches[1].vt_sum)


def test_cache_summaries_match_oracle():
    B, H, Hkv, d, W, C, L0, steps = 1, 2, 2, 64, 32, 8, 50, 90
    cache = run_sequence(B, H, Hkv, d, W, C, L0=L0, steps=steps, seed=27, check_every=1000)
    q, k, v = inputs.qkv(B, H, Hkv, L0 + steps, d, torch.bfloat16, seed=27)
    n_sum = oracle.visible_summaries(L0 + steps - 1, W, C)
    for g in range(Hkv):
        rK, rV = oracle.summaries(k[0, g], v[0, g], C)
        got_k = to64(cache.k_sum[0, g, :n_sum])
        # [S_max/32, d, 32] tiles -> [S_max, d]
        got_v = to64(cache.vt_sum[0, g].permute(0, 2, 1).reshape(-1, d)[:n_sum])
        assert_parity(got_k, rK[:n_sum], torch.bfloat16, "k_sum")
        assert_parity(got_v, rV[:n_sum], torch.bfloat16, "vt_sum")


def test_decode_workload_full_size_sampled():
    w = inputs.DECODE_BF16
    print(f"full-size {w.name}", flush=True)
    L0 = w.context
    _, k, v = inputs.qkv(w.B, 1, w.Hkv, L0 + 1, w.d, w.dtype, seed=w.seed)
    # history queries only shape the history's prefill outputs, which decode
    # never reads; draw them on the device
    gen = torch.Generator(device="cuda").manual_seed(w.seed)
    qh = torch.randn(w.B, w.H, L0, w.d, generator=gen, device="cuda").to(w.dtype)
    q_new = inputs.normal((w.B, w.H, w.d), w.seed + 100, w.dtype)
    cache = eva.Cache(w.B, w.H, w.Hkv, w.d, w.W, w.C, max_tokens=L0 + 1, dtype=w.dtype)
    eva.prefill(qh, k[:, :, :L0].contiguous().cuda(), v[:, :, :L0].contiguous().cuda(), w.W, w.C, cache=cache)
    del qh
    eva.cache_append(cache, k[:, :, L0].contiguous().cuda(), v[:, :, L0].contiguous().cuda())
    o = eva.decode_step(cache, q_new.cuda())
    torch.cuda.synchronize()
    p = L0
    assert oracle.visible_summaries(p, w.W, w.C) == 60
    got = to64(o)
    for b in (0, 17, w.B - 1):
        for g in (0, w.Hkv - 1):
            K64, V64 = to64(k[b, g]), to64(v[b, g])
            Ks, Vs = oracle.summaries(K64, V64, w.C)
            heads = list(range(g * (w.H // w.Hkv), (g + 1) * (w.H // w.Hkv)))
            ref = oracle.attend_rows(to64(q_new[b, heads]), np.full(len(heads), p), K64, V64, Ks, Vs, w.W, w.C)
            assert_parity(got[b, heads], ref, w.dtype, f"b{b} g{g}")


def test_prefill_with_cache_matches_parts_on_a_stream():
    # eva_prefill with a cache, called on a non-default stream and followed
    # at once (no host sync) by a decode that reads the cache, gives the
    # bytes of the separate calls
    B, H, Hkv, L, d, W, C = 2, 4, 2, 700, 128, 100, 64
    print(f"prefill+cache on a stream B{B} H{H}/{Hkv} L{L} d{d} W{W} C{C}", flush=True)
    q, k, v = (t.cuda() for t in inputs.qkv(B, H, Hkv, L, d, torch.bfloat16, seed=43))
    qn = inputs.normal((B, H, d), 44, torch.bfloat16).cuda()
    a = eva.Cache(B, H, Hkv, d, W, C, max_tokens=L + 1, fill=0.0)
    b = eva.Cache(B, H, Hkv, d, W, C, max_tokens=L + 1, fill=0.0)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        O, Ks, Vs = eva.prefill(q, k, v, W, C, cache=a, return_summaries=True)
        snap = {name: getattr(a, name).clone() for name in ("k_ring", "vt_ring", "k_sum", "vt_sum")}
        oa = eva.decode_step(a, qn)
    torch.cuda.current_stream().wait_stream(s)
    Ks2, Vs2 = eva.build_summaries(k, v, C)
    eva.cache_fill(b, k, v, Ks2, Vs2)
    O2 = eva.prefill_attention(q, k, v, Ks2, Vs2, W, C)
    ob = eva.decode_step(b, qn)
    torch.cuda.synchronize()
    assert torch.equal(O, O2) and torch.equal(Ks, Ks2) and torch.equal(Vs, Vs2)
    for name, t in snap.items():
        assert torch.equal(t, getattr(b, name)), name
    assert torch.equal(oa, ob)


# ---- fp32 caches (their own decode kernel, fp32 matrix-core products):
# held to the fp32 bound, 1e-5 row-normwise relative error
F32_DECODE = [
    # B, H, Hkv, d, W, C, L0, steps, check_every, fill, window
    (2, 8, 2, 128, 64, 16, 300, 1, 1, None, oracle.SLIDING),
    (1, 4, 2, 128, 64, 16, 100, 260, 7, None, oracle.SLIDING),       # chunk completions, ring wraps
    (2, 4, 2, 64, 40, 8, 77, 60, 3, float("nan"), oracle.SLIDING),   # stale slots must not leak
    (1, 4, 2, 128, 1, 8, 30, 40, 1, None, oracle.SLIDING),           # W = 1
    (1, 48, 1, 128, 48, 16, 200, 20, 6, None, oracle.SLIDING),       # G = 48: three head groups
    (1, 4, 1, 64, 24, 8, 0, 120, 5, None, oracle.SLIDING),           # from an empty cache
    (1, 8, 2, 128, 64, 16, 150, 140, 3, None, oracle.CHUNK_ALIGNED),
    (1, 8, 2, 128, 64, 16, 150, 140, 3, None, oracle.BLOCKED),
]


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("shape", F32_DECODE)
def test_decode_fp32(shape, fused):
    B, H, Hkv, d, W, C, L0, steps, every, fill, window = shape
    run_sequence(B, H, Hkv, d, W, C, L0=L0, steps=steps, seed=34, fill=fill, check_every=every, fused=fused,
                 window=window, dtype=torch.float32)


def test_noalloc_fp32_cache():
    # the allocation-free fused step on an fp32 cache (no split partials):
    # the bytes of eva_append_decode
    B, H, Hkv, d, W, C, L0 = 2, 8, 2, 128, 64, 16, 300
    q, k, v = inputs.qkv(B, H, Hkv, L0 + 1, d, torch.float32, seed=35)
    outs = []
    for noalloc in (False, True):
        cache = eva.Cache(B, H, Hkv, d, W, C, max_tokens=L0 + 1, dtype=torch.float32)
        eva.prefill(q[:, :, :L0].contiguous().cuda(), k[:, :, :L0].contiguous().cuda(),
                    v[:, :, :L0].contiguous().cuda(), W, C, cache=cache)
        qn, kn, vn = (x[:, :, L0].contiguous().cuda() for x in (q, k, v))
        outs.append(eva.append_decode_noalloc(cache, qn, kn, vn) if noalloc else eva.append_decode(cache, qn, kn, vn))
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])


# ---- stochastic (random-feature) summaries through decode: the cache
# builds, for every chunk an append completes, the paper's single-sample
# summary with the counter-based draw eva_rf_noise gives that chunk, so the
# decoded rows equal the oracle's rows over summaries_rf of the whole history
# with the oracle's own draws (same counters, computed independently)
def test_rf_noise_matches_oracle_generator():
    for d in (64, 128):
        eps = eva.rf_noise(3, 5, 37, d, seed=2 ** 40 + 7)
        torch.cuda.synchronize()
        ref = oracle.rf_noise(15, 37, d, seed=2 ** 40 + 7).reshape(3, 5, 37, d)
        assert_parity(to64(eps), ref, torch.float32, f"rf noise d{d}")


def rf_oracle_row(qrow, K, V, p, W, C, lam, seed, seq):
    """Oracle row at position p over the stochastic summaries of positions 0..p
    of sequence-head `seq` (its draws from the counter-based generator)."""
    n_chunks = (p + 1) // C
    eps = oracle.rf_noise(seq + 1, max(n_chunks, 1), K.shape[1], seed)[seq, :n_chunks]
    Ks, Vs = oracle.summaries_rf(K[: p + 1], V[: p + 1], eps, C, lam)
    return oracle.attend_rows(qrow[None], np.array([p]), K[: p + 1], V[: p + 1], Ks, Vs, W, C)[0]


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("fused", [False, True])
def test_decode_rf_summaries(fused, dtype):
    B, H, Hkv, d, W, C, L0, steps, lam, seed = 2, 8, 2, 128, 48, 16, 150, 90, 0.3, 1234567
    print(f"rf decode fused={fused} {dtype}", flush=True)
    q, k, v = inputs.qkv(B, H, Hkv, L0 + steps, d, dtype, seed=36)
    cache = eva.Cache(B, H, Hkv, d, W, C, max_tokens=L0 + steps, dtype=dtype, fill=float("nan"), rf_lambda=lam,
                      rf_seed=seed)
    kp, vp = k[:, :, :L0].contiguous().cuda(), v[:, :, :L0].contiguous().cuda()
    eps = eva.rf_noise(B, Hkv, L0 // C, d, seed)
    Ks, Vs = eva.build_summaries_rf(kp, vp, eps, C, lam=lam)
    eva.cache_fill(cache, kp, vp, Ks, Vs)
    k64, v64 = to64(k), to64(v)
    for t in range(steps):
        p = L0 + t
        kn, vn, qn = (x[:, :, p].contiguous().cuda() for x in (k, v, q))
        if fused:
            o = eva.append_decode(cache, qn, kn, vn)
        else:
            eva.cache_append(cache, kn, vn)
            o = eva.decode_step(cache, qn)
        if t % 11 and t != steps - 1:
            continue
        torch.cuda.synchronize()
        got = to64(o)
        for b in range(B):
            for h in (0, H - 1):
                g = h // (H // Hkv)
                ref = rf_oracle_row(to64(q[b, h, p]), k64[b, g], v64[b, g], p, W, C, lam, seed, b * Hkv + g)
                assert_parity(got[b, h][None], ref[None], dtype, f"p={p} b{b} h{h}")
    # every summary the cache holds is the stochastic one of its chunk
    n = (L0 + steps) // C
    for b in range(B):
        for g in range(Hkv):
            eps_o = oracle.rf_noise(b * Hkv + g + 1, n, d, seed)[b * Hkv + g]
            rK, rV = oracle.summaries_rf(k64[b, g, : n * C], v64[b, g, : n * C], eps_o, C, lam)
            got_v = to64(cache.vt_sum[b, g].permute(0, 2, 1).reshape(-1, d)[:n])
            assert_parity(to64(cache.k_sum[b, g, :n]), rK, dtype, "k_sum")
            assert_parity(got_v, rV, dtype, "vt_sum")
