"""GPU parity on shapes drawn at random from fixed seeds: the hand-picked
shapes of the other tests pin each boundary on purpose; these spread over
the space of (B, G, H_kv, L, d, W, C, window variant, dtype) so that a
combination nobody thought of is still compared element by element with the
fp64 oracle: the prefill, its backward, decode after a prefill (prompt
length, steps, fused or separate append, NaN-filled caches), ragged
generation (per-sequence prompt lengths, active masks, caches that fill
up), and stochastic summaries with the prefill over them.  Every case is
deterministic (its seed is its index)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2511_00576_amd import eva, inputs
from parity import assert_grad_parity, assert_parity, to64

pytestmark = pytest.mark.gpu

VARIANTS = (oracle.SLIDING, oracle.CHUNK_ALIGNED, oracle.BLOCKED, oracle.NONCAUSAL)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    eva._lib.load()


def prefill_case(i):
    r = np.random.RandomState(1000 + i)
    Hkv = int(r.choice([1, 2, 3]))
    G = int(r.choice([1, 2, 3, 4, 5, 8, 16]))
    while G * Hkv > 16:
        Hkv -= 1
    B = int(r.choice([1, 2]))
    d = int(r.choice([64, 128]))
    L = int(r.randint(1, 601))
    W = int(r.choice([1, 2, 7, 16, 31, 32, 33, 64, 100, 257, 600, 1000]))
    C = int(r.choice([1, 2, 3, 8, 16, 24, 32, 64, 100, 128, 300]))
    var = VARIANTS[int(r.randint(0, 4))]
    dtype = torch.float32 if i % 4 == 3 else torch.bfloat16
    if i >= 24:
        # G > 1 with a window beyond 512 keys: the bf16 kernel's 8-wave,
        # 64-key-block configuration, over several query tiles
        G, Hkv, B = int(r.choice([2, 4, 8])), int(r.choice([1, 2])), 1
        L, W = int(r.randint(520, 1201)), int(r.choice([513, 600, 777, 1000]))
        dtype = torch.bfloat16
    return B, G * Hkv, Hkv, L, d, W, C, var, dtype


@pytest.mark.parametrize("i", range(28))
def test_prefill_random_shape(i):
    B, H, Hkv, L, d, W, C, var, dtype = prefill_case(i)
    print(f"random prefill {i}: B{B} H{H}/{Hkv} L{L} d{d} W{W} C{C} window {var} {dtype}", flush=True)
    q, k, v = inputs.qkv(B, H, Hkv, L, d, dtype=dtype, seed=2000 + i)
    O = eva.prefill(q.cuda(), k.cuda(), v.cuda(), W, C, window=var)
    torch.cuda.synchronize()
    ref = oracle.prefill_variant(q, k, v, W, C, var)
    assert_parity(to64(O), ref, dtype, f"case {i}")


def backward_case(i):
    r = np.random.RandomState(3000 + i)
    Hkv = int(r.choice([1, 2]))
    G = int(r.choice([1, 2, 4, 8]))
    B = int(r.choice([1, 2]))
    d = int(r.choice([64, 128]))
    L = int(r.randint(1, 401))
    W = int(r.choice([1, 5, 16, 33, 64, 130, 500]))
    C = int(r.choice([1, 3, 8, 16, 32, 64, 128]))
    var = VARIANTS[int(r.randint(0, 4))]
    return B, G * Hkv, Hkv, L, d, W, C, var


@pytest.mark.parametrize("i", range(12))
def test_backward_random_shape(i):
    B, H, Hkv, L, d, W, C, var = backward_case(i)
    print(f"random backward {i}: B{B} H{H}/{Hkv} L{L} d{d} W{W} C{C} window {var}", flush=True)
    q, k, v = inputs.qkv(B, H, Hkv, L, d, torch.bfloat16, seed=4000 + i)
    dO = inputs.normal((B, H, L, d), 5000 + i, torch.bfloat16)
    qc, kc, vc, gc = (t.cuda() for t in (q, k, v, dO))
    O, lse, Ks, Vs, O_lo = eva.prefill_forward(qc, kc, vc, W, C, residual=True, window=var)
    dQ, dK, dV = eva.prefill_backward(qc, kc, vc, Ks, Vs, O, lse, gc, W, C, O_lo=O_lo, window=var)
    torch.cuda.synchronize()
    rq, rk, rv = oracle.backward(q, k, v, dO, W, C, variant=var)
    tq, tk, tv = oracle.backward_terms(q, k, v, dO, W, C, variant=var)
    for g, rf, t, name in ((dQ, rq, tq, "dQ"), (dK, rk, tk, "dK"), (dV, rv, tv, "dV")):
        assert_grad_parity(to64(g), rf, t, f"case {i} {name}")


CAUSAL = (oracle.SLIDING, oracle.CHUNK_ALIGNED, oracle.BLOCKED)


def decode_case(i):
    r = np.random.RandomState(6000 + i)
    Hkv = int(r.choice([1, 2]))
    G = int(r.choice([1, 2, 4, 8]))
    B = int(r.choice([1, 2, 3]))
    d = int(r.choice([64, 128]))
    W = int(r.choice([1, 2, 7, 16, 33, 100, 256]))
    C = int(r.choice([1, 3, 4, 16, 24, 64]))
    L0 = int(r.randint(0, 401))
    steps = int(r.randint(1, 41))
    var = CAUSAL[int(r.randint(0, 3))]
    fused = bool(r.randint(0, 2))
    fill = float("nan") if r.randint(0, 2) else None
    dtype = torch.float32 if i % 4 == 3 else torch.bfloat16
    return B, G * Hkv, Hkv, d, W, C, L0, steps, var, fused, fill, dtype


@pytest.mark.parametrize("i", range(16))
def test_decode_random_shape(i):
    # prefill of L0 tokens into a cache (none when L0 = 0), then `steps`
    # appended tokens, each decoded and compared with the oracle's row of
    # the whole sequence; caches filled with NaN must not leak stale slots
    from test_gpu_decode import run_sequence

    B, H, Hkv, d, W, C, L0, steps, var, fused, fill, dtype = decode_case(i)
    print(f"random decode {i}", flush=True)
    run_sequence(B, H, Hkv, d, W, C, L0=L0, steps=steps, seed=7000 + i, fill=fill, fused=fused, window=var,
                 dtype=dtype, check_every=max(1, steps // 8))


def ragged_case(i):
    r = np.random.RandomState(8000 + i)
    Hkv = int(r.choice([1, 2]))
    G = int(r.choice([1, 2, 4]))
    B = int(r.randint(1, 6))
    d = int(r.choice([64, 128]))
    W = int(r.choice([1, 5, 16, 48, 100]))
    C = int(r.choice([1, 4, 8, 16, 32]))
    lens = [int(x) for x in r.randint(0, 301, size=B)]
    steps = int(r.randint(1, 41))
    var = CAUSAL[int(r.randint(0, 3))]
    fused = bool(r.randint(0, 2))
    use_ws = bool(r.randint(0, 2))
    fill = float("nan") if r.randint(0, 2) else None
    dtype = torch.float32 if i % 4 == 3 else torch.bfloat16
    # some caches hold fewer tokens than the sequences reach: full
    # sequences stop growing and keep decoding their last position
    max_tokens = max(lens) + steps - (int(r.randint(0, 20)) if i % 3 == 0 else 0)
    active = r.rand(steps, B) < 0.75  # seeded active masks
    return B, G * Hkv, Hkv, d, W, C, lens, steps, var, fused, use_ws, fill, dtype, max(max_tokens, 1), active


@pytest.mark.parametrize("i", range(16))
def test_ragged_random_shape(i):
    from test_gpu_generate import run_steps

    B, H, Hkv, d, W, C, lens, steps, var, fused, use_ws, fill, dtype, max_tokens, active = ragged_case(i)
    print(f"random ragged {i} max_tokens={max_tokens}", flush=True)
    run_steps(B, H, Hkv, d, W, C, lens=lens, steps=steps, seed=9000 + i, fill=fill,
              active_fn=lambda t, b: active[t, b], use_ws=use_ws, max_tokens=max_tokens,
              check_every=max(1, steps // 8), fused=fused, window=var, dtype=dtype)


def rf_case(i):
    r = np.random.RandomState(10000 + i)
    Hkv = int(r.choice([1, 2]))
    G = int(r.choice([1, 2, 4, 8]))
    B = int(r.choice([1, 2]))
    d = int(r.choice([64, 128]))
    C = int(r.choice([1, 4, 16, 24, 64]))
    L = int(r.randint(2 * C, 2 * C + 500))
    W = int(r.choice([1, 7, 32, 100, 257]))
    var = VARIANTS[int(r.randint(0, 4))]
    lam = float(r.choice([0.0, 0.05, 0.1, 0.5]))
    dtype = torch.float32 if i % 3 == 2 else torch.bfloat16
    return B, G * Hkv, Hkv, L, d, W, C, var, lam, dtype


@pytest.mark.parametrize("i", range(12))
def test_prefill_rf_random_shape(i):
    # stochastic summaries (draws passed in) and the fused prefill over them,
    # every output element against the oracle's rows over its own summaries
    B, H, Hkv, L, d, W, C, var, lam, dtype = rf_case(i)
    print(f"random rf prefill {i}: B{B} H{H}/{Hkv} L{L} d{d} W{W} C{C} window {var} lam {lam} {dtype}", flush=True)
    q, k, v = inputs.qkv(B, H, Hkv, L, d, dtype, seed=11000 + i)
    eps = inputs.normal((B, Hkv, L // C, d), 12000 + i)
    qc, kc, vc = q.cuda(), k.cuda(), v.cuda()
    Ks, Vs = eva.build_summaries_rf(kc, vc, eps.cuda(), C, lam=lam)
    O = eva.prefill_attention(qc, kc, vc, Ks, Vs, W, C, window=var)
    torch.cuda.synchronize()
    rows = np.arange(L, dtype=np.int64)
    G = H // Hkv
    for b in range(B):
        for g in range(Hkv):
            rK, rV = oracle.summaries_rf(k[b, g], v[b, g], eps[b, g], C, lam=lam)
            assert_parity(to64(Ks[b, g]), rK, dtype, f"case {i} Ksum b{b} g{g}")
            assert_parity(to64(Vs[b, g]), rV, dtype, f"case {i} Vsum b{b} g{g}")
            for h in range(g * G, (g + 1) * G):
                ref = oracle.attend_rows_variant(to64(q[b, h]), rows, to64(k[b, g]), to64(v[b, g]), rK, rV, W, C,
                                                 var)
                assert_parity(to64(O[b, h]), ref, dtype, f"case {i} b{b} h{h}")
