"""GPU parity of the EVA prefill backward (bf16, every window variant) against the
fp64 oracle's gradients (themselves pinned by finite differences and by
autograd of exact attention).

The training forward (eva_prefill_forward) must give the inference forward's
output; the backward's dQ, dK, dV are compared row-normwise (per query row of
dQ, per key row of dK and dV).  Small windows and chunks make a wrongly masked
row change a key's gradient by a large fraction, and spiked keys on the window
and chunk edges make it change by O(1).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2511_00576_amd import eva, inputs
from parity import assert_grad_parity, to64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    eva._lib.load()


def run_backward(q, k, v, dO, W, C, residual=True, window=oracle.SLIDING):
    """Training forward + backward.  With `residual` the forward keeps its
    output's rounding residual and the backward's row dots D = dO . O are
    exact; without it D comes from the bf16 O."""
    qc, kc, vc, gc = (t.cuda() for t in (q, k, v, dO))
    if residual:
        O, lse, Ks, Vs, O_lo = eva.prefill_forward(qc, kc, vc, W, C, residual=True, window=window)
    else:
        (O, lse, Ks, Vs), O_lo = eva.prefill_forward(qc, kc, vc, W, C, window=window), None
    dQ, dK, dV = eva.prefill_backward(qc, kc, vc, Ks, Vs, O, lse, gc, W, C, O_lo=O_lo, window=window)
    torch.cuda.synchronize()
    return O, lse, dQ, dK, dV


SHAPES = [
    # B, H, Hkv, L, d, W, C
    (1, 2, 1, 300, 64, 40, 16),     # G = 2
    (2, 8, 2, 517, 128, 64, 24),    # G = 4, ragged tail (517 % 24 != 0)
    (1, 4, 4, 400, 128, 7, 4),      # small window and chunk: masks matter
    (1, 2, 1, 250, 128, 1, 5),      # W = 1
    (1, 2, 2, 120, 64, 200, 16),    # W >= L: no summaries
    (1, 2, 2, 100, 128, 10, 128),   # C > L: no chunk
    (2, 2, 1, 17, 128, 5, 3),       # shorter than one block
    (1, 16, 2, 300, 128, 48, 32),   # G = 8
    (1, 4, 2, 400, 128, 96, 64),    # chunk of 4 rows per thread in the per-chunk pass
    (1, 2, 1, 333, 64, 50, 32),     # d = 64, one row per thread in the per-chunk pass
    (1, 2, 2, 260, 128, 32, 16),    # d = 128, one row per thread in the per-chunk pass
    (1, 2, 1, 400, 64, 80, 64),     # d = 64, one wave per chunk, 8 rows per lane
    (1, 2, 1, 520, 64, 100, 128),   # d = 64, one wave per chunk, 16 rows per lane
    (1, 16, 1, 2048, 128, 128, 32), # G = 16: 16 query-range splits of each summary tile
    (1, 8, 1, 4096, 128, 256, 64),  # 16 splits, one wave per chunk, 16 rows per lane
]


@pytest.mark.parametrize("shape", SHAPES)
def test_backward_matches_oracle(shape):
    B, H, Hkv, L, d, W, C = shape
    print(f"backward B{B} H{H}/{Hkv} L{L} d{d} W{W} C{C}", flush=True)
    q, k, v = inputs.qkv(B, H, Hkv, L, d, torch.bfloat16, seed=60)
    dO = inputs.normal((B, H, L, d), 61, torch.bfloat16)
    O, lse, dQ, dK, dV = run_backward(q, k, v, dO, W, C)
    # the training forward is the inference forward
    O_inf = eva.prefill(q.cuda(), k.cuda(), v.cuda(), W, C)
    assert torch.equal(O, O_inf)
    rq, rk, rv = oracle.backward(q, k, v, dO, W, C)
    tq, tk, tv = oracle.backward_terms(q, k, v, dO, W, C)
    errs = [assert_grad_parity(to64(g), r, t, name)
            for g, r, t, name in ((dQ, rq, tq, "dQ"), (dK, rk, tk, "dK"), (dV, rv, tv, "dV"))]
    print("row-normwise errors dQ %.2e dK %.2e dV %.2e" % tuple(errs), flush=True)


def test_backward_lse_is_the_log_denominator():
    # with V = identity rows (d >= L) the output row is the softmax itself, so
    # lse must make exp(logit - lse) sum to one: sum over the row's weights of
    # O recovers 1, and log of the oracle's denominator matches
    B, H, Hkv, L, d, W, C = 1, 2, 2, 64, 128, 16, 4
    q, k, _ = inputs.qkv(B, H, Hkv, L, d, torch.bfloat16, seed=62)
    v = torch.zeros(B, Hkv, L, d, dtype=torch.bfloat16)
    v[0, :, torch.arange(L), torch.arange(L)] = 1.0
    O, lse, _, _ = eva.prefill_forward(q.cuda(), k.cuda(), v.cuda(), W, C)
    torch.cuda.synchronize()
    # row n attends window keys and summaries: the window part of O is the
    # window weights exp(l - lse); check them against logits from q, k
    q64, k64, lse64 = to64(q), to64(k), to64(lse)
    for h in range(H):
        for n in (0, 5, 20, 40, 63):
            lo = max(0, n - W + 1)
            logits = q64[0, h, n] @ k64[0, h, lo:n + 1].T / np.sqrt(d)
            np.testing.assert_allclose(np.exp(logits - lse64[0, h, n]), to64(O)[0, h, n, lo:n + 1] -
                                       0.0, rtol=0, atol=2e-2)


def test_backward_full_size_sampled():
    # the LLM workload at full size; the oracle checks two (batch, kv head)
    # groups exactly (each group's dK, dV depend on that group alone)
    w = inputs.LLM_BF16
    print(f"backward full-size {w.name}", flush=True)
    q, k, v = inputs.workload_qkv(w)
    dO = inputs.normal((w.B, w.H, w.L, w.d), w.seed + 7, w.dtype)
    _, _, dQ, dK, dV = run_backward(q, k, v, dO, w.W, w.C)
    G = w.H // w.Hkv
    for b, g in ((0, 0), (w.B - 1, w.Hkv - 1)):
        hs = slice(g * G, (g + 1) * G)
        args = (q[b:b + 1, hs], k[b:b + 1, g:g + 1], v[b:b + 1, g:g + 1], dO[b:b + 1, hs], w.W, w.C)
        rq, rk, rv = oracle.backward(*args)
        tq, tk, tv = oracle.backward_terms(*args)
        errs = [assert_grad_parity(to64(x), r, t, f"{name} b{b} g{g}")
                for x, r, t, name in ((dQ[b:b + 1, hs], rq, tq, "dQ"), (dK[b:b + 1, g:g + 1], rk, tk, "dK"),
                                      (dV[b:b + 1, g:g + 1], rv, tv, "dV"))]
        print("b%d g%d row-normwise errors dQ %.2e dK %.2e dV %.2e" % ((b, g) + tuple(errs)), flush=True)


@pytest.mark.parametrize("alpha", [3.0, 1.2, 0.6])
@pytest.mark.parametrize("shape", [(1, 4, 2, 400, 128, 7, 4), (1, 2, 1, 300, 64, 40, 16), (1, 8, 2, 600, 128, 96, 32)])
def test_backward_spiked_edges(shape, alpha):
    # keys on the window's first and last positions, the token before the
    # window and chunk last tokens spiked: with alpha 3 a spike takes all of
    # a row's weight, so dV of a spike key is the sum of dO over exactly the
    # rows that see it; with alpha 1.2 and 0.6 it takes a part, so dQ and dK
    # of the spike keys depend on the same row sets.  (At alpha 3, rows
    # dominated by a summary of several spiked keys have logits near 80; the
    # bf16 storage of the summary keys then moves such a row's logits by
    # ~|q| |khat| 2^-9, about 0.01, which the fp64 summaries of the oracle do
    # not have, so at that alpha only dV, whose rows do not depend on the
    # logits' last bits, is held to the bound.)
    B, H, Hkv, L, d, W, C = shape
    anchors = [n for n in range(W, L, max(1, (L - W) // 23))] + [L - 1]
    pos = inputs.window_edge_positions(L, W, C, anchors)
    print(f"backward spikes B{B} H{H}/{Hkv} L{L} d{d} W{W} C{C} alpha {alpha} keys {len(pos)}", flush=True)
    q, k, v = inputs.spike_at_qkv(B, H, Hkv, L, d, pos, (), C, torch.bfloat16, seed=63, alpha=alpha)
    dO = inputs.normal((B, H, L, d), 64, torch.bfloat16)
    _, _, dQ, dK, dV = run_backward(q, k, v, dO, W, C)
    rq, rk, rv = oracle.backward(q, k, v, dO, W, C)
    tq, tk, tv = oracle.backward_terms(q, k, v, dO, W, C)
    checks = ((dV, rv, tv, "dV"),) if alpha >= 3.0 else ((dQ, rq, tq, "dQ"), (dK, rk, tk, "dK"), (dV, rv, tv, "dV"))
    errs = [assert_grad_parity(to64(g), r, t, name) for g, r, t, name in checks]
    print("row-normwise errors " + " ".join("%s %.2e" % (c[3], e) for c, e in zip(checks, errs)), flush=True)


def test_backward_full_size_gqa_sampled():
    # the GQA workload (G = 4) at full size; the oracle checks two
    # (batch, kv head) groups exactly: dQ of their four query heads, dK, dV
    w = inputs.GQA_BF16
    print(f"backward full-size {w.name}", flush=True)
    q, k, v = inputs.workload_qkv(w)
    dO = inputs.normal((w.B, w.H, w.L, w.d), w.seed + 7, w.dtype)
    _, _, dQ, dK, dV = run_backward(q, k, v, dO, w.W, w.C)
    G = w.H // w.Hkv
    for b, g in ((0, 0), (w.B - 1, w.Hkv - 1)):
        hs = slice(g * G, (g + 1) * G)
        args = (q[b:b + 1, hs], k[b:b + 1, g:g + 1], v[b:b + 1, g:g + 1], dO[b:b + 1, hs], w.W, w.C)
        rq, rk, rv = oracle.backward(*args)
        tq, tk, tv = oracle.backward_terms(*args)
        errs = [assert_grad_parity(to64(x), r, t, f"{name} b{b} g{g}")
                for x, r, t, name in ((dQ[b:b + 1, hs], rq, tq, "dQ"), (dK[b:b + 1, g:g + 1], rk, tk, "dK"),
                                      (dV[b:b + 1, g:g + 1], rv, tv, "dV"))]
        print("b%d g%d row-normwise errors dQ %.2e dK %.2e dV %.2e" % ((b, g) + tuple(errs)), flush=True)


@pytest.mark.parametrize("shape", [SHAPES[1], SHAPES[2], SHAPES[7]])
def test_backward_without_output_residual(shape):
    # D from the bf16 output alone: dV does not depend on D and is held row by
    # row; dQ and dK rows move by the rounding of O inside D (about
    # 2^-8 |dO| |O| |k| / sqrt(d), which an fp64 emulation of exactly that
    # rounding reproduces), so they are held to the tensor-wide bound
    B, H, Hkv, L, d, W, C = shape
    print(f"backward without residual B{B} H{H}/{Hkv} L{L} d{d} W{W} C{C}", flush=True)
    q, k, v = inputs.qkv(B, H, Hkv, L, d, torch.bfloat16, seed=60)
    dO = inputs.normal((B, H, L, d), 61, torch.bfloat16)
    O, _, dQ, dK, dV = run_backward(q, k, v, dO, W, C, residual=False)
    O_r, _, _, _, _ = run_backward(q, k, v, dO, W, C, residual=True)
    assert torch.equal(O, O_r)
    rq, rk, rv = oracle.backward(q, k, v, dO, W, C)
    assert_grad_parity(to64(dV), rv, oracle.backward_terms(q, k, v, dO, W, C)[2], "dV")
    for g, r, name in ((dQ, rq, "dQ"), (dK, rk, "dK")):
        err = float(np.abs(to64(g) - r).max()) / float(np.abs(r).max())
        assert err <= 2e-2, f"{name}: max abs error {err:.3e} x max |ref| > 2e-2"


VARIANTS = [oracle.CHUNK_ALIGNED, oracle.BLOCKED, oracle.NONCAUSAL]
VARIANT_SHAPES = [
    # B, H, Hkv, L, d, W, C
    (1, 4, 2, 400, 128, 7, 4),      # small window and chunk: masks matter
    (2, 8, 2, 517, 128, 64, 24),    # G = 4, ragged tail; chunk not dividing the window
    (1, 2, 1, 300, 64, 40, 16),     # d = 64
    (1, 2, 2, 333, 128, 96, 32),    # blocks of 96 rows (three workgroup tiles of keys)
    (2, 2, 1, 17, 128, 5, 3),       # shorter than one block
    (1, 2, 2, 120, 64, 200, 16),    # W >= L: one block, no prefix summaries
]


@pytest.mark.parametrize("window", VARIANTS)
@pytest.mark.parametrize("shape", VARIANT_SHAPES)
def test_backward_variants_match_oracle(shape, window):
    # the window variants of the ablation: each row's window and summaries
    # move (chunk-aligned start, blocks, whole blocks with summaries on both
    # sides), so the rows that see a key or a summary are different sets
    B, H, Hkv, L, d, W, C = shape
    print(f"backward variant {window} B{B} H{H}/{Hkv} L{L} d{d} W{W} C{C}", flush=True)
    q, k, v = inputs.qkv(B, H, Hkv, L, d, torch.bfloat16, seed=65)
    dO = inputs.normal((B, H, L, d), 66, torch.bfloat16)
    O, lse, dQ, dK, dV = run_backward(q, k, v, dO, W, C, window=window)
    O_inf = eva.prefill(q.cuda(), k.cuda(), v.cuda(), W, C, window=window)
    assert torch.equal(O, O_inf)
    rq, rk, rv = oracle.backward(q, k, v, dO, W, C, variant=window)
    tq, tk, tv = oracle.backward_terms(q, k, v, dO, W, C, variant=window)
    errs = [assert_grad_parity(to64(g), r, t, name)
            for g, r, t, name in ((dQ, rq, tq, "dQ"), (dK, rk, tk, "dK"), (dV, rv, tv, "dV"))]
    print("row-normwise errors dQ %.2e dK %.2e dV %.2e" % tuple(errs), flush=True)


@pytest.mark.parametrize("window", VARIANTS)
def test_backward_variants_spiked_edges(window):
    # spikes on the keys that bound the windows and chunks of each variant
    # (alpha 1.2: a spike takes a part of its rows' weight, so a key counted
    # by the wrong row set moves dQ, dK and dV by O(1))
    B, H, Hkv, L, d, W, C = 1, 4, 2, 400, 128, 24, 8
    anchors = [n for n in range(W, L, 17)] + [L - 1]
    pos = sorted(set(inputs.window_edge_positions(L, W, C, anchors)) |
                 {m for m in range(0, L, W)} | {min(L - 1, m + W - 1) for m in range(0, L, W)})
    print(f"backward variant {window} spikes keys {len(pos)}", flush=True)
    q, k, v = inputs.spike_at_qkv(B, H, Hkv, L, d, pos, (), C, torch.bfloat16, seed=67, alpha=1.2)
    dO = inputs.normal((B, H, L, d), 68, torch.bfloat16)
    _, _, dQ, dK, dV = run_backward(q, k, v, dO, W, C, window=window)
    rq, rk, rv = oracle.backward(q, k, v, dO, W, C, variant=window)
    tq, tk, tv = oracle.backward_terms(q, k, v, dO, W, C, variant=window)
    errs = [assert_grad_parity(to64(g), r, t, name)
            for g, r, t, name in ((dQ, rq, tq, "dQ"), (dK, rk, tk, "dK"), (dV, rv, tv, "dV"))]
    print("row-normwise errors dQ %.2e dK %.2e dV %.2e" % tuple(errs), flush=True)
