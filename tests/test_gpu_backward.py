"""GPU parity of the EVA prefill backward (bf16, sliding window) against the
fp64 oracle's gradients (themselves pinned by finite differences and by
autograd of exact attention).

The training forward (eva_prefill_forward) must give the inference forward's
output; the backward's dQ, dK, dV are compared normwise per tensor.  Small
windows and chunks make a wrongly masked row change a key's gradient by a
large fraction.
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


def run_backward(q, k, v, dO, W, C):
    qc, kc, vc, gc = (t.cuda() for t in (q, k, v, dO))
    O, lse, Ks, Vs = eva.prefill_forward(qc, kc, vc, W, C)
    dQ, dK, dV = eva.prefill_backward(qc, kc, vc, Ks, Vs, O, lse, gc, W, C)
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
    errs = [assert_grad_parity(to64(g), r, name) for g, r, name in ((dQ, rq, "dQ"), (dK, rk, "dK"), (dV, rv, "dV"))]
    print("normwise errors dQ %.2e dK %.2e dV %.2e" % tuple(errs), flush=True)


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
        rq, rk, rv = oracle.backward(q[b:b + 1, hs], k[b:b + 1, g:g + 1], v[b:b + 1, g:g + 1], dO[b:b + 1, hs],
                                     w.W, w.C)
        assert_grad_parity(to64(dQ[b:b + 1, hs]), rq, f"dQ b{b} g{g}")
        assert_grad_parity(to64(dK[b:b + 1, g:g + 1]), rk, f"dK b{b} g{g}")
        assert_grad_parity(to64(dV[b:b + 1, g:g + 1]), rv, f"dV b{b} g{g}")
