"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests re-types the oracle's formula: each checks it against a
library routine it must reduce to, a closed form worked out for a structured
input, a hand-expanded fixture, or an invariant of softmax attention.  A
plausible slip in the oracle (window off by one, summary logit without ln C or
with log2, sum instead of mean for the summary key, missing 1/sqrt(d), the gap
tokens counted, a transposed head mapping) fails at least one of them.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def sdpa(q, k, v, mask=None, causal=False):
    """torch's scaled_dot_product_attention in fp64 on the CPU."""
    q, k, v = (torch.from_numpy(np.asarray(x, dtype=np.float64)) for x in (q, k, v))
    out = torch.nn.functional.scaled_dot_product_attention(
        q, k, v, attn_mask=None if mask is None else torch.from_numpy(mask), is_causal=causal)
    return out.numpy()


def expand_kv(k, G):
    return np.repeat(k, G, axis=1)


# ---------------------------------------------------------------------------
# Reductions to exact softmax attention (eq. softmax_attn, causal case)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("W", [1, 2, 5, 17])
def test_chunk_of_one_is_exact_causal_attention(W):
    # C = 1: every summary is the token itself (mean of one key, softmax over
    # one value, ln 1 = 0), so EVA is exact causal softmax attention.
    B, H, Hkv, L, d = 2, 4, 2, 37, 8
    q, k, v = rand((B, H, L, d), 1), rand((B, Hkv, L, d), 2), rand((B, Hkv, L, d), 3)
    o = oracle.prefill(q, k, v, W=W, C=1)
    ref = sdpa(q, expand_kv(k, H // Hkv), expand_kv(v, H // Hkv), causal=True)
    np.testing.assert_allclose(o, ref, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("C", [1, 3, 8, 64])
def test_window_covering_sequence_is_exact_causal_attention(C):
    B, H, Hkv, L, d = 1, 3, 1, 29, 16
    q, k, v = rand((B, H, L, d), 4), rand((B, Hkv, L, d), 5), rand((B, Hkv, L, d), 6)
    o = oracle.prefill(q, k, v, W=L, C=C)
    ref = sdpa(q, expand_kv(k, H), expand_kv(v, H), causal=True)
    np.testing.assert_allclose(o, ref, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("W", [1, 4, 9])
def test_no_complete_chunk_is_sliding_window_attention(W):
    # C > L: no summaries at all, only the W-token sliding window (self included).
    B, H, L, d = 1, 2, 23, 4
    q, k, v = rand((B, H, L, d), 7), rand((B, H, L, d), 8), rand((B, H, L, d), 9)
    o = oracle.prefill(q, k, v, W=W, C=L + 1)
    n = np.arange(L)[:, None]
    m = np.arange(L)[None, :]
    mask = (m <= n) & (m > n - W)
    ref = sdpa(q, k, v, mask=mask)
    np.testing.assert_allclose(o, ref, rtol=1e-11, atol=1e-12)


# ---------------------------------------------------------------------------
# Closed forms
# ---------------------------------------------------------------------------

def attended_token_sets(L, W, C):
    """For each row, (window positions, positions inside summarized chunks)."""
    out = []
    for n in range(L):
        start = n - W + 1
        win = list(range(max(0, start), n + 1))
        s = max(0, start) // C if start > 0 else 0
        summarized = list(range(0, s * C))
        out.append((win, summarized))
    return out


@pytest.mark.parametrize("L,W,C", [(40, 7, 4), (33, 5, 3), (64, 16, 8), (19, 1, 2)])
def test_equal_keys_gives_uniform_mean_over_attended_tokens(L, W, C):
    # All keys equal to u: each summary softmax is uniform so vhat is the chunk
    # mean; the summary key is u (mean, not sum), its logit is q.u/sqrt(d) + ln C,
    # exactly the window logit plus ln C.  Every attended token thus carries
    # the same weight: o_n is the plain mean of v over window + summarized chunks.
    d = 6
    u = rand((d,), 11)
    q = rand((1, 1, L, d), 12) * 2.0
    k = np.broadcast_to(u, (1, 1, L, d)).copy()
    v = rand((1, 1, L, d), 13)
    o = oracle.prefill(q, k, v, W=W, C=C)[0, 0]
    for n, (win, summ) in enumerate(attended_token_sets(L, W, C)):
        toks = win + summ
        np.testing.assert_allclose(o[n], v[0, 0, toks].mean(axis=0), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("L,W,C", [(50, 6, 5), (41, 10, 4)])
def test_zero_query_chunk_constant_values(L, W, C):
    # Q = 0, random K, V constant inside each chunk (value c_j for chunk j):
    # every window logit is 0, every summary logit is ln C, and vhat_j = c_j
    # whatever K is.  So o_n = (sum_window v + C * sum_{j<s(n)} c_j) / (w + C s).
    d = 3
    n_chunks = -(-L // C)
    cvals = rand((n_chunks, d), 21)
    v = np.repeat(cvals, C, axis=0)[:L][None, None]
    k = rand((1, 1, L, d), 22) * 3.0
    q = np.zeros((1, 1, L, d))
    o = oracle.prefill(q, k, v, W=W, C=C)[0, 0]
    for n, (win, summ) in enumerate(attended_token_sets(L, W, C)):
        s = len(summ) // C
        num = v[0, 0, win].sum(axis=0) + C * cvals[:s].sum(axis=0)
        np.testing.assert_allclose(o[n], num / (len(win) + C * s), rtol=1e-12, atol=1e-12)


def test_summary_with_one_spiked_key_closed_form():
    # Chunk of C = 4 keys in d = 4: k_0 = (a,0,0,0), others 0.  The mean key is
    # (a/4,0,0,0); scores are a^2/(4*sqrt(4)) = a^2/8 for j = 0 and 0 otherwise.
    a = 3.0
    C, d = 4, 4
    K = np.zeros((C, d))
    K[0, 0] = a
    V = rand((C, d), 31)
    Ks, Vs = oracle.summaries(K, V, C)
    np.testing.assert_allclose(Ks[0], [a / 4, 0, 0, 0], rtol=0, atol=0)
    w0 = math.exp(a * a / 8.0)
    expect = (w0 * V[0] + V[1] + V[2] + V[3]) / (w0 + 3.0)
    np.testing.assert_allclose(Vs[0], expect, rtol=1e-13)


def test_summary_two_level_keys_closed_form():
    # Chunk of C = 3 in d = 2 with keys (1,0), (1,0), (-1,2): mean (1/3, 2/3).
    # Scores /sqrt(2): (1/3)/sqrt2, (1/3)/sqrt2, (-1/3 + 4/3)/sqrt2 = 1/sqrt2.
    K = np.array([[1.0, 0.0], [1.0, 0.0], [-1.0, 2.0]])
    V = np.array([[1.0, 0.0], [0.0, 1.0], [2.0, 2.0]])
    Ks, Vs = oracle.summaries(K, V, 3)
    np.testing.assert_allclose(Ks[0], [1 / 3, 2 / 3], rtol=1e-15)
    e1 = math.exp((1 / 3) / math.sqrt(2))
    e3 = math.exp(1 / math.sqrt(2))
    expect = (e1 * V[0] + e1 * V[1] + e3 * V[2]) / (2 * e1 + e3)
    np.testing.assert_allclose(Vs[0], expect, rtol=1e-14)


def test_summaries_cover_complete_chunks_only():
    L, C, d = 23, 5, 3
    K, V = rand((L, d), 41), rand((L, d), 42)
    Ks, Vs = oracle.summaries(K, V, C)
    assert Ks.shape == (4, d)
    # Chunk 2 depends only on tokens 10..14.
    K2, V2 = K.copy(), V.copy()
    K2[:10] += 5.0
    K2[15:] -= 3.0
    V2[20:] = 0.0
    Ks2, Vs2 = oracle.summaries(K2, V2, C)
    np.testing.assert_array_equal(Ks[2], Ks2[2])
    np.testing.assert_array_equal(Vs[2], Vs2[2])


def test_summary_logit_offset_is_natural_log():
    # A single row attending one window token and one summarized chunk with
    # Q = 0: weights 1 (window) and C (summary, exp(ln C)).
    L, W, C, d = 5, 1, 4, 1
    v = np.array([[1.0], [1.0], [1.0], [1.0], [0.0]])[None, None]
    q = np.zeros((1, 1, L, d))
    k = np.zeros((1, 1, L, d))
    o = oracle.prefill(q, k, v, W=W, C=C)[0, 0]
    # Row 4: window {4} (v = 0) and chunk {0..3} (vhat = 1, weight 4).
    assert o[4, 0] == pytest.approx(4.0 / 5.0, rel=1e-15)


def test_hand_expanded_golden_cases():
    with open(os.path.join(GOLDEN, "zero_query_cases.json")) as f:
        cases = json.load(f)["cases"]
    for case in cases:
        L, W, C = case["L"], case["W"], case["C"]
        v = np.array(case["v"], dtype=np.float64).reshape(1, 1, L, 1)
        z = np.zeros_like(v)
        o = oracle.prefill(z, z, v, W=W, C=C)[0, 0, :, 0]
        expect = [float(Fraction(a, b)) for a, b in case["expected"]]
        np.testing.assert_allclose(o, expect, rtol=1e-14, err_msg=case["name"])


def test_visible_summary_count():
    # s(n) = floor(max(0, n-W+1)/C); spot values worked out by hand.
    assert oracle.visible_summaries(0, 4, 3) == 0
    assert oracle.visible_summaries(5, 4, 3) == 0
    assert oracle.visible_summaries(6, 4, 3) == 1
    assert oracle.visible_summaries(8, 4, 3) == 1
    assert oracle.visible_summaries(9, 4, 3) == 2
    # 8192-token context decoded at position 8192 with W = 512, C = 128:
    # the window is 7681..8192 and 60 chunks lie fully before it.
    assert oracle.visible_summaries(8192, 512, 128) == 60


# ---------------------------------------------------------------------------
# Invariants of softmax attention over an augmented key/value set
# ---------------------------------------------------------------------------

def _case(seed, L=45, d=8, H=2, Hkv=1):
    q = rand((1, H, L, d), seed)
    k = rand((1, Hkv, L, d), seed + 1)
    v = rand((1, Hkv, L, d), seed + 2)
    return q, k, v


def test_rows_are_convex_combinations_of_past_values():
    q, k, v = _case(51)
    W, C = 6, 4
    o = oracle.prefill(q, k, v, W=W, C=C)
    for h in range(2):
        for n in range(45):
            past = v[0, 0, : n + 1]
            assert np.all(o[0, h, n] <= past.max(axis=0) + 1e-12)
            assert np.all(o[0, h, n] >= past.min(axis=0) - 1e-12)


def test_constant_values_shift_and_linearity():
    q, k, v = _case(61)
    W, C = 5, 3
    o = oracle.prefill(q, k, v, W=W, C=C)
    const = np.broadcast_to(rand((8,), 64), v.shape).copy()
    np.testing.assert_allclose(oracle.prefill(q, k, const, W=W, C=C), np.broadcast_to(const, o.shape),
                               rtol=1e-12, atol=1e-12)
    shift = rand((8,), 65)
    np.testing.assert_allclose(oracle.prefill(q, k, v + shift, W=W, C=C), o + shift, rtol=1e-11, atol=1e-11)
    v2 = rand(v.shape, 66)
    np.testing.assert_allclose(oracle.prefill(q, k, 2.0 * v - 3.0 * v2, W=W, C=C),
                               2.0 * o - 3.0 * oracle.prefill(q, k, v2, W=W, C=C), rtol=1e-10, atol=1e-11)


def test_causality():
    q, k, v = _case(71)
    W, C = 7, 5
    o = oracle.prefill(q, k, v, W=W, C=C)
    cut = 20
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    q2[:, :, cut:] = rand(q2[:, :, cut:].shape, 72)
    k2[:, :, cut:] = rand(k2[:, :, cut:].shape, 73)
    v2[:, :, cut:] = rand(v2[:, :, cut:].shape, 74)
    o2 = oracle.prefill(q2, k2, v2, W=W, C=C)
    np.testing.assert_array_equal(o[:, :, :cut], o2[:, :, :cut])


def test_permutation_inside_summarized_chunk():
    q, k, v = _case(81, L=40)
    W, C = 6, 5
    o = oracle.prefill(q, k, v, W=W, C=C)
    perm = np.array([3, 0, 4, 1, 2]) + 5  # chunk 1 = tokens 5..9
    k2, v2 = k.copy(), v.copy()
    k2[:, :, 5:10] = k[:, :, perm]
    v2[:, :, 5:10] = v[:, :, perm]
    o2 = oracle.prefill(q, k2, v2, W=W, C=C)
    # rows whose window starts at or after token 10 see chunk 1 only as a summary
    rows = [n for n in range(40) if n - W + 1 >= 10]
    np.testing.assert_allclose(o2[:, :, rows], o[:, :, rows], rtol=1e-12, atol=1e-13)
    # a row whose window starts inside the permuted chunk sees a different
    # subset of its tokens (row 12: window 7..12, tokens 5 and 6 in no term)
    assert not np.allclose(o2[:, :, 12], o[:, :, 12])


def test_gqa_head_mapping_consecutive_heads_share_kv():
    # H = 4 query heads over 2 kv heads: heads 0,1 read kv head 0; 2,3 read 1.
    L, d, W, C = 21, 4, 4, 3
    q = rand((1, 4, L, d), 91)
    k = rand((1, 2, L, d), 92)
    v = rand((1, 2, L, d), 93)
    o = oracle.prefill(q, k, v, W=W, C=C)
    for h in range(4):
        g = h // 2
        oh = oracle.prefill(q[:, h:h + 1], k[:, g:g + 1], v[:, g:g + 1], W=W, C=C)
        np.testing.assert_array_equal(o[:, h], oh[:, 0])


def test_rows_entry_matches_whole_prefill():
    q, k, v = _case(101, L=50)
    W, C = 8, 4
    o = oracle.prefill(q, k, v, W=W, C=C)
    Ks, Vs = oracle.summaries(k[0, 0], v[0, 0], C)
    rows = np.array([0, 7, 8, 11, 12, 31, 49])
    got = oracle.attend_rows(q[0, 1, rows], rows, k[0, 0], v[0, 0], Ks, Vs, W, C)
    np.testing.assert_array_equal(got, o[0, 1, rows])


# ---------------------------------------------------------------------------
# Stochastic random-feature summaries (section "EVA Attention", single sample
# per chunk; xi from section "Random Feature Attention"; the clipped,
# downscaled proposal from the ablation "Impact of random feature sampling
# distribution")
# ---------------------------------------------------------------------------

def test_rf_summary_is_ratio_of_control_variate_sums():
    # The chunk value of eq. (eva) with S = 1: sum_m g_m / sum_m h_m, with g_m
    # and h_m carrying the importance weight N(w; 0, I) / (Z q(w)) and the
    # query feature xi(q_n, w).  Evaluated literally here for an arbitrary
    # query and weight: every query-dependent factor must cancel.
    C, d, lam = 6, 4, 0.1
    L = 3 * C
    k, v, eps = 0.5 * rand((L, d), 40), rand((L, d), 41), 2.0 * rand((L // C, d), 42)
    _, vs = oracle.summaries_rf(k, v, eps, C, lam)
    r4 = d ** 0.25
    xi = lambda x, w: math.exp(float(np.dot(w, x)) - 0.5 * float(np.dot(x, x)))
    q = rand(d, 43) / r4
    for c in range(L // C):
        xs = k[c * C:(c + 1) * C] / r4
        w = xs.mean(axis=0) + lam * np.clip(eps[c], -1.0, 1.0)
        weight = math.exp(-0.5 * float(np.dot(w, w))) / (2.0 * math.pi) ** (d / 2) / (3.7 * 0.21)
        g = sum(weight * xi(q, w) * xi(xs[j], w) * v[c * C + j] for j in range(C))
        h = sum(weight * xi(q, w) * xi(xs[j], w) for j in range(C))
        np.testing.assert_allclose(vs[c], g / h, rtol=1e-11, atol=1e-12)


def test_rf_summary_without_noise_and_equal_norms_is_deterministic_summary():
    # lambda = 0 and keys of one norm inside each chunk: the -|x|^2/2 term is
    # common to the chunk and cancels, leaving softmax(mean . k / sqrt(d)).
    C, d = 8, 16
    k = rand((4 * C, d), 44)
    k = 3.0 * k / np.linalg.norm(k, axis=1, keepdims=True)
    v = rand((4 * C, d), 45)
    ks, vs = oracle.summaries_rf(k, v, rand((4, d), 46), C, lam=0.0)
    ks0, vs0 = oracle.summaries(k, v, C)
    np.testing.assert_allclose(ks, ks0, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(vs, vs0, rtol=1e-11, atol=1e-12)


def test_rf_summary_norm_term_closed_form():
    # Two keys 0 and x: the sample (lambda = 0) is x/2 in scaled units, so
    # both log-weights are 0 (x/2 . x - |x|^2/2 = 0): the value is the plain
    # mean.  Without the norm term the second key would weigh exp(|x|^2/2)
    # times more.
    d = 4
    x = np.array([[0.0, 0.0, 0.0, 0.0], [1.5, -2.0, 0.5, 1.0]])
    v = rand((2, d), 47)
    _, vs = oracle.summaries_rf(x, v, np.zeros((1, d)), 2, lam=0.0)
    np.testing.assert_allclose(vs[0], v.mean(axis=0), rtol=1e-13, atol=1e-14)
    _, vs_det = oracle.summaries(x, v, 2)
    assert np.abs(vs_det[0] - v.mean(axis=0)).max() > 1e-3


def test_rf_summary_clips_noise_before_scaling():
    # omega = mean + lambda * clip(eps, -1, 1): noise beyond +-1 saturates,
    # and lambda multiplies the clipped value (halving in-range noise and
    # doubling lambda changes nothing).
    C, d = 5, 8
    k, v = rand((3 * C, d), 48), rand((3 * C, d), 49)
    e = rand((3, d), 50)
    big = np.sign(e) * 5.0
    unit = np.sign(e)
    np.testing.assert_allclose(oracle.summaries_rf(k, v, big, C, 0.3)[1], oracle.summaries_rf(k, v, unit, C, 0.3)[1],
                               rtol=1e-13, atol=1e-14)
    small = np.clip(e, -0.9, 0.9)
    np.testing.assert_allclose(oracle.summaries_rf(k, v, small / 2, C, 0.4)[1],
                               oracle.summaries_rf(k, v, small, C, 0.2)[1], rtol=1e-12, atol=1e-13)


def test_rf_summary_noise_direction():
    # A large lambda along +e0 favours the chunk key with the largest first
    # feature: the value tends to that key's value.
    d, C = 4, 4
    k = np.zeros((C, d))
    k[:, 0] = [-1.0, 0.0, 0.5, 2.0]
    v = np.eye(C, d)
    eps = np.zeros((1, d))
    eps[0, 0] = 3.0  # clipped to 1
    _, vs = oracle.summaries_rf(k, v, eps, C, lam=40.0)
    assert vs[0, 3] > 0.999
    eps[0, 0] = -3.0
    _, vs = oracle.summaries_rf(k, v, eps, C, lam=40.0)
    assert vs[0, 0] > 0.999


# ---------------------------------------------------------------------------
# Window variants (ablation "EVA Local Window Attention Variants"; the
# non-causal form of section "FlashEVA")
# ---------------------------------------------------------------------------

VARIANTS = (oracle.SLIDING, oracle.CHUNK_ALIGNED, oracle.BLOCKED, oracle.NONCAUSAL)


def test_sliding_variant_is_the_main_definition():
    B, H, Hkv, L, d, W, C = 1, 2, 1, 90, 8, 13, 5
    q, k, v = rand((B, H, L, d), 60), rand((B, Hkv, L, d), 61), rand((B, Hkv, L, d), 62)
    np.testing.assert_array_equal(oracle.prefill_variant(q, k, v, W, C, oracle.SLIDING), oracle.prefill(q, k, v, W, C))


@pytest.mark.parametrize("variant", [oracle.CHUNK_ALIGNED, oracle.BLOCKED])
@pytest.mark.parametrize("W,C", [(7, 1), (40, 3), (50, 50)])
def test_causal_variants_reduce_to_exact_attention(variant, W, C):
    # C = 1 (every summary is its token) or W >= L (no summaries): causal
    # softmax attention.
    B, H, Hkv, L, d = 1, 2, 2, 40, 8
    q, k, v = rand((B, H, L, d), 63), rand((B, Hkv, L, d), 64), rand((B, Hkv, L, d), 65)
    o = oracle.prefill_variant(q, k, v, W, C, variant)
    if C == 1 or W >= L:
        np.testing.assert_allclose(o, sdpa(q, k, v, causal=True), rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("W,C", [(7, 1), (40, 3), (41, 41)])
def test_noncausal_reduces_to_full_attention(W, C):
    B, H, Hkv, L, d = 1, 2, 2, 40, 8
    q, k, v = rand((B, H, L, d), 66), rand((B, Hkv, L, d), 67), rand((B, Hkv, L, d), 68)
    o = oracle.prefill_variant(q, k, v, W, C, oracle.NONCAUSAL)
    if C == 1 or W >= L:
        np.testing.assert_allclose(o, sdpa(q, k, v, causal=False), rtol=1e-11, atol=1e-12)


def equal_key_outputs(L, W, C, variant, seed):
    # all keys equal: every attended item has logit q.k/sqrt(d) (+ ln C for a
    # summary, whose value is its chunk's mean), so the output is the plain
    # mean over the attended tokens
    d = 4
    k = np.tile(rand((1, 1, 1, d), seed), (1, 1, L, 1))
    q = rand((1, 1, L, d), seed + 1)
    v = rand((1, 1, L, d), seed + 2)
    return oracle.prefill_variant(q, k, v, W, C, variant)[0, 0], v[0, 0]


@pytest.mark.parametrize("L,W,C", [(60, 10, 4), (33, 5, 7), (50, 1, 3)])
def test_chunk_aligned_has_no_gap(L, W, C):
    # window + summaries cover exactly tokens 0..n
    o, v = equal_key_outputs(L, W, C, oracle.CHUNK_ALIGNED, 69)
    for n in range(L):
        np.testing.assert_allclose(o[n], v[:n + 1].mean(axis=0), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("L,W,C", [(60, 12, 4), (61, 9, 3), (50, 10, 4)])
def test_blocked_window_token_sets(L, W, C):
    # row n: its block [floor(n/W) W, n] and the chunks ending at or before
    # the block start
    o, v = equal_key_outputs(L, W, C, oracle.BLOCKED, 70)
    for n in range(L):
        lo = (n // W) * W
        toks = list(range((lo // C) * C)) + list(range(lo, n + 1))
        np.testing.assert_allclose(o[n], v[toks].mean(axis=0), rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("L,W,C", [(60, 12, 4), (61, 9, 3), (50, 10, 4), (23, 30, 5)])
def test_noncausal_token_sets(L, W, C):
    # row n: its whole block and every complete chunk wholly outside it
    o, v = equal_key_outputs(L, W, C, oracle.NONCAUSAL, 71)
    for n in range(L):
        lo = (n // W) * W
        hi = min(L, lo + W) - 1
        toks = set(range(lo, hi + 1))
        for c in range(L // C):
            if (c + 1) * C <= lo or c * C > hi:
                toks.update(range(c * C, (c + 1) * C))
        np.testing.assert_allclose(o[n], v[sorted(toks)].mean(axis=0), rtol=1e-12, atol=1e-13)


def test_noncausal_rows_of_a_block_share_keys():
    # the attended set depends only on the block: equal queries inside a
    # block give equal outputs, and changing a token of another block that
    # lies in a summarized chunk changes them all alike
    L, W, C, d = 48, 12, 4, 8
    q, k, v = rand((1, 1, L, d), 72), rand((1, 1, L, d), 73), rand((1, 1, L, d), 74)
    q[0, 0, 12:24] = q[0, 0, 12]
    o = oracle.prefill_variant(q, k, v, W, C, oracle.NONCAUSAL)[0, 0]
    np.testing.assert_allclose(o[12:24], np.tile(o[12], (12, 1)), rtol=1e-13, atol=1e-14)


# ---------------------------------------------------------------------------
# Backward pass (the paper benchmarks forward + backward, section "FlashEVA
# Attention speedup"; training runs the kernels both ways)
# ---------------------------------------------------------------------------

def numeric_grad(f, x, h=1e-5):
    g = np.zeros_like(x)
    it = np.nditer(x, flags=["multi_index"])
    for _ in it:
        i = it.multi_index
        old = x[i]
        x[i] = old + h
        up = f()
        x[i] = old - h
        dn = f()
        x[i] = old
        g[i] = (up - dn) / (2 * h)
    return g


@pytest.mark.parametrize("L,W,C", [(11, 4, 2), (13, 3, 4), (9, 20, 3), (12, 1, 2)])
def test_backward_matches_finite_differences(L, W, C):
    # loss = sum(O * R) for a fixed R: dO = R; every gradient of Q, K, V
    # (through window, summary keys/values and the summaries' own K, V
    # dependence) against central differences of the forward
    B, H, Hkv, d = 1, 2, 1, 3
    q, k, v = rand((B, H, L, d), 80), rand((B, Hkv, L, d), 81), rand((B, Hkv, L, d), 82)
    R = rand((B, H, L, d), 83)
    loss = lambda: float((oracle.prefill(q, k, v, W, C) * R).sum())
    dq, dk, dv = oracle.backward(q, k, v, R, W, C)
    for x, g in ((q, dq), (k, dk), (v, dv)):
        np.testing.assert_allclose(g, numeric_grad(loss, x), rtol=1e-6, atol=1e-8)


def test_backward_chunk_of_one_is_exact_attention_autograd():
    # C = 1: the forward is exact causal attention, so its gradients are the
    # library's (torch autograd through scaled_dot_product_attention, fp64)
    B, H, Hkv, L, d, W = 1, 4, 2, 24, 8, 5
    q, k, v = rand((B, H, L, d), 84), rand((B, Hkv, L, d), 85), rand((B, Hkv, L, d), 86)
    R = rand((B, H, L, d), 87)
    tq, tk, tv = (torch.from_numpy(x.copy()).requires_grad_() for x in (q, k, v))
    o = torch.nn.functional.scaled_dot_product_attention(tq, tk.repeat_interleave(H // Hkv, 1),
                                                         tv.repeat_interleave(H // Hkv, 1), is_causal=True)
    (o * torch.from_numpy(R)).sum().backward()
    dq, dk, dv = oracle.backward(q, k, v, R, W, 1)
    np.testing.assert_allclose(dq, tq.grad.numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dk, tk.grad.numpy(), rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(dv, tv.grad.numpy(), rtol=1e-10, atol=1e-11)


# Term magnitudes of the backward (oracle.backward_terms): the scale of the
# GPU gradients' rounding-error bound.  Not part of the method; pinned by
# the properties such a magnitude must have.
@pytest.mark.parametrize("L,W,C", [(40, 6, 4), (33, 50, 5), (30, 1, 3), (41, 8, 1)])
def test_backward_terms_bound_the_gradients(L, W, C):
    # a sum's absolute value never exceeds the sum of its terms' absolute values
    B, H, Hkv, d = 1, 4, 2, 6
    q, k, v = rand((B, H, L, d), 90), rand((B, Hkv, L, d), 91), rand((B, Hkv, L, d), 92)
    R = rand((B, H, L, d), 93)
    for g, t in zip(oracle.backward(q, k, v, R, W, C), oracle.backward_terms(q, k, v, R, W, C)):
        assert np.all(t >= np.abs(g) * (1 - 1e-12))
        assert t.max() > 0


def test_backward_terms_exact_without_cancellation():
    # dV: with an all-positive output gradient every term of every dV entry
    # (p dO, and b_j dvhat through the summaries) is non-negative, so the
    # magnitude is the gradient itself
    B, H, Hkv, L, d, W, C = 1, 2, 1, 30, 5, 6, 4
    q, k, v = rand((B, H, L, d), 94), rand((B, Hkv, L, d), 95), rand((B, Hkv, L, d), 96)
    R = np.abs(rand((B, H, L, d), 97)) + 0.1
    np.testing.assert_allclose(oracle.backward_terms(q, k, v, R, W, C)[2], oracle.backward(q, k, v, R, W, C)[2],
                               rtol=1e-12, atol=0)
    # dQ: with a two-token window, no chunk, zero queries (both weights 1/2)
    # and values +-a of alternating sign, every row n >= 1 has output 0, so
    # D = 0 and its gradient is (dO.v_n / 2) (k_n - k_{n-1}) / sqrt(d); a
    # positive dO makes |dO.v_n| = sum_e |dO_e v_e| and keys of alternating
    # sign make |k_n - k_{n-1}| = |k_n| + |k_{n-1}| entry by entry, so no term
    # cancels
    L = 12
    q = np.zeros((B, H, L, d))
    v = np.abs(rand((B, Hkv, L, d), 99)[:, :, :1]) + 0.1 + np.zeros((B, Hkv, L, d))
    v[:, :, 1::2] *= -1
    k = np.abs(rand((B, Hkv, L, d), 100)) + 0.1
    k[:, :, 1::2] *= -1
    R = np.abs(rand((B, H, L, d), 101)) + 0.1
    tq = oracle.backward_terms(q, k, v, R, 2, L + 1)[0]
    dq = oracle.backward(q, k, v, R, 2, L + 1)[0]
    np.testing.assert_allclose(tq[:, :, 1:], np.abs(dq[:, :, 1:]), rtol=1e-12, atol=1e-15)


def test_backward_terms_single_token_window():
    # W = 1 and no chunk: every row attends only itself (weight 1), so
    # D = dO.v_n, the logit gradient dO.v_n - D is exactly 0 and so are dQ and
    # dK, while each of its two dot products has term magnitude
    # m = sum_e |dO_e v_e|: T_q = 2 m |k_n| / sqrt(d), T_k = 2 m |q_n| / sqrt(d)
    # (one query head per key here), and T_v = |dO_n| = dV
    B, H, Hkv, L, d = 1, 1, 1, 9, 5
    q, k, v = rand((B, H, L, d), 130), rand((B, Hkv, L, d), 131), rand((B, Hkv, L, d), 132)
    R = rand((B, H, L, d), 133)
    dq, dk, dv = oracle.backward(q, k, v, R, 1, L + 1)
    tq, tk, tv = oracle.backward_terms(q, k, v, R, 1, L + 1)
    gv = np.abs(R * v).sum(-1, keepdims=True)
    np.testing.assert_allclose(dq, 0.0, atol=1e-14)
    np.testing.assert_allclose(dk, 0.0, atol=1e-14)
    np.testing.assert_allclose(tq, 2 * gv * np.abs(k) / np.sqrt(d), rtol=1e-12, atol=0)
    np.testing.assert_allclose(tk, 2 * gv * np.abs(q) / np.sqrt(d), rtol=1e-12, atol=0)
    np.testing.assert_allclose(tv, np.abs(R), rtol=1e-12, atol=0)
    np.testing.assert_allclose(dv, R, rtol=1e-12, atol=1e-15)


def test_backward_terms_scale_with_the_output_gradient():
    B, H, Hkv, L, d, W, C = 1, 2, 2, 25, 4, 5, 3
    q, k, v = rand((B, H, L, d), 102), rand((B, Hkv, L, d), 103), rand((B, Hkv, L, d), 104)
    R = rand((B, H, L, d), 105)
    for t1, t2 in zip(oracle.backward_terms(q, k, v, R, W, C), oracle.backward_terms(q, k, v, -2.5 * R, W, C)):
        np.testing.assert_allclose(t2, 2.5 * t1, rtol=1e-12, atol=0)


# ---------------------------------------------------------------------------
# Counter-based noise for the stochastic summaries (so that a chunk's draw
# is the same whether its summary is built at prefill or during decode)
# ---------------------------------------------------------------------------

def test_philox_known_answers():
    # Philox4x32-10 known-answer vectors of its authors' reference suite
    # (Salmon et al., SC 2011): counter, key -> output
    cases = [
        ([0, 0, 0, 0], [0, 0], [0x6627e8d5, 0xe169c58d, 0xbc57ac4c, 0x9b00dbd8]),
        ([0xffffffff] * 4, [0xffffffff] * 2, [0x408f276d, 0x41c83b0e, 0xa20bc7c6, 0x6d5451fd]),
        ([0x243f6a88, 0x85a308d3, 0x13198a2e, 0x03707344], [0xa4093822, 0x299f31d0],
         [0xd16cfe09, 0x94fdcceb, 0x5001e420, 0x24126ea1]),
    ]
    for ctr, key, want in cases:
        assert oracle.philox4x32_10(ctr, key) == want


def test_rf_noise_is_standard_normal():
    from scipy import stats
    eps = oracle.rf_noise(64, 64, 128, seed=12345).ravel()
    assert abs(eps.mean()) < 5e-3 and abs(eps.var() - 1.0) < 1e-2
    assert stats.kstest(eps, "norm").pvalue > 1e-3
    # pairs from one Box-Muller draw, and neighbouring blocks, are uncorrelated
    e = eps.reshape(-1, 4)
    for i, j in ((0, 1), (2, 3), (1, 2)):
        assert abs(np.corrcoef(e[:, i], e[:, j])[0, 1]) < 1e-2


def test_rf_noise_depends_on_counter_and_seed_only():
    big = oracle.rf_noise(5, 7, 64, seed=99)
    small = oracle.rf_noise(2, 3, 64, seed=99)
    np.testing.assert_array_equal(small, big[:2, :3])
    other = oracle.rf_noise(2, 3, 64, seed=100)
    assert np.abs(other - small).max() > 0.5
    # seed words go to the key: the high word matters too
    assert np.abs(oracle.rf_noise(1, 1, 64, seed=99 + (1 << 32)) - small[:1, :1]).max() > 0.5


# Backward under the window variants: the same chain rule over each row's
# variant item set
@pytest.mark.parametrize("variant", [oracle.CHUNK_ALIGNED, oracle.BLOCKED, oracle.NONCAUSAL])
@pytest.mark.parametrize("L,W,C", [(13, 4, 2), (14, 5, 3), (12, 20, 3)])
def test_backward_variant_matches_finite_differences(variant, L, W, C):
    B, H, Hkv, d = 1, 2, 1, 3
    q, k, v = rand((B, H, L, d), 110), rand((B, Hkv, L, d), 111), rand((B, Hkv, L, d), 112)
    R = rand((B, H, L, d), 113)
    loss = lambda: float((oracle.prefill_variant(q, k, v, W, C, variant) * R).sum())
    dq, dk, dv = oracle.backward(q, k, v, R, W, C, variant)
    for x, g in ((q, dq), (k, dk), (v, dv)):
        np.testing.assert_allclose(g, numeric_grad(loss, x), rtol=1e-6, atol=1e-8)
    for g, t in zip((dq, dk, dv), oracle.backward_terms(q, k, v, R, W, C, variant)):
        assert np.all(t >= np.abs(g) * (1 - 1e-12))


def test_backward_variants_reduce_to_exact_attention():
    # C = 1 with a window covering the sequence: every causal variant is exact
    # causal attention and the non-causal one full attention, so the
    # gradients are the library's (torch autograd through SDPA, fp64)
    B, H, Hkv, L, d = 1, 2, 1, 16, 4
    q, k, v = rand((B, H, L, d), 114), rand((B, Hkv, L, d), 115), rand((B, Hkv, L, d), 116)
    R = rand((B, H, L, d), 117)
    for variant, causal in ((oracle.CHUNK_ALIGNED, True), (oracle.BLOCKED, True), (oracle.NONCAUSAL, False)):
        tq, tk, tv = (torch.from_numpy(x.copy()).requires_grad_() for x in (q, k, v))
        o = torch.nn.functional.scaled_dot_product_attention(tq, tk.repeat_interleave(H // Hkv, 1),
                                                             tv.repeat_interleave(H // Hkv, 1), is_causal=causal)
        (o * torch.from_numpy(R)).sum().backward()
        dq, dk, dv = oracle.backward(q, k, v, R, L, 1, variant)
        np.testing.assert_allclose(dq, tq.grad.numpy(), rtol=1e-10, atol=1e-11)
        np.testing.assert_allclose(dk, tk.grad.numpy(), rtol=1e-10, atol=1e-11)
        np.testing.assert_allclose(dv, tv.grad.numpy(), rtol=1e-10, atol=1e-11)
