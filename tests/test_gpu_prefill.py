"""GPU parity of eva_build_summaries and eva_prefill against the fp64 oracle.

Small shapes are compared element by element over every row (several query
tiles, ragged tails, GQA packings, degenerate windows and chunks).  The
LLM-shaped workloads are run at full size in the launch configuration the
benchmark times and compared on sampled rows around every boundary.  Mask
probes (zero Q/K with one-hot values, and dominant spiked keys) make a token
wrongly included or excluded cost far more than the bf16 tolerance.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2511_00576_amd import eva, inputs
from parity import assert_parity, edge_rows, oracle_sampled, to64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    eva._lib.load()


def cuda(*ts):
    return [t.cuda() for t in ts]


def check_prefill(B, H, Hkv, L, d, W, C, dtype, seed, maker=inputs.qkv):
    print(f"prefill B{B} H{H}/{Hkv} L{L} d{d} W{W} C{C} {dtype} seed{seed} {maker.__name__}", flush=True)
    q, k, v = maker(B, H, Hkv, L, d, dtype=dtype, seed=seed)
    O, Ks, Vs = eva.prefill(*cuda(q, k, v), W, C, return_summaries=True)
    torch.cuda.synchronize()
    ref, rKs, rVs = oracle.prefill(q, k, v, W, C, return_summaries=True)
    err = assert_parity(to64(O), ref, dtype, "O")
    assert_parity(to64(Ks), rKs, dtype, "Ksum")
    assert_parity(to64(Vs), rVs, dtype, "Vsum")
    return err


SMALL = [
    # B, H, Hkv, L, d, W, C
    (1, 2, 2, 256, 64, 32, 16),     # the tiny fp32 workload
    (2, 4, 2, 300, 128, 50, 7),     # ragged tail, odd chunk, G = 2
    (1, 8, 2, 517, 64, 64, 32),     # G = 4, ragged
    (1, 16, 2, 400, 128, 96, 16),   # G = 8: two head groups per kv head
    (1, 3, 1, 333, 64, 40, 8),      # G = 3: one head per workgroup
    (1, 2, 1, 200, 128, 1, 3),      # W = 1: self plus summaries only
    (1, 2, 2, 150, 64, 200, 16),    # W >= L: exact causal attention
    (1, 2, 2, 130, 64, 20, 1),      # C = 1: exact causal attention
    (1, 2, 2, 100, 128, 10, 128),   # C > L: no summaries, sliding window
    (1, 2, 2, 1, 64, 4, 4),         # one token
    (2, 2, 1, 17, 128, 5, 3),       # shorter than one query tile
    (1, 4, 4, 1030, 128, 256, 64),  # many summary blocks + window blocks
]


@pytest.mark.parametrize("shape", SMALL)
def test_prefill_f32(shape):
    check_prefill(*shape, torch.float32, seed=11)


@pytest.mark.parametrize("shape", SMALL)
def test_prefill_bf16(shape):
    check_prefill(*shape, torch.bfloat16, seed=12)


def test_tiny_f32_workload():
    w = inputs.TINY_F32
    check_prefill(w.B, w.H, w.Hkv, w.L, w.d, w.W, w.C, w.dtype, seed=w.seed)


@pytest.mark.parametrize("W,C", [(256, 64), (512, 128), (200, 48)])
def test_prefill_f32_llm_head_shape(W, C):
    # fp32 instantiation of the same tiling at LLM head shapes: pins every
    # mask boundary to 1e-5 (bf16 tolerance is too loose for a one-token slip).
    check_prefill(1, 4, 1, 4096, 128, W, C, torch.float32, seed=13)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
@pytest.mark.parametrize("W,C", [(256, 64), (77, 13), (512, 128)])
def test_mask_probe_one_hot_values(dtype, W, C):
    check_prefill(1, 4, 2, 2048, 128, W, C, dtype, seed=14, maker=inputs.needle_qkv)


@pytest.mark.parametrize("W,C", [(256, 64), (100, 20)])
def test_mask_probe_spiked_keys(W, C):
    check_prefill(2, 4, 2, 1500, 128, W, C, torch.bfloat16, seed=15, maker=inputs.spike_qkv)


def test_prefill_deterministic():
    q, k, v = cuda(*inputs.qkv(2, 8, 2, 777, 128, torch.bfloat16, seed=16))
    a = eva.prefill(q, k, v, 100, 16)
    b = eva.prefill(q, k, v, 100, 16)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# chunk sizes that take the register-resident kernel (C = 256/(d/8) rows per
# step times 1, 2, 4, 8, and 16 for bf16: C 256 at d 128) and ones that take
# the three-pass kernel
@pytest.mark.parametrize("L,C", [(1000, 7), (64, 64), (63, 64), (4096, 256), (300, 16), (300, 32),
                                 (600, 128), (1100, 512), (640, 160)])
@pytest.mark.parametrize("d", [64, 128])
def test_summaries(L, C, d):
    for dtype in (torch.float32, torch.bfloat16):
        _, k, v = inputs.qkv(2, 1, 3, L, d, dtype, seed=17)
        Ks, Vs = eva.build_summaries(*cuda(k, v), C)
        torch.cuda.synchronize()
        assert Ks.shape == (2, 3, L // C, d)
        for b in range(2):
            for g in range(3):
                rK, rV = oracle.summaries(k[b, g], v[b, g], C)
                assert_parity(to64(Ks[b, g]), rK, dtype, "Ksum")
                assert_parity(to64(Vs[b, g]), rV, dtype, "Vsum")


@pytest.mark.parametrize("L,C", [(1000, 7), (64, 64), (4096, 256), (300, 32), (600, 128), (640, 160)])
@pytest.mark.parametrize("d", [64, 128])
def test_summaries_rf(L, C, d):
    # both summary kernels (register-resident and three-pass), both dtypes;
    # lambda large enough that the noise term matters, noise beyond +-1
    for dtype in (torch.float32, torch.bfloat16):
        _, k, v = inputs.qkv(2, 1, 3, L, d, dtype, seed=18)
        eps = inputs.normal((2, 3, L // C, d), 19) * 1.5
        Ks, Vs = eva.build_summaries_rf(*cuda(k, v), eps.cuda(), C, lam=0.3)
        torch.cuda.synchronize()
        for b in range(2):
            for g in range(3):
                rK, rV = oracle.summaries_rf(k[b, g], v[b, g], eps[b, g], C, lam=0.3)
                assert_parity(to64(Ks[b, g]), rK, dtype, "Ksum")
                assert_parity(to64(Vs[b, g]), rV, dtype, "Vsum")


def test_prefill_with_rf_summaries():
    # the fused prefill with stochastic summaries against oracle rows over the
    # oracle's stochastic summaries
    B, H, Hkv, L, d, W, C = 2, 8, 2, 700, 128, 64, 32
    for dtype in (torch.float32, torch.bfloat16):
        q, k, v = inputs.qkv(B, H, Hkv, L, d, dtype, seed=20)
        eps = inputs.normal((B, Hkv, L // C, d), 21)
        qc, kc, vc = cuda(q, k, v)
        Ks, Vs = eva.build_summaries_rf(kc, vc, eps.cuda(), C, lam=0.1)
        O = eva.prefill_attention(qc, kc, vc, Ks, Vs, W, C)
        torch.cuda.synchronize()
        rows = edge_rows(L, W, C, extra=16, seed=3)
        for b, h in ((0, 0), (1, 5)):
            g = h // (H // Hkv)
            rK, rV = oracle.summaries_rf(k[b, g], v[b, g], eps[b, g], C, lam=0.1)
            ref = oracle.attend_rows(to64(q[b, h, torch.from_numpy(rows)]), rows, k[b, g], v[b, g], rK, rV, W, C)
            assert_parity(to64(O[b, h, torch.from_numpy(rows)]), ref, dtype, f"rf prefill b{b} h{h}")


# ---- window variants ----
VARIANTS = [oracle.CHUNK_ALIGNED, oracle.BLOCKED, oracle.NONCAUSAL]
VARIANT_SHAPES = [
    # B, H, Hkv, L, d, W, C
    (1, 2, 2, 300, 64, 40, 16),     # G = 1: one head per workgroup tile
    (2, 8, 2, 517, 128, 64, 24),    # G = 4: four heads per tile, ragged tail
    (1, 4, 4, 700, 128, 100, 7),    # odd chunk, window not a multiple of 16
    (1, 2, 1, 250, 128, 1, 5),      # W = 1
    (1, 2, 2, 120, 64, 200, 16),    # W >= L
    (1, 16, 2, 400, 128, 96, 32),   # G = 8: two head groups per kv head
]


def check_variant(B, H, Hkv, L, d, W, C, dtype, variant, seed, maker=inputs.qkv):
    print(f"variant {variant} B{B} H{H}/{Hkv} L{L} d{d} W{W} C{C} {dtype} {maker.__name__}", flush=True)
    q, k, v = maker(B, H, Hkv, L, d, dtype=dtype, seed=seed)
    O = eva.prefill(*cuda(q, k, v), W, C, window=variant)
    torch.cuda.synchronize()
    ref = oracle.prefill_variant(q, k, v, W, C, variant)
    assert_parity(to64(O), ref, dtype, f"variant {variant}")


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", VARIANT_SHAPES)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_prefill_variants(variant, shape, dtype):
    check_variant(*shape, dtype, variant, seed=30)


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_prefill_variant_mask_probe(variant, dtype):
    # one-hot values make a token wrongly in or out cost far more than the
    # bf16 tolerance
    check_variant(1, 4, 2, 1500, 128, 96, 16, dtype, variant, seed=31, maker=inputs.needle_qkv)


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("w", [inputs.LLM_BF16, inputs.GQA_BF16], ids=lambda w: w.name.split()[0])
def test_prefill_variant_full_size_sampled(variant, w):
    print(f"full-size {w.name} variant {variant}", flush=True)
    q, k, v = inputs.workload_qkv(w)
    O = eva.prefill(*cuda(q, k, v), w.W, w.C, window=variant)
    torch.cuda.synchronize()
    rows = edge_rows(w.L, w.W, w.C, extra=24, seed=variant)
    rows = np.unique(np.concatenate([rows, np.arange(0, w.L, w.W), np.arange(w.W - 1, w.L, w.W)]))
    for b, h in ((0, 0), (w.B - 1, w.H - 1)):
        g = h // (w.H // w.Hkv)
        Ks, Vs = oracle.summaries(k[b, g], v[b, g], w.C)
        ref = oracle.attend_rows_variant(to64(q[b, h, torch.from_numpy(rows)]), rows, k[b, g], v[b, g], Ks, Vs,
                                         w.W, w.C, variant)
        assert_parity(to64(O[b, h, torch.from_numpy(rows)]), ref, w.dtype, f"{w.name} variant {variant} b{b} h{h}")


FULL = [inputs.LLM_BF16, inputs.GQA_BF16, inputs.LONG_BF16, inputs.KBENCH_BF16]


@pytest.mark.parametrize("w", FULL, ids=lambda w: w.name.split()[0])
def test_full_size_sampled(w):
    print(f"full-size {w.name}", flush=True)
    q, k, v = inputs.workload_qkv(w)
    O = eva.prefill(*cuda(q, k, v), w.W, w.C)
    torch.cuda.synchronize()
    rows = edge_rows(w.L, w.W, w.C, extra=48, seed=w.seed)
    heads = [(0, 0), (w.B - 1, w.H - 1), (w.B // 2, w.H // 3)]
    ref = oracle_sampled(q, k, v, w.W, w.C, heads, rows)
    for (b, h), r in ref.items():
        got = to64(O[b, h, torch.from_numpy(rows)])
        assert_parity(got, r, w.dtype, f"{w.name} b{b} h{h}")


@pytest.mark.parametrize("C", [64, 128])
def test_long_context_chunk_sweep_sampled(C):
    w = inputs.LONG_BF16
    print(f"long-context sweep C={C}", flush=True)
    q, k, v = inputs.workload_qkv(w)
    O = eva.prefill(*cuda(q, k, v), w.W, C)
    torch.cuda.synchronize()
    rows = edge_rows(w.L, w.W, C, extra=32, seed=C)
    ref = oracle_sampled(q, k, v, w.W, C, [(0, 5), (0, 30)], rows)
    for (b, h), r in ref.items():
        assert_parity(to64(O[b, h, torch.from_numpy(rows)]), r, w.dtype, f"C={C} h{h}")


def test_full_size_mask_probe():
    # dominant spiked keys at the LLM workload's window/chunk geometry: a spike
    # entering or leaving a window moves that row by O(1)
    w = inputs.LLM_BF16
    q, k, v = inputs.spike_qkv(1, 2, 2, w.L, w.d, w.dtype, seed=18)
    O = eva.prefill(*cuda(q, k, v), w.W, w.C)
    torch.cuda.synchronize()
    ref = oracle.prefill(q, k, v, w.W, w.C)
    assert_parity(to64(O), ref, w.dtype, "needles")


# ---- the 8-wave, 64-key-block configuration of the bf16 kernel ----
# The kernel takes it when a kv head serves several query heads (G > 1) and
# the window exceeds 512 keys (the long-context workload's case); every shape
# here does.  Compared element by element over every row.
WIDE = [
    # B, H, Hkv, L, d, W, C
    (1, 8, 2, 1500, 128, 600, 32),
    (1, 16, 4, 2100, 64, 777, 48),    # d = 64, ragged tail, W mod 16 = 9
    (1, 8, 2, 800, 128, 799, 16),     # W = L - 1: only the last row drops token 0 (a gap token)
    (2, 4, 2, 1100, 128, 1024, 64),   # W mod 16 = 0, G = 2
    (1, 24, 8, 1400, 128, 520, 24),   # G = 3: one head per workgroup, 256 positions
    (1, 8, 2, 1300, 128, 513, 1),     # C = 1: exact causal attention
]


@pytest.mark.parametrize("shape", WIDE)
def test_prefill_bf16_wide_config(shape):
    check_prefill(*shape, torch.bfloat16, seed=40)


def _spike_check(B, H, Hkv, L, d, W, C, positions, chunks, seed, variant=oracle.SLIDING):
    print(f"spikes B{B} H{H}/{Hkv} L{L} d{d} W{W} C{C} variant {variant} positions {len(positions)} "
          f"chunks {list(chunks)}", flush=True)
    q, k, v = inputs.spike_at_qkv(B, H, Hkv, L, d, positions, chunks, C, torch.bfloat16, seed)
    O = eva.prefill(*cuda(q, k, v), W, C, window=variant)
    torch.cuda.synchronize()
    ref = oracle.prefill_variant(q, k, v, W, C, variant)
    assert_parity(to64(O), ref, torch.bfloat16, f"spikes variant {variant}")


def _anchor_rows(L, W, C):
    # rows whose window edges are probed: the first rows with a summary, rows
    # at every 16-row offset class of a tile, and the last rows
    rows = [W - 1, W, W + C - 1, W + C, 2 * C + W - 1, L - 1, L - 2]
    rows += [W + 64 * t + off for t, off in ((1, 0), (2, 1), (3, 15), (4, 16), (5, 31), (6, 47), (7, 63))]
    return [r for r in rows if W <= r < L]


@pytest.mark.parametrize("shape", [WIDE[0], WIDE[1], WIDE[3], (1, 4, 4, 1500, 128, 300, 32)])
def test_spiked_window_edges(shape):
    # dominant keys on the first and last window positions, the token before
    # the window (a gap token or a chunk's last token) and chunk last tokens:
    # a one-token slip of the window's lower edge, the diagonal or s(n) moves
    # a row by O(1) at any window length
    B, H, Hkv, L, d, W, C = shape
    pos = inputs.window_edge_positions(L, W, C, _anchor_rows(L, W, C))
    _spike_check(B, H, Hkv, L, d, W, C, pos, (), seed=41)


@pytest.mark.parametrize("shape", [WIDE[0], WIDE[1], WIDE[3], (1, 4, 4, 1500, 128, 300, 32)])
def test_spiked_whole_chunk(shape):
    # every key of a chunk spiked: its summary key dominates exactly the rows
    # with s(n) > c, and the chunk's own keys the rows whose window holds them
    B, H, Hkv, L, d, W, C = shape
    n_chunks = L // C
    chunks = sorted({1, n_chunks // 3}) if n_chunks > 1 else []
    _spike_check(B, H, Hkv, L, d, W, C, (), chunks, seed=42)


VARIANT_WIDE = [WIDE[0], WIDE[1]]


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", VARIANT_WIDE)
def test_prefill_variants_wide_config(variant, shape):
    check_variant(*shape, torch.bfloat16, variant, seed=43)


@pytest.mark.parametrize("variant", VARIANTS)
@pytest.mark.parametrize("shape", VARIANT_WIDE)
def test_spiked_variants_wide_config(variant, shape):
    # spikes on the variants' own edges (block starts kW, chunk starts kC and
    # the tokens beside them) plus a regular comb, and one wholly spiked chunk
    B, H, Hkv, L, d, W, C = shape
    pos = set(range(7, L, 53))
    for kk in range(1, L // W + 1):
        pos.update((kk * W - 1, kk * W, kk * W + 1))
    for kk in range(1, L // C + 1, 5):
        pos.update((kk * C - 1, kk * C))
    _spike_check(B, H, Hkv, L, d, W, C, sorted(pos), (), seed=44, variant=variant)
    _spike_check(B, H, Hkv, L, d, W, C, (), (L // C // 2,), seed=45, variant=variant)


# ---- 4-wave configuration without any summary block: waves whose first two
# blocks are both outside their window start from untouched score registers
@pytest.mark.parametrize("W,C", [(64, 2048), (33, 4096)])
def test_prefill_bf16_no_summary_blocks(W, C):
    check_prefill(1, 2, 2, 1024, 128, W, C, torch.bfloat16, seed=46)
    check_prefill(1, 2, 2, 1024, 128, W, C, torch.bfloat16, seed=47, maker=inputs.needle_qkv)
