"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module draws random numbers and names workload shapes; it holds none of
the attention arithmetic.  Every draw uses a torch CPU generator seeded by the
caller: Q first, then K, then V, as float32 N(0, 1), then cast to the requested
dtype with round-to-nearest-even (torch's cast).  Both the HIP path and the
oracle read the same rounded host tensors.
"""
from dataclasses import dataclass

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    Hkv: int
    L: int
    d: int
    W: int
    C: int
    dtype: torch.dtype
    seed: int


# Workloads shaped like the LLM attention layers the method targets (head dim
# 128, 32 query heads, grouped-query attention, contexts of 4k to 32k tokens).
TINY_F32 = Workload("tiny-f32 B1 H2 L256 d64 W32 C16", 1, 2, 2, 256, 64, 32, 16, torch.float32, 1)
LLM_BF16 = Workload("llm-bf16 B8 H32 L4096 d128 W256 C64", 8, 32, 32, 4096, 128, 256, 64, torch.bfloat16, 2)
GQA_BF16 = Workload("gqa-bf16 B4 H32/8 L8192 d128 W512 C128", 4, 32, 8, 8192, 128, 512, 128, torch.bfloat16, 3)
LONG_BF16 = Workload("long-bf16 B1 H32/8 L32768 d128 W1024 C256", 1, 32, 8, 32768, 128, 1024, 256,
                     torch.bfloat16, 5)
# shaped like the paper's kernel benchmark (section "FlashEVA Attention
# speedup": window 256, 128-token chunks, 16k tokens at batch 8)
KBENCH_BF16 = Workload("kbench-bf16 B8 H32 L16384 d128 W256 C128", 8, 32, 32, 16384, 128, 256, 128,
                       torch.bfloat16, 7)


@dataclass(frozen=True)
class DecodeWorkload:
    name: str
    B: int
    H: int
    Hkv: int
    d: int
    W: int
    C: int
    context: int  # tokens already held by the cache before the decoded token
    dtype: torch.dtype
    seed: int


# 64 sequences, 8192 tokens of context held as a 512-token exact window plus
# 60 chunk summaries of 128 tokens each.
DECODE_BF16 = DecodeWorkload("decode-bf16 B64 H32/8 d128 ctx8192 W512 C128", 64, 32, 8, 128, 512, 128, 8192,
                             torch.bfloat16, 4)


@dataclass(frozen=True)
class GenerateWorkload:
    name: str
    B: int
    H: int
    Hkv: int
    d: int
    W: int
    C: int
    prompt_min: int  # prompt lengths are uniform in [prompt_min, prompt_max]
    prompt_max: int
    steps: int       # tokens generated per sequence
    dtype: torch.dtype
    seed: int


# Batched generation after a prompt: 32 sequences with prompts of 1024 to
# 3072 tokens (mean 2048), 1024 tokens generated each, the method's main
# window / chunk setting (W = 256, C = 16).
GENERATE_BF16 = GenerateWorkload("generate-bf16 B32 H32/8 d128 W256 C16 prompt1024-3072 gen1024", 32, 32, 8, 128,
                                 256, 16, 1024, 3072, 1024, torch.bfloat16, 6)


def prompt_lengths(w: GenerateWorkload) -> list:
    """Seeded ragged prompt lengths of a generation workload."""
    g = torch.Generator().manual_seed(w.seed + 500)
    return torch.randint(w.prompt_min, w.prompt_max + 1, (w.B,), generator=g).tolist()


def normal(shape, seed: int, dtype=torch.float32, generator=None) -> torch.Tensor:
    g = generator if generator is not None else torch.Generator().manual_seed(seed)
    return torch.randn(*shape, generator=g, dtype=torch.float32).to(dtype)


def qkv(B, H, Hkv, L, d, dtype=torch.bfloat16, seed=0):
    """Q [B,H,L,d], K, V [B,Hkv,L,d], i.i.d. N(0,1), drawn in that order."""
    g = torch.Generator().manual_seed(seed)
    q = normal((B, H, L, d), seed, dtype, g)
    k = normal((B, Hkv, L, d), seed, dtype, g)
    v = normal((B, Hkv, L, d), seed, dtype, g)
    return q, k, v


def workload_qkv(w: Workload):
    return qkv(w.B, w.H, w.Hkv, w.L, w.d, w.dtype, w.seed)


def needle_qkv(B, H, Hkv, L, d, dtype=torch.bfloat16, seed=0, magnitude=8.0):
    """Mask probe: Q = K = 0 and V zero except one token per feature.

    Feature e of V is `magnitude` at one position m_e (spread over the whole
    sequence, seeded) and 0 elsewhere, so output feature e of row n is
    magnitude times the weight row n gives token m_e: a token wrongly included
    in or excluded from a row moves that feature by magnitude / (tokens
    attended).  magnitude 8 keeps |O| <= 8, where bf16 output rounding stays
    below 0.016.
    """
    g = torch.Generator().manual_seed(seed)
    q = torch.zeros(B, H, L, d, dtype=dtype)
    k = torch.zeros(B, Hkv, L, d, dtype=dtype)
    v = torch.zeros(B, Hkv, L, d, dtype=torch.float32)
    pos = torch.randint(0, L, (B, Hkv, d), generator=g)
    v.scatter_(2, pos.unsqueeze(2), magnitude)
    return q, k, v.to(dtype)


def spike_qkv(B, H, Hkv, L, d, dtype=torch.bfloat16, seed=0, alpha=3.0):
    """Mask probe through the logit path: N(0,1) Q, K, V plus, per (b, kv head),
    a set of positions whose key is alpha * u and every query gets + alpha * u
    (u a fixed random unit direction scaled to norm sqrt(d)), so those keys
    dominate any row that attends them exactly."""
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(B, H, L, d, generator=g)
    k = torch.randn(B, Hkv, L, d, generator=g)
    v = torch.randn(B, Hkv, L, d, generator=g)
    u = torch.randn(d, generator=g)
    u = u / u.norm() * (d ** 0.5)
    n_spikes = max(1, L // 97)
    pos = torch.randint(0, L, (B, Hkv, n_spikes), generator=g)
    for b in range(B):
        for hk in range(Hkv):
            k[b, hk, pos[b, hk]] = alpha * u
    q = q * 0.25 + alpha * u
    return q.to(dtype), k.to(dtype), v.to(dtype)


def spike_at_qkv(B, H, Hkv, L, d, positions, chunks=(), C=1, dtype=torch.bfloat16, seed=0, alpha=3.0):
    """Mask probe with spikes at chosen places: N(0,1) Q, K, V; the keys at
    `positions`, and every key of the chunks in `chunks` (chunk c covers
    [cC, cC + C)), are set to alpha * u in every (b, kv head), and every query
    gets + alpha * u (u a seeded direction of norm sqrt(d)).  A row that
    attends one of those keys, or the summary of a wholly spiked chunk, is
    dominated by it, so a single key wrongly in or out of a window, or a
    summary wrongly visible or hidden, moves the row by O(1)."""
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(B, H, L, d, generator=g)
    k = torch.randn(B, Hkv, L, d, generator=g)
    v = torch.randn(B, Hkv, L, d, generator=g)
    u = torch.randn(d, generator=g)
    u = u / u.norm() * (d ** 0.5)
    idx = sorted({int(p) for p in positions if 0 <= p < L})
    for c in chunks:
        idx.extend(range(c * C, min((c + 1) * C, L)))
    if idx:
        k[:, :, torch.tensor(sorted(set(idx)))] = alpha * u
    q = q * 0.25 + alpha * u
    return q.to(dtype), k.to(dtype), v.to(dtype)


def window_edge_positions(L, W, C, anchors):
    """Key positions that sit on the window and chunk edges of the rows in
    `anchors`: for row n the first and the last key before its window
    (n - W + 1, n - W), the key two before it, and the last token of the
    last chunk wholly before the window.  Geometry only."""
    pos = set()
    for n in anchors:
        lo = n - W + 1
        pos.update((lo, lo - 1, lo - 2))
        if lo > 0 and lo // C > 0:
            pos.add((lo // C) * C - 1)
    return sorted(p for p in pos if 0 <= p < L)
