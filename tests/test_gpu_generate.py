"""GPU parity of ragged batched generation: a right-padded prefill loads a
ragged cache (every sequence at its own length), then generation steps
append one token per active sequence and decode it.

Sequence b's token at position p is (q, k, v)[b, :, p]; its prompt is
positions [0, lens[b]) and step t of its generation is position
lens[b] + (number of earlier steps it was active in).  The decode output
must equal the oracle's EVA row at that position over that sequence's own
tokens.  The prefill pads each prompt with tokens drawn from another seed
and scale, so a fill that copied padding would show; caches pre-filled
with NaN prove that no stale slot or unused summary row leaks in.
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


def padded_prefill_inputs(q, k, v, lens, seed):
    """Prompts of lens[b] tokens right-padded to max(lens) with foreign tokens."""
    L = int(max(lens))
    B, H, _, d = q.shape
    Hkv = k.shape[1]
    pad_k = inputs.normal((B, Hkv, L, d), seed + 1000, torch.float32) * 3.0
    pad_v = inputs.normal((B, Hkv, L, d), seed + 2000, torch.float32) * 3.0
    K = k[:, :, :L].clone()
    V = v[:, :, :L].clone()
    for b, n in enumerate(lens):
        K[b, :, n:] = pad_k[b, :, n:].to(k.dtype)
        V[b, :, n:] = pad_v[b, :, n:].to(v.dtype)
    return q[:, :, :L].contiguous(), K.contiguous(), V.contiguous()


def load_ragged(q, k, v, lens, W, C, max_tokens, seed, fill=None, window=oracle.SLIDING):
    B, H, _, d = q.shape
    Hkv = k.shape[1]
    Qp, Kp, Vp = (t.cuda() for t in padded_prefill_inputs(q, k, v, lens, seed))
    cache = eva.RaggedCache(B, H, Hkv, d, W, C, max_tokens=max_tokens, dtype=q.dtype, fill=fill, window=window)
    _, Ks, Vs = eva.prefill(Qp, Kp, Vp, W, C, return_summaries=True, window=window)
    eva.rcache_fill(cache, Kp, Vp, Ks, Vs, torch.tensor(lens, dtype=torch.int32, device="cuda"))
    return cache


class SequenceOracle:
    """Oracle rows of sequence b over its own tokens k[b], v[b] (by position)."""

    def __init__(self, q, k, v, W, C, window=oracle.SLIDING):
        self.q, self.W, self.C, self.window = q, W, C, window
        self.G = q.shape[1] // k.shape[1]
        self.kv = {}
        self.k, self.v = k, v

    def kv_of(self, b, g):
        if (b, g) not in self.kv:
            K64, V64 = to64(self.k[b, g]), to64(self.v[b, g])
            self.kv[(b, g)] = (K64, V64) + oracle.summaries(K64, V64, self.C)
        return self.kv[(b, g)]

    def rows(self, b, h, positions, qrows=None):
        """Rows at `positions`; the queries are q[b, h, positions] unless given."""
        pos = np.asarray(positions, dtype=np.int64)
        if qrows is None:
            qrows = self.q[b, h, torch.from_numpy(pos)]
        if self.window == oracle.SLIDING:
            return oracle.attend_rows(to64(qrows), pos, *self.kv_of(b, h // self.G), self.W, self.C)
        # causal variants: the summaries of the tokens up to the row suffice
        K64, V64, _, _ = self.kv_of(b, h // self.G)
        out = []
        for r, p in enumerate(pos):
            Ks, Vs = oracle.summaries(K64[: p + 1], V64[: p + 1], self.C)
            out.append(oracle.attend_rows_variant(to64(qrows[r:r + 1]), pos[r:r + 1], K64[: p + 1], V64[: p + 1],
                                                  Ks, Vs, self.W, self.C, self.window)[0])
        return np.stack(out)


def step_inputs(q, k, v, pos):
    """Per-sequence inputs at positions pos[b]: q [B, H, d], k, v [B, Hkv, d]."""
    idx = torch.as_tensor(pos)
    b = torch.arange(q.shape[0])
    return (q[b, :, idx].contiguous(), k[b, :, idx].contiguous(), v[b, :, idx].contiguous())


def run_steps(B, H, Hkv, d, W, C, lens, steps, seed, fill=None, active_fn=None, use_ws=True, max_tokens=None,
              check_every=1, fused=False, window=oracle.SLIDING, dtype=torch.bfloat16):
    print(f"ragged B{B} H{H}/{Hkv} d{d} W{W} C{C} lens={lens} steps={steps} fill={fill} ws={use_ws} "
          f"fused={fused} {dtype}", flush=True)
    total = max(lens) + steps
    q, k, v = inputs.qkv(B, H, Hkv, total, d, dtype, seed=seed)
    if max_tokens is None:
        max_tokens = total
    cache = load_ragged(q, k, v, lens, W, C, max_tokens, seed, fill=fill, window=window)
    assert cache.n_tok.cpu().tolist() == [min(n, max_tokens) for n in lens]
    orc = SequenceOracle(q, k, v, W, C, window)
    n = [min(x, max_tokens) for x in lens]
    sentinel = torch.full((B, H, d), 7.0, dtype=dtype, device="cuda")
    for t in range(steps):
        act = [True] * B if active_fn is None else [bool(active_fn(t, b)) for b in range(B)]
        active = None if active_fn is None else torch.tensor(act, dtype=torch.int32, device="cuda")
        pos = [min(n[b], total - 1) for b in range(B)]
        qs, ks, vs = (x.cuda() for x in step_inputs(q, k, v, pos))
        if fused:
            o = eva.rappend_decode(cache, qs, ks, vs, active=active, out=sentinel.clone(), use_workspace=use_ws)
        else:
            eva.rcache_append(cache, ks, vs, active=active)
            o = eva.rdecode_step(cache, qs, active=active, out=sentinel.clone(), use_workspace=use_ws)
        for b in range(B):
            if act[b] and n[b] < max_tokens:
                n[b] += 1
        if t % check_every and t != steps - 1:
            continue
        torch.cuda.synchronize()
        assert cache.n_tok.cpu().tolist() == n, f"step {t}"
        got = to64(o)
        for b in range(B):
            if not act[b] or n[b] == 0:
                assert np.all(got[b] == 7.0), f"step {t}: inactive sequence {b} was written"
                continue
            p = n[b] - 1  # a full sequence decodes this step's query over its last position
            for h in range(H):
                ref = orc.rows(b, h, [p], qrows=qs[b, h][None].cpu())
                assert_parity(got[b, h][None], ref, dtype, f"step {t} b{b} h{h} p={p}")
    return cache


@pytest.mark.parametrize("fused", [False, True])
def test_ragged_generation_crosses_chunks_and_wraps(fused):
    # R = 96 for W = 64, C = 16; 150 steps wrap every ring and make summaries
    # due at different steps for every sequence
    run_steps(4, 8, 2, 128, 64, 16, lens=[100, 37, 250, 1], steps=150, seed=41, check_every=7, fused=fused)


@pytest.mark.parametrize("fused", [False, True])
def test_ragged_generation_nan_cache_and_empty_prompt(fused):
    run_steps(3, 4, 2, 64, 40, 8, lens=[0, 77, 9], steps=70, seed=42, fill=float("nan"), check_every=3, fused=fused)


@pytest.mark.parametrize("fused", [False, True])
def test_ragged_generation_active_mask(fused):
    # sequence 1 pauses for steps 5..24, sequence 2 is active on even steps only
    def active(t, b):
        return not ((b == 1 and 5 <= t < 25) or (b == 2 and t % 2))
    run_steps(3, 8, 2, 128, 48, 16, lens=[60, 130, 200], steps=60, seed=43, active_fn=active, check_every=4, fused=fused)


@pytest.mark.parametrize("use_ws", [True, False])
@pytest.mark.parametrize("fused", [False, True])
def test_ragged_generation_split_and_unsplit(use_ws, fused):
    # B * Hkv = 2 units: with the workspace the rows split over many workgroups
    run_steps(2, 8, 1, 128, 256, 32, lens=[1500, 700], steps=40, seed=44, use_ws=use_ws, check_every=13,
              fused=fused)


@pytest.mark.parametrize("window", [oracle.CHUNK_ALIGNED, oracle.BLOCKED])
def test_ragged_window_variants(window):
    run_steps(3, 8, 2, 128, 48, 16, lens=[60, 130, 7], steps=70, seed=50, check_every=3, fused=True, window=window)


def test_ragged_window_of_one():
    run_steps(2, 4, 2, 128, 1, 8, lens=[20, 3], steps=30, seed=49, check_every=1, fused=True)


@pytest.mark.parametrize("fused", [False, True])
def test_ragged_full_sequences_stop_growing(fused):
    # max_tokens = 90: sequence 0 starts full, sequence 1 fills up mid-run
    run_steps(2, 4, 2, 128, 32, 8, lens=[95, 70], steps=30, seed=45, max_tokens=90, check_every=1, fused=fused)


@pytest.mark.parametrize("H,Hkv", [(32, 2), (48, 1)])
def test_ragged_head_groupings(H, Hkv):
    run_steps(2, H, Hkv, 128, 48, 16, lens=[200, 90], steps=12, seed=46, check_every=5)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_generate_equals_step_loop_and_oracle(dtype):
    B, H, Hkv, d, W, C, T = 3, 8, 2, 128, 64, 16, 40
    lens = [150, 33, 90]
    seed = 47
    total = max(lens) + T
    q, k, v = inputs.qkv(B, H, Hkv, total, d, dtype, seed=seed)
    pos = [[n + t for n in lens] for t in range(T)]
    qs = torch.stack([step_inputs(q, k, v, p)[0] for p in pos]).cuda()
    ks = torch.stack([step_inputs(q, k, v, p)[1] for p in pos]).cuda()
    vs = torch.stack([step_inputs(q, k, v, p)[2] for p in pos]).cuda()
    print("generate vs step loop", flush=True)
    c1 = load_ragged(q, k, v, lens, W, C, total, seed)
    o_gen = eva.generate(c1, qs, ks, vs)
    c2 = load_ragged(q, k, v, lens, W, C, total, seed)
    o_loop = torch.stack([(eva.rcache_append(c2, ks[t], vs[t]), eva.rdecode_step(c2, qs[t]))[1] for t in range(T)])
    torch.cuda.synchronize()
    assert torch.equal(o_gen, o_loop)
    assert c1.n_tok.cpu().tolist() == [n + T for n in lens]
    orc = SequenceOracle(q, k, v, W, C)
    got = to64(o_gen)
    for b in range(B):
        for h in (0, H - 1):
            ref = orc.rows(b, h, [lens[b] + t for t in range(T)])
            assert_parity(got[:, b, h], ref, dtype, f"b{b} h{h}")


def test_generate_graph_replays():
    # one captured graph of T steps, replayed from a freshly filled cache each
    # time, with eager work and synchronizations between the replays
    B, H, Hkv, d, W, C, T = 2, 8, 2, 128, 32, 8, 24
    lens = [70, 41]
    seed = 48
    total = max(lens) + T
    q, k, v = inputs.qkv(B, H, Hkv, total, d, torch.bfloat16, seed=seed)
    pos = [[n + t for n in lens] for t in range(T)]
    qs = torch.stack([step_inputs(q, k, v, p)[0] for p in pos]).cuda()
    ks = torch.stack([step_inputs(q, k, v, p)[1] for p in pos]).cuda()
    vs = torch.stack([step_inputs(q, k, v, p)[2] for p in pos]).cuda()
    Qp, Kp, Vp = (t.cuda() for t in padded_prefill_inputs(q, k, v, lens, seed))
    lens_d = torch.tensor(lens, dtype=torch.int32, device="cuda")
    cache = eva.RaggedCache(B, H, Hkv, d, W, C, max_tokens=total)
    _, Ks, Vs = eva.prefill(Qp, Kp, Vp, W, C, return_summaries=True)
    print("eager reference", flush=True)
    eva.rcache_fill(cache, Kp, Vp, Ks, Vs, lens_d)
    ref = eva.generate(cache, qs, ks, vs)
    torch.cuda.synchronize()
    out = torch.zeros_like(qs)
    graph = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        eva.rcache_fill(cache, Kp, Vp, Ks, Vs, lens_d)
        torch.cuda.synchronize()
        print("capture", flush=True)
        with torch.cuda.graph(graph, stream=s):
            eva.generate(cache, qs, ks, vs, out=out)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for r in range(3):
        print(f"replay {r}", flush=True)
        out.zero_()
        eva.rcache_fill(cache, Kp, Vp, Ks, Vs, lens_d)
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"replay {r}"
        assert cache.n_tok.cpu().tolist() == [n + T for n in lens]


def test_generation_workload_sampled():
    w = inputs.GENERATE_BF16
    lens = inputs.prompt_lengths(w)
    steps = 48
    total = max(lens) + steps
    print(f"full-size {w.name}: {steps} steps", flush=True)
    q, k, v = inputs.qkv(w.B, w.H, w.Hkv, total, w.d, w.dtype, seed=w.seed)
    cache = load_ragged(q, k, v, lens, w.W, w.C, max(lens) + w.steps, w.seed)
    pos = [[n + t for n in lens] for t in range(steps)]
    qs = torch.stack([step_inputs(q, k, v, p)[0] for p in pos]).cuda()
    ks = torch.stack([step_inputs(q, k, v, p)[1] for p in pos]).cuda()
    vs = torch.stack([step_inputs(q, k, v, p)[2] for p in pos]).cuda()
    o = eva.generate(cache, qs, ks, vs)
    torch.cuda.synchronize()
    assert cache.n_tok.cpu().tolist() == [n + steps for n in lens]
    orc = SequenceOracle(q, k, v, w.W, w.C)
    got = to64(o)
    rng = np.random.default_rng(w.seed)
    for b in sorted({0, w.B - 1, *rng.integers(0, w.B, size=4).tolist()}):
        for h in (0, w.H // 2 + 1, w.H - 1):
            ts = [0, steps // 2, steps - 1]
            ref = orc.rows(b, h, [lens[b] + t for t in ts])
            assert_parity(got[ts, b, h], ref, w.dtype, f"b{b} h{h}")


# fp32 ragged caches (fp32 decode kernel; the fused calls append, then decode)
@pytest.mark.parametrize("fused", [False, True])
def test_ragged_generation_fp32(fused):
    def active(t, b):
        return not (b == 1 and 5 <= t < 25)
    run_steps(4, 8, 2, 128, 64, 16, lens=[100, 37, 250, 1], steps=120, seed=45, check_every=7, fused=fused,
              active_fn=active, dtype=torch.float32)
    run_steps(3, 4, 2, 64, 40, 8, lens=[0, 77, 9], steps=50, seed=46, fill=float("nan"), check_every=5,
              fused=fused, max_tokens=110, dtype=torch.float32)


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_ragged_generation_rf_summaries(dtype):
    # ragged cache of stochastic summaries: prompts loaded from
    # eva_build_summaries_rf with the counter-based draws, every chunk the
    # generation completes summarized with its own draw; rows against the
    # oracle over summaries_rf of each sequence's tokens
    B, H, Hkv, d, W, C, steps, lam, seed = 3, 8, 2, 128, 48, 16, 60, 0.3, 99
    lens = [60, 130, 7]
    total = max(lens) + steps
    print(f"ragged rf generation {dtype}", flush=True)
    q, k, v = inputs.qkv(B, H, Hkv, total, d, dtype, seed=51)
    Qp, Kp, Vp = (t.cuda() for t in padded_prefill_inputs(q, k, v, lens, 51))
    cache = eva.RaggedCache(B, H, Hkv, d, W, C, max_tokens=total, dtype=dtype, fill=float("nan"), rf_lambda=lam,
                            rf_seed=seed)
    L = Kp.shape[2]
    eps = eva.rf_noise(B, Hkv, L // C, d, seed)
    Ks, Vs = eva.build_summaries_rf(Kp, Vp, eps, C, lam=lam)
    eva.rcache_fill(cache, Kp, Vp, Ks, Vs, torch.tensor(lens, dtype=torch.int32, device="cuda"))
    k64, v64 = to64(k), to64(v)
    n = list(lens)
    for t in range(steps):
        pos = list(n)
        qs, ks, vs = (x.cuda() for x in step_inputs(q, k, v, pos))
        o = eva.rappend_decode(cache, qs, ks, vs)
        n = [x + 1 for x in n]
        if t % 9 and t != steps - 1:
            continue
        torch.cuda.synchronize()
        got = to64(o)
        for b in range(B):
            p = n[b] - 1
            nc = (p + 1) // C
            for h in (0, H - 1):
                g = h // (H // Hkv)
                seq = b * Hkv + g
                e = oracle.rf_noise(seq + 1, max(nc, 1), d, seed)[seq, :nc]
                rK, rV = oracle.summaries_rf(k64[b, g, : p + 1], v64[b, g, : p + 1], e, C, lam)
                ref = oracle.attend_rows(to64(qs[b, h])[None], np.array([p]), k64[b, g, : p + 1], v64[b, g, : p + 1],
                                         rK, rV, W, C)
                assert_parity(got[b, h][None], ref, dtype, f"step {t} b{b} h{h} p={p}")
