#!/usr/bin/env python
"""EVA attention benchmark on one MI355X (gfx950).

Step = one pass of the whole hot path over one batch of the LLM-shaped
prefill workload (B=8, H=H_kv=32, L=4096, d=128, W=256, C=64, bf16):
  summaries -> fused window+summary prefill -> cache fill -> append -> decode.
Each part is bracketed by HIP events on the stream the kernels run on.
value = algorithmic prefill FLOPs per step / step time (TFLOP/s).

The generation workload (32 sequences, prompts of 1024-3072 tokens, H=32,
H_kv=8, d=128, W=256, C=16) is run for its 1024 generated tokens over 8 layer
caches (one generation step = append + decode in each layer; 8 layers keep
the working set above the Infinity Cache), one step captured as a HIP graph.

The decode workload (64 sequences, H=32, H_kv=8, d=128, 8192-token context
held as a 512-token window plus 60 chunk summaries of 128 tokens) is timed in
the same run: append + decode per token, over 4 rotating caches so the
151 MB working set is read from HBM rather than the 256 MB Infinity Cache;
the iterations are captured in one HIP graph so host launch latency does not
enter the kernel timing.

Prints ONE JSON line.  Algorithmic counts:
  prefill FLOPs  = B*H*4d*sum_n (w(n) + s(n))      (QK^T and PV of attended keys)
  prefill bytes  = Q + K + V + Ksum + Vsum + O     (fused attention kernel)
  summary bytes  = K + V + Ksum + Vsum
  decode bytes   = B*H_kv*(w + s)*d*2*e + q + o
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2516.6  # dense bf16 MFMA: 256 CU x 2.4 GHz x 4096 flop/clk/CU
N_CACHES = 4
N_LAYERS = 8
WARMUP_S = 0.25
PROFILE_DIR = os.path.join(ROOT, "profiles")
PREFILL_SOURCES = ("paper_2511_00576_amd/csrc/prefill_mfma.hip", "paper_2511_00576_amd/csrc/eva_device.hpp")
DECODE_SOURCES = ("paper_2511_00576_amd/csrc/decode.hip", "paper_2511_00576_amd/csrc/eva_device.hpp",
                  "paper_2511_00576_amd/build.py")


def attended(L, W, C):
    """sum_n (w(n) + s(n)) over n < L."""
    import numpy as np
    n = np.arange(L, dtype=np.int64)
    w = np.minimum(W, n + 1)
    start = n - W + 1
    s = np.where(start > 0, start // C, 0)
    return int((w + s).sum())


def attended_variant(L, W, C, variant):
    """sum_n (exact keys + summaries) attended by row n under a window variant
    (0 sliding, 1 chunk-aligned, 2 blocked, 3 non-causal blocks)."""
    import numpy as np
    n = np.arange(L, dtype=np.int64)
    if variant == 0:
        lo, hi = np.maximum(0, n - W + 1), n
    elif variant == 1:
        lo, hi = (np.maximum(0, n - W + 1) // C) * C, n
    else:
        lo = (n // W) * W
        hi = np.minimum(L, lo + W) - 1 if variant == 3 else n
    n_chunks = L // C
    s = lo // C
    if variant == 3:
        s = s + np.maximum(0, n_chunks - (hi // C + 1))
    return int((hi - lo + 1 + s).sum())


def prefill_counts(B, H, Hkv, L, d, W, C, e):
    nc = L // C
    flops = B * H * 4 * d * attended(L, W, C)
    attn_bytes = (2 * B * H * L * d + 2 * B * Hkv * L * d + 2 * B * Hkv * nc * d) * e
    summ_bytes = (2 * B * Hkv * L * d + 2 * B * Hkv * nc * d) * e
    return flops, attn_bytes, summ_bytes


def attn_bytes_of(B, H, Hkv, L, d, C, e):
    """Q + K + V + Ksum + Vsum reads and O write of the fused kernel."""
    return (2 * B * H * L * d + 2 * B * Hkv * L * d + 2 * B * Hkv * (L // C) * d) * e


def decode_counts(B, H, Hkv, d, W, C, p, e):
    w = min(W, p + 1)
    s = max(0, p - W + 1) // C
    return B * H * 4 * d * (w + s), B * Hkv * (w + s) * d * 2 * e + 2 * B * H * d * e


def _code_only(path, text):
    """Source text without comments and blank lines: the counters describe
    the code, which an edited comment does not change."""
    if path.endswith(".py"):
        lines = [l for l in text.splitlines() if not l.strip().startswith("#")]
    else:
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        lines = [re.sub(r"//.*", "", l) for l in text.splitlines()]
    return "\n".join(l.rstrip() for l in lines if l.strip())


def source_sha(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p)) as f:
            h.update(_code_only(p, f.read()).encode())
    return h.hexdigest()[:16]


def read_traffic(name, sources):
    """HBM bytes per launch from a committed counter summary, or None when
    missing or taken on a different kernel source."""
    path = os.path.join(PROFILE_DIR, name)
    if not os.path.exists(path):
        return None
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line:
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("source_sha") != source_sha(sources):
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model():
    """The host CPU's model name (/proc/cpuinfo, as lscpu reports it)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(w):
    """The oracle on a bounded sample of the prefill workload, on this host:
    all threads on two batch elements, then one thread on one (b, h) slice."""
    import numpy as np

    import oracle
    from paper_2511_00576_amd import inputs

    n_batch = 2  # two of the eight sequences, every head, every row
    q, k, v = inputs.workload_qkv(w)
    qs, ks, vs = q[:n_batch], k[:n_batch], v[:n_batch]
    threads = oracle.num_threads()
    t0 = time.perf_counter()
    oracle.prefill(qs, ks, vs, w.W, w.C)
    dt = time.perf_counter() - t0
    flops = n_batch * w.H * 4 * w.d * attended(w.L, w.W, w.C)
    # one (b, h) slice on one thread: its summaries and every row
    oracle.set_num_threads(1)
    try:
        t1 = time.perf_counter()
        Kb, Vb = k[0, 0].double().numpy(), v[0, 0].double().numpy()
        Ks, Vs = oracle.summaries(Kb, Vb, w.C)
        oracle.attend_rows(q[0, 0].double().numpy(), np.arange(w.L), Kb, Vb, Ks, Vs, w.W, w.C)
        dt1 = time.perf_counter() - t1
    finally:
        oracle.set_num_threads(threads)
    flops1 = 4 * w.d * attended(w.L, w.W, w.C)
    return {"value": flops / dt / 1e12, "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "nproc": os.cpu_count(),
            "sample": f"batch elements 0-{n_batch - 1} of {w.name} (all {w.H} heads, all {w.L} rows, "
                      f"summaries included), {dt:.2f} s wall on {threads} threads",
            "single_thread_slice": {"slice": f"(b, h) = (0, 0) of {w.name}: summaries and all {w.L} rows",
                                    "seconds": dt1, "gflops": flops1 / dt1 / 1e9}}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    # the GPU reaches its steady clocks only after ~0.1 s of load: 200 warmup
    # steps (about 0.1 s) before the timed ones
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--warmup-seconds", type=float, default=WARMUP_S,
                    help="minimum wall-clock length of the warmup (counter runs, which serialise every "
                         "dispatch, set 0)")
    ap.add_argument("--decode-iters", type=int, default=64, help="graph-captured decode tokens (x4 caches)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--decode-eager", action="store_true",
                    help="launch the decode iterations one by one instead of replaying a captured graph "
                         "(for per-dispatch counter runs)")
    ap.add_argument("--no-generate", action="store_true")
    ap.add_argument("--no-other-prefill", action="store_true",
                    help="skip the GQA and long-context prefill workloads")
    ap.add_argument("--gen-layers", type=int, default=N_LAYERS,
                    help="layer caches a generation step visits (working set beyond the Infinity Cache)")
    ap.add_argument("--gen-steps", type=int, default=None,
                    help="generated tokens per sequence (default: the workload's 1024)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a 1 GiB device-to-device copy (counter scaling for profiles)")
    ap.add_argument("--prefill-only", choices=sorted(PREFILL_ONLY),
                    help="profiling mode: only this prefill workload's summaries and fused attention "
                         "(--warmup launches, then --steps timed launches); prints its own JSON line")
    ap.add_argument("--backward-only", choices=("llm", "gqa"),
                    help="profiling mode: the training forward of this workload once, then --warmup and "
                         "--steps backward calls (dQ, dK, dV); prints its own JSON line")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path. The EVA step shards "
              "by (batch, kv head) with no exchange; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2511_00576_amd import eva, inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    eva._lib.load()
    dev = torch.device("cuda:0")
    if args.prefill_only:
        bench_prefill_only(args, torch, eva, inputs, dev)
        return
    if args.backward_only:
        bench_backward_only(args, torch, eva, inputs, dev)
        return
    w = inputs.LLM_BF16
    B, H, Hkv, L, d, W, C = w.B, w.H, w.Hkv, w.L, w.d, w.W, w.C
    e = 2

    print(f"# prefill workload {w.name}: generating inputs", file=sys.stderr, flush=True)
    q, k, v = (t.to(dev) for t in inputs.workload_qkv(w))
    kn = inputs.normal((B, Hkv, d), w.seed + 100, w.dtype).to(dev)
    vn = inputs.normal((B, Hkv, d), w.seed + 101, w.dtype).to(dev)
    qn = inputs.normal((B, H, d), w.seed + 102, w.dtype).to(dev)
    # two buffer sets (inputs, summaries, output, cache), used by turns, so
    # that no step starts on what the previous one left in the caches
    sets = []
    for r in range(2):
        qq, kk, vv = (q, k, v) if r == 0 else (q.clone(), k.clone(), v.clone())
        Ks_r = torch.empty(B, Hkv, L // C, d, dtype=w.dtype, device=dev)
        sets.append({"q": qq, "k": kk, "v": vv, "Ks": Ks_r, "Vs": torch.empty_like(Ks_r), "O": torch.empty_like(qq),
                     "cache": eva.Cache(B, H, Hkv, d, W, C, max_tokens=L + 1, dtype=w.dtype, device=dev),
                     "od": torch.empty_like(qn)})
    Ks, Vs, O = sets[0]["Ks"], sets[0]["Vs"], sets[0]["O"]

    # one step: summaries, cache fill (right after the summaries, while the
    # last rows of K and V are still in the caches), the fused attention,
    # then one appended token and a decode step with it (one fused launch)
    def step(i, ev=None):
        st = sets[i % 2]
        if ev: ev[0].record()
        eva.build_summaries(st["k"], st["v"], C, out=(st["Ks"], st["Vs"]))
        if ev: ev[1].record()
        eva.cache_fill(st["cache"], st["k"], st["v"], st["Ks"], st["Vs"])
        if ev: ev[2].record()
        eva.prefill_attention(st["q"], st["k"], st["v"], st["Ks"], st["Vs"], W, C, out=st["O"])
        if ev: ev[3].record()
        eva.append_decode(st["cache"], qn, kn, vn, out=st["od"])
        if ev: ev[4].record()

    if args.copy_calibration:
        a = torch.empty(1 << 29, dtype=torch.float16, device=dev)  # 1 GiB
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    # warm-up: at least --warmup steps and at least WARMUP_S seconds of them
    # (the clocks reach their steady state only after ~0.1 s of load)
    print(f"# warmup >= {args.warmup} steps and >= {args.warmup_seconds} s, steps {args.steps}", file=sys.stderr,
          flush=True)
    w0 = time.perf_counter()
    n_warm = 0
    while n_warm < args.warmup or time.perf_counter() - w0 < args.warmup_seconds:
        for i in range(10):
            step(i)
        n_warm += 10
        torch.cuda.synchronize()
    warm_s = time.perf_counter() - w0
    # the step time over K steps with no markers inside them; then K more
    # steps with an event between the parts for the breakdown
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for i in range(args.steps):
        step(i)
    t1.record()
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / args.steps
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    for i in range(args.steps):
        step(i, evs[i])
    torch.cuda.synchronize()

    def avg(i, j):
        return sum(ev[i].elapsed_time(ev[j]) for ev in evs) / len(evs)

    ms_summ, ms_fill, ms_attn, ms_app_dec = avg(0, 1), avg(1, 2), avg(2, 3), avg(3, 4)

    # training step of the same layer: forward with log-sum-exp, then the
    # backward for a random output gradient (algorithmic FLOPs: five products
    # per attended (row, key) pair, S recomputed once: 10 d)
    dO_t = torch.randn(B, H, L, d, device=dev).to(w.dtype)
    lse_t = torch.empty(B, H, L, dtype=torch.float32, device=dev)
    lib = eva._lib.load()
    ws_b = torch.empty((lib.eva_prefill_backward_workspace_bytes(B, H, Hkv, L, d, C) + 3) // 4, dtype=torch.float32,
                       device=dev)
    dQ_t, dK_t, dV_t = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    # the forward keeps its output's rounding residual, so the backward's row
    # dots D = dO . O are exact (the training path the tests pin row by row)
    Olo_t = torch.empty_like(O)

    def fwd_bwd(ev=None):
        if ev: ev[0].record()
        eva._lib.check("eva_prefill_forward", lib.eva_prefill_forward(
            eva._ptr(q), eva._ptr(k), eva._ptr(v), eva._ptr(Ks), eva._ptr(Vs), eva._ptr(O), eva._ptr(lse_t),
            eva._ptr(Olo_t), B, H, Hkv, L, d, W, C, eva._lib.EVA_BF16, eva._stream()))
        if ev: ev[1].record()
        eva._lib.check("eva_prefill_backward", lib.eva_prefill_backward(
            eva._ptr(q), eva._ptr(k), eva._ptr(v), eva._ptr(Ks), eva._ptr(Vs), eva._ptr(O), eva._ptr(Olo_t),
            eva._ptr(dO_t), eva._ptr(lse_t), eva._ptr(dQ_t), eva._ptr(dK_t), eva._ptr(dV_t), eva._ptr(ws_b),
            ws_b.numel() * 4, B, H, Hkv, L, d, W, C, eva._lib.EVA_BF16, eva._stream()))
        if ev: ev[2].record()

    fwd_bwd()
    n_tr = max(args.steps // 2, 1)
    tev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_tr)]
    for i in range(n_tr):
        fwd_bwd(tev[i])
    torch.cuda.synchronize()
    ms_fwd_t = sum(e[0].elapsed_time(e[1]) for e in tev) / n_tr
    ms_bwd_t = sum(e[1].elapsed_time(e[2]) for e in tev) / n_tr
    bwd_flops = B * H * 10 * d * attended(L, W, C)
    training = {"output_residual": True, "forward_lse_ms": ms_fwd_t, "backward_ms": ms_bwd_t, "backward_alg_flops": bwd_flops,
                "backward_tflops": bwd_flops / (ms_bwd_t * 1e-3) / 1e12,
                "backward_mfma_frac": bwd_flops / (ms_bwd_t * 1e-3) / 1e12 / PEAK_BF16_TFLOPS}
    del dO_t, dQ_t, dK_t, dV_t, ws_b, Olo_t

    # window variants of the fused kernel on the same inputs (summaries as built)
    variants = {}
    for var, name in ((1, "chunk_aligned"), (2, "blocked"), (3, "noncausal")):
        eva.prefill_attention(q, k, v, Ks, Vs, W, C, out=O, window=var)
        v0 = torch.cuda.Event(enable_timing=True)
        v1 = torch.cuda.Event(enable_timing=True)
        n_var = max(args.steps, 1)
        v0.record()
        for _ in range(n_var):
            eva.prefill_attention(q, k, v, Ks, Vs, W, C, out=O, window=var)
        v1.record()
        torch.cuda.synchronize()
        ms_v = v0.elapsed_time(v1) / n_var
        fl = B * H * 4 * d * attended_variant(L, W, C, var)
        variants[name] = {"attention_ms": ms_v, "alg_flops": fl, "tflops": fl / (ms_v * 1e-3) / 1e12,
                          "hbm_gbs": attn_bytes_of(B, H, Hkv, L, d, C, 2) / (ms_v * 1e-3) / 1e9}

    # stochastic random-feature summaries of the same K, V (one noise draw
    # per chunk, read once more: + n_chunks * d * 4 bytes per (b, kv head))
    eps = torch.randn(B, Hkv, L // C, d, device=dev)
    eva.build_summaries_rf(k, v, eps, C, lam=0.1, out=(Ks, Vs))
    r0 = torch.cuda.Event(enable_timing=True)
    r1 = torch.cuda.Event(enable_timing=True)
    n_rf = max(args.steps, 1)
    r0.record()
    for _ in range(n_rf):
        eva.build_summaries_rf(k, v, eps, C, lam=0.1, out=(Ks, Vs))
    r1.record()
    torch.cuda.synchronize()
    ms_summ_rf = r0.elapsed_time(r1) / n_rf
    flops, attn_bytes, summ_bytes = prefill_counts(B, H, Hkv, L, d, W, C, e)
    attn_gbs = attn_bytes / (ms_attn * 1e-3) / 1e9
    attn_tflops = flops / (ms_attn * 1e-3) / 1e12
    print(f"# step {ms_step:.3f} ms: summaries {ms_summ:.3f}, cache fill {ms_fill:.3f}, attention {ms_attn:.3f}, "
          f"append+decode {ms_app_dec:.3f}; stochastic summaries {ms_summ_rf:.3f}", file=sys.stderr,
          flush=True)

    traffic = read_traffic("prefill_attention_llm-bf16_traffic.txt", PREFILL_SOURCES)
    out = {
        "metric": "EVA prefill TFLOP/s (% MFMA peak); decode tokens/s + HBM GB/s (% peak)",
        "value": flops / (ms_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_run": {"steps": n_warm, "seconds": warm_s},
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic N(0,1), seeded",
        "config": {"workload": w.name, "B": B, "H": H, "H_kv": Hkv, "L": L, "d": d, "W": W, "C": C,
                   "step": "summaries + cache fill + fused prefill + fused append/decode",
                   "buffer_sets": 2},
        "roofline": {"bound": "hbm", "achieved": attn_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": attn_gbs / PEAK_HBM_GBS,
                     "traffic": traffic,
                     "kernel": "prefill_mfma_kernel<128> (eva_prefill_attention, bf16)"},
        "prefill": {"attention_ms": ms_attn, "attention_tflops": attn_tflops,
                    "attention_mfma_frac": attn_tflops / PEAK_BF16_TFLOPS,
                    "summaries_ms": ms_summ, "summaries_gbs": summ_bytes / (ms_summ * 1e-3) / 1e9,
                    "window_variants": variants,
                    "training": training,
                    "summaries_rf_ms": ms_summ_rf,
                    "summaries_rf_gbs": (summ_bytes + B * Hkv * (L // C) * d * 4) / (ms_summ_rf * 1e-3) / 1e9,
                    "cache_fill_ms": ms_fill, "append_decode_ms": ms_app_dec,
                    "alg_flops": flops, "alg_bytes_attention": attn_bytes, "alg_bytes_summaries": summ_bytes},
    }
    del q, k, v, O, Ks, Vs, sets

    if not args.no_other_prefill:
        out["prefill_workloads"] = bench_other_prefill(args, torch, eva, inputs, dev)
    if not args.no_decode:
        out["decode"] = bench_decode(args, torch, eva, inputs, dev)
    if not args.no_generate:
        out["generate"] = bench_generate(args, torch, eva, inputs, dev)

    if not args.no_cpu_baseline:
        print("# oracle baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(out), flush=True)


def prefill_only_workload(name, inputs):
    import dataclasses
    lw = inputs.LONG_BF16
    if name.startswith("long"):
        c = int(name[4:])
        return dataclasses.replace(lw, C=c, name=lw.name.replace("C256", f"C{c}"))
    return {"llm": inputs.LLM_BF16, "gqa": inputs.GQA_BF16, "kbench": inputs.KBENCH_BF16}[name]


def bench_prefill_only(args, torch, eva, inputs, dev):
    """One prefill workload alone (for per-kernel profiles): summaries once,
    then --warmup and --steps fused-attention launches."""
    wk = prefill_only_workload(args.prefill_only, inputs)
    print(f"# prefill-only {wk.name}", file=sys.stderr, flush=True)
    q, k, v = (t.to(dev) for t in inputs.workload_qkv(wk))
    Ks, Vs = eva.build_summaries(k, v, wk.C)
    O = torch.empty_like(q)
    for _ in range(args.warmup):
        eva.prefill_attention(q, k, v, Ks, Vs, wk.W, wk.C, out=O)
    torch.cuda.synchronize()
    a0 = torch.cuda.Event(enable_timing=True)
    a1 = torch.cuda.Event(enable_timing=True)
    n = max(args.steps, 1)
    a0.record()
    for _ in range(n):
        eva.prefill_attention(q, k, v, Ks, Vs, wk.W, wk.C, out=O)
    a1.record()
    torch.cuda.synchronize()
    ms = a0.elapsed_time(a1) / n
    flops = wk.B * wk.H * 4 * wk.d * attended(wk.L, wk.W, wk.C)
    tf = flops / (ms * 1e-3) / 1e12
    print(json.dumps({"prefill_only": wk.name, "launches": args.warmup + n, "attention_ms": ms, "alg_flops": flops,
                      "tflops": tf, "mfma_frac": tf / PEAK_BF16_TFLOPS,
                      "prefill_source_sha": source_sha(PREFILL_SOURCES)}), flush=True)


PREFILL_ONLY = ("llm", "gqa", "long64", "long128", "long256", "kbench")


def bench_backward_only(args, torch, eva, inputs, dev):
    """One workload's backward alone (for per-kernel profiles): the training
    forward with the output residual once, then --warmup and --steps
    backward calls into one workspace."""
    wk = {"llm": inputs.LLM_BF16, "gqa": inputs.GQA_BF16}[args.backward_only]
    print(f"# backward-only {wk.name}", file=sys.stderr, flush=True)
    q, k, v = (t.to(dev) for t in inputs.workload_qkv(wk))
    dO = inputs.normal((wk.B, wk.H, wk.L, wk.d), wk.seed + 7, wk.dtype).to(dev)
    O, lse, Ks, Vs, O_lo = eva.prefill_forward(q, k, v, wk.W, wk.C, residual=True)
    lib = eva._lib.load()
    ws = torch.empty((lib.eva_prefill_backward_workspace_bytes(wk.B, wk.H, wk.Hkv, wk.L, wk.d, wk.C) + 3) // 4,
                     dtype=torch.float32, device=dev)
    run = lambda: eva.prefill_backward(q, k, v, Ks, Vs, O, lse, dO, wk.W, wk.C, workspace=ws, O_lo=O_lo)
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    a0 = torch.cuda.Event(enable_timing=True)
    a1 = torch.cuda.Event(enable_timing=True)
    n = max(args.steps, 1)
    a0.record()
    for _ in range(n):
        run()
    a1.record()
    torch.cuda.synchronize()
    ms = a0.elapsed_time(a1) / n
    flops = wk.B * wk.H * 10 * wk.d * attended(wk.L, wk.W, wk.C)
    tf = flops / (ms * 1e-3) / 1e12
    print(json.dumps({"backward_only": wk.name, "calls": args.warmup + n, "backward_ms": ms, "alg_flops": flops,
                      "tflops": tf, "mfma_frac": tf / PEAK_BF16_TFLOPS}), flush=True)


def bench_other_prefill(args, torch, eva, inputs, dev):
    """The GQA workload, the long-context workload at C = 64, 128, 256
    (fixed W = 1024) and a workload shaped like the paper's kernel benchmark
    (B8 L16384 W256 C128): fused attention time, algorithmic TFLOP/s against the
    bf16 MFMA peak, and the summaries' time.  For the C sweep also the
    approximation side of the trade-off: on sampled rows, the relative
    distance of the EVA output from exact causal softmax attention over the
    whole prefix (computed here in fp32 with plain torch ops)."""
    import dataclasses
    import math
    res = {}
    lw = inputs.LONG_BF16
    cases = [(inputs.GQA_BF16, False)]
    cases += [(dataclasses.replace(lw, C=c, name=lw.name.replace("C256", f"C{c}")), True) for c in (64, 128, 256)]
    cases += [(inputs.KBENCH_BF16, False)]
    cached = {}
    for wk, sample in cases:
        print(f"# prefill workload {wk.name}", file=sys.stderr, flush=True)
        key = (wk.B, wk.H, wk.Hkv, wk.L, wk.d, wk.seed)
        if key not in cached:
            cached.clear()
            cached[key] = tuple(t.to(dev) for t in inputs.workload_qkv(wk))
        q, k, v = cached[key]
        Ks, Vs = eva.build_summaries(k, v, wk.C)
        O = torch.empty_like(q)
        n = max(args.steps, 1)

        def timed(fn):
            # the clocks drop while the inputs are drawn on the host: warm up
            # for ~0.2 s of this launch before timing
            fn()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            torch.cuda.synchronize()
            for _ in range(min(2000, int(0.2 / max(time.perf_counter() - t0, 1e-5)))):
                fn()
            a0 = torch.cuda.Event(enable_timing=True)
            a1 = torch.cuda.Event(enable_timing=True)
            a0.record()
            for _ in range(n):
                fn()
            a1.record()
            torch.cuda.synchronize()
            return a0.elapsed_time(a1) / n

        ms_summ = timed(lambda: eva.build_summaries(k, v, wk.C, out=(Ks, Vs)))
        ms_attn = timed(lambda: eva.prefill_attention(q, k, v, Ks, Vs, wk.W, wk.C, out=O))
        flops = wk.B * wk.H * 4 * wk.d * attended(wk.L, wk.W, wk.C)
        tf = flops / (ms_attn * 1e-3) / 1e12
        r = {"attention_ms": ms_attn, "alg_flops": flops, "tflops": tf, "mfma_frac": tf / PEAK_BF16_TFLOPS,
             "summaries_ms": ms_summ}
        if sample:
            G = wk.H // wk.Hkv
            errs = []
            for h in (0, 13, wk.H - 1):
                for row in (wk.W + wk.C, wk.L // 3, wk.L // 2, wk.L - 1):
                    qr = q[0, h, row].float()
                    kk = k[0, h // G, : row + 1].float()
                    vv = v[0, h // G, : row + 1].float()
                    pr = torch.softmax(kk @ qr / math.sqrt(wk.d), dim=0)
                    exact = pr @ vv
                    errs.append(float((O[0, h, row].float() - exact).norm() / exact.norm()))
            r["rel_dev_from_exact_mean"] = sum(errs) / len(errs)
            r["rel_dev_from_exact_max"] = max(errs)
            r["rel_dev_rows"] = "heads 0, 13, 31 x rows W+C, L/3, L/2, L-1"
        print(f"# {wk.name}: attention {ms_attn * 1e3:.1f} us ({tf:.0f} TFLOP/s, "
              f"{100 * tf / PEAK_BF16_TFLOPS:.1f}% MFMA), summaries {ms_summ * 1e3:.1f} us"
              + (f", deviation from exact {r['rel_dev_from_exact_mean']:.3f}" if sample else ""),
              file=sys.stderr, flush=True)
        res[wk.name] = r
        del Ks, Vs, O
    cached.clear()
    return res


def bench_decode(args, torch, eva, inputs, dev):
    dw = inputs.DECODE_BF16
    B, H, Hkv, d, W, C, ctx = dw.B, dw.H, dw.Hkv, dw.d, dw.W, dw.C, dw.context
    print(f"# decode workload {dw.name}: building {N_CACHES} caches", file=sys.stderr, flush=True)
    gen = torch.Generator(device=dev).manual_seed(dw.seed)
    qh = torch.randn(B, H, ctx, d, generator=gen, device=dev).to(dw.dtype)
    kh = torch.randn(B, Hkv, ctx, d, generator=gen, device=dev).to(dw.dtype)
    vh = torch.randn(B, Hkv, ctx, d, generator=gen, device=dev).to(dw.dtype)
    caches = [eva.Cache(B, H, Hkv, d, W, C, max_tokens=ctx + 1, dtype=dw.dtype, device=dev) for _ in range(N_CACHES)]
    eva.prefill(qh, kh, vh, W, C, cache=caches[0])
    del qh, kh, vh
    for c in caches[1:]:
        for name in ("k_ring", "vt_ring", "k_sum", "vt_sum"):
            getattr(c, name).copy_(getattr(caches[0], name))
        c.struct.n_tok = caches[0].struct.n_tok
    kn = torch.randn(B, Hkv, d, generator=gen, device=dev).to(dw.dtype)
    vn = torch.randn(B, Hkv, d, generator=gen, device=dev).to(dw.dtype)
    qn = torch.randn(B, H, d, generator=gen, device=dev).to(dw.dtype)
    od = torch.empty_like(qn)
    torch.cuda.synchronize()

    def token(c):
        c.struct.n_tok = ctx  # re-append position ctx: same work every iteration
        eva.append_decode(c, qn, kn, vn, out=od)

    def decode_only(c):
        eva.decode_step(c, qn, out=od)

    # eager reference for the graph replays
    token(caches[0])
    ref = od.clone()
    iters = args.decode_iters * N_CACHES
    if args.decode_eager:
        for i in range(iters):
            token(caches[i % N_CACHES])
        for c in caches:
            c.struct.n_tok = ctx + 1
        for i in range(iters):
            decode_only(caches[i % N_CACHES])
        torch.cuda.synchronize()
        return {"workload": dw.name, "eager_iterations": iters, "graph_matches_eager": None}
    stream = torch.cuda.Stream()
    graphs = {}
    for name, fn in (("token", token), ("decode", decode_only)):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for i in range(iters):
                fn(caches[i % N_CACHES])
        graphs[name] = g
    for c in caches:
        c.struct.n_tok = ctx + 1
    res = {}
    for name, g in graphs.items():
        g.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        reps = 3
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        res[name] = e0.elapsed_time(e1) / (reps * iters)
    graph_ok = bool(torch.equal(od, ref))
    p = ctx
    flops, nbytes = decode_counts(B, H, Hkv, d, W, C, p, 2)
    dec_gbs = nbytes / (res["decode"] * 1e-3) / 1e9
    traffic = read_traffic("decode_bf16_traffic.txt", DECODE_SOURCES)
    print(f"# decode {res['decode'] * 1e3:.1f} us/step ({dec_gbs:.0f} GB/s), append+decode "
          f"{res['token'] * 1e3:.1f} us/token-step", file=sys.stderr, flush=True)
    return {
        "workload": dw.name,
        "tokens_per_s": B / (res["token"] * 1e-3),
        "us_per_token_step": res["token"] * 1e3,  # fused append + decode (eva_append_decode)
        "decode_us": res["decode"] * 1e3,
        "hbm_gbs": dec_gbs,
        "roofline": {"bound": "hbm", "achieved": dec_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": dec_gbs / PEAK_HBM_GBS, "traffic": traffic,
                     "kernel": "decode_kernel<128> (eva_decode_step)"},
        "alg_bytes": nbytes,
        "alg_flops": flops,
        "rotating_caches": N_CACHES,
        "graph_matches_eager": graph_ok,
    }


def generation_counts(lens, B, H, Hkv, d, W, C, e):
    """Decode bytes and FLOPs of one step of every sequence at lengths `lens`
    (tokens held, the decoded query at position len - 1)."""
    nbytes = 2 * B * H * d * e
    flops = 0
    for n in lens:
        p = n - 1
        rows = min(W, p + 1) + max(0, p - W + 1) // C
        nbytes += Hkv * rows * d * 2 * e
        flops += H * 4 * d * rows
    return flops, nbytes


def bench_generate(args, torch, eva, inputs, dev):
    """Ragged batched generation: per step, every layer cache appends one token
    per sequence (building the summaries that fall due) and decodes it."""
    gw = inputs.GENERATE_BF16
    B, H, Hkv, d, W, C = gw.B, gw.H, gw.Hkv, gw.d, gw.W, gw.C
    T = gw.steps if args.gen_steps is None else args.gen_steps
    n_layers = args.gen_layers
    lens = inputs.prompt_lengths(gw)
    Lp = max(lens)
    print(f"# generation workload {gw.name}: {n_layers} layer caches, prompts {min(lens)}-{Lp}",
          file=sys.stderr, flush=True)
    gen = torch.Generator(device=dev).manual_seed(gw.seed)
    qh = torch.randn(B, H, Lp, d, generator=gen, device=dev).to(gw.dtype)
    kh = torch.randn(B, Hkv, Lp, d, generator=gen, device=dev).to(gw.dtype)
    vh = torch.randn(B, Hkv, Lp, d, generator=gen, device=dev).to(gw.dtype)
    _, Ks, Vs = eva.prefill(qh, kh, vh, W, C, return_summaries=True)
    del qh
    lens_d = torch.tensor(lens, dtype=torch.int32, device=dev)
    caches = [eva.RaggedCache(B, H, Hkv, d, W, C, max_tokens=Lp + T + 1, dtype=gw.dtype, device=dev)
              for _ in range(n_layers)]

    def fill_all():
        for c in caches:
            eva.rcache_fill(c, kh, vh, Ks, Vs, lens_d)

    qn = torch.randn(B, H, d, generator=gen, device=dev).to(gw.dtype)
    kn = torch.randn(B, Hkv, d, generator=gen, device=dev).to(gw.dtype)
    vn = torch.randn(B, Hkv, d, generator=gen, device=dev).to(gw.dtype)
    outs = [torch.zeros_like(qn) for _ in range(n_layers)]

    def gen_step():
        for c, o in zip(caches, outs):
            eva.rappend_decode(c, qn, kn, vn, out=o)

    def dec_step():
        for c, o in zip(caches, outs):
            eva.rdecode_step(c, qn, out=o)

    # eager reference of the first step
    fill_all()
    gen_step()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs]
    if args.decode_eager:
        # per-dispatch counter runs: T eager steps, then one plain decode per
        # layer at the final lengths; no graphs
        fill_all()
        for _ in range(T):
            gen_step()
        dec_step()
        torch.cuda.synchronize()
        return {"workload": gw.name, "eager_steps": T, "graph_matches_eager": None}
    stream = torch.cuda.Stream()
    graphs = {}
    fill_all()
    torch.cuda.synchronize()
    for name, fn in (("step", gen_step), ("decode", dec_step)):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            fn()
        graphs[name] = g
    # capture launched nothing: the caches still hold the prompts
    assert caches[0].n_tok.cpu().tolist() == lens
    graphs["step"].replay()
    torch.cuda.synchronize()
    graph_ok = all(torch.equal(o, r) for o, r in zip(outs, ref))

    # whole generation: T steps from the prompts
    fill_all()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(T):
        graphs["step"].replay()
    e1.record()
    torch.cuda.synchronize()
    ms_gen = e0.elapsed_time(e1)
    final = caches[0].n_tok.cpu().tolist()
    assert final == [n + T for n in lens], "generation did not advance every sequence"
    # decode kernel alone at the final lengths
    reps = 64
    graphs["decode"].replay()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(reps):
        graphs["decode"].replay()
    e1.record()
    torch.cuda.synchronize()
    us_dec = e0.elapsed_time(e1) * 1e3 / (reps * n_layers)
    flops, nbytes = generation_counts(final, B, H, Hkv, d, W, C, 2)
    dec_gbs = nbytes / (us_dec * 1e-6) / 1e9
    us_layer_step = ms_gen * 1e3 / (T * n_layers)
    print(f"# generation {us_layer_step:.1f} us per layer-step (fused append + decode), decode alone {us_dec:.1f} us "
          f"({dec_gbs:.0f} GB/s) at the final lengths", file=sys.stderr, flush=True)
    del caches, outs, graphs
    scaling = ragged_decode_scaling(torch, eva, gw, kh, vh, Ks, Vs, lens, qn, dev)
    return {
        "workload": gw.name,
        "layers": n_layers,
        "tokens_per_s_per_layer": B / (us_layer_step * 1e-6),
        "us_per_layer_step": us_layer_step,
        "generation_ms": ms_gen,
        "decode_us_final_lengths": us_dec,
        "roofline": {"bound": "hbm", "achieved": dec_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": dec_gbs / PEAK_HBM_GBS,
                     "kernel": "decode_kernel<128, ragged> (eva_rdecode_step)"},
        "alg_bytes_decode_final": nbytes,
        "alg_flops_decode_final": flops,
        "graph_matches_eager": graph_ok,
        "decode_batch_scaling": scaling,
    }


def ragged_decode_scaling(torch, eva, gw, kh, vh, Ks, Vs, lens, qn, dev):
    """How much of a small ragged decode launch is fixed cost: the decode
    kernel on the prompts replicated 1, 2 and 4 times along the batch (about
    400 MB of caches rotated at every size, beyond the Infinity Cache; one
    captured graph per size, replayed), and
    a least-squares fit time = fixed + bytes / bandwidth.  `fixed_share` is
    the fixed part's share of the 32-sequence launch (ramp-up, the tail of
    the longest sequences, launch)."""
    import numpy as np
    B, H, Hkv, d, W, C = gw.B, gw.H, gw.Hkv, gw.d, gw.W, gw.C
    rows = []
    for r in (1, 2, 4):
        lens_r = lens * r
        n_caches = 8 // r
        cat = lambda t: torch.cat([t] * r, dim=0)
        k_r, v_r, ks_r, vs_r = cat(kh), cat(vh), cat(Ks), cat(Vs)
        lens_d = torch.tensor(lens_r, dtype=torch.int32, device=dev)
        q_r = cat(qn)
        caches = [eva.RaggedCache(B * r, H, Hkv, d, W, C, max_tokens=max(lens) + 1, dtype=gw.dtype, device=dev)
                  for _ in range(n_caches)]
        for c in caches:
            eva.rcache_fill(c, k_r, v_r, ks_r, vs_r, lens_d)
        del k_r, v_r, ks_r, vs_r
        out = torch.empty_like(q_r)
        # one graph per size (eager launches of ~15 us kernels would time the host)
        g = torch.cuda.CUDAGraph()
        stream = torch.cuda.Stream()
        with torch.cuda.graph(g, stream=stream):
            for c in caches:
                eva.rdecode_step(c, q_r, out=out)
        for _ in range(10):
            g.replay()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        reps = 32
        e0.record()
        for _ in range(reps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / (reps * n_caches)
        rows.append((B * r, us, generation_counts(lens_r, B * r, H, Hkv, d, W, C, 2)[1]))
        del caches, out, q_r, g
    us = np.array([x[1] for x in rows])
    nb = np.array([x[2] for x in rows], dtype=np.float64)
    slope, fixed = np.polyfit(nb, us, 1)
    return {"lengths": "the prompts (1024-3072 tokens)", "batch": [x[0] for x in rows],
            "us": [float(x) for x in us], "alg_bytes": [int(x) for x in nb],
            "fixed_us": float(fixed), "asymptotic_gbs": float(1e-3 / slope),
            "fixed_share": float(fixed / us[0])}


if __name__ == "__main__":
    main()
