"""Parity helpers: error metrics and oracle evaluation of sampled rows.

Tolerances (stated by the build target, applied in the tests):
  fp32 data path: max row-normwise relative error <= 1e-5, i.e.
      max_n ||gpu_n - ref_n||_inf / ||ref_n||_inf
  (element-wise relative error is meaningless where an output is ~0);
  bf16 inputs with fp32 accumulation: max absolute error <= 2e-2.
"""
import numpy as np
import torch

import oracle

F32_ROW_REL = 1e-5
BF16_ABS = 2e-2


def to64(t):
    return t.detach().to("cpu").double().numpy()


def row_rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    d = got.shape[-1]
    g = got.reshape(-1, d)
    r = ref.reshape(-1, d)
    num = np.abs(g - r).max(axis=1)
    den = np.abs(r).max(axis=1)
    return float((num / np.maximum(den, 1e-300)).max()) if num.size else 0.0


def max_abs_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.abs(got - ref).max()) if got.size else 0.0


def assert_parity(got, ref, dtype, what=""):
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    if dtype == torch.float32:
        e = row_rel_err(got, ref)
        assert e <= F32_ROW_REL, f"{what}: row-normwise relative error {e:.3e} > {F32_ROW_REL}"
    else:
        e = max_abs_err(got, ref)
        assert e <= BF16_ABS, f"{what}: max abs error {e:.3e} > {BF16_ABS}"
    return e


def edge_rows(L, W, C, extra, seed=0):
    """Rows around every boundary the method has, plus `extra` random rows."""
    rows = {0, 1, L - 1, L - 2}
    for n in (W - 2, W - 1, W, W + 1, W + C - 2, W + C - 1, W + C, 2 * C + W - 1, 2 * C + W):
        rows.add(n)
    for k in range(1, 6):
        for off in (-1, 0, 1):
            rows.add(k * C + W - 1 + off)
    rng = np.random.default_rng(seed)
    rows.update(rng.integers(0, L, size=extra).tolist())
    return np.array(sorted(r for r in rows if 0 <= r < L), dtype=np.int64)


def oracle_sampled(Q, K, V, W, C, heads, rows):
    """Oracle outputs at (b, h, rows) for each (b, h) in heads: {(b, h): [n_rows, d]}."""
    B, H, L, d = Q.shape
    G = H // K.shape[1]
    out, summ = {}, {}
    for b, h in heads:
        g = h // G
        if (b, g) not in summ:
            summ[(b, g)] = (to64(K[b, g]), to64(V[b, g])) + oracle.summaries(K[b, g], V[b, g], C)
        Kb, Vb, Ks, Vs = summ[(b, g)]
        out[(b, h)] = oracle.attend_rows(to64(Q[b, h, torch.from_numpy(rows)]), rows, Kb, Vb, Ks, Vs, W, C)
    return out


GRAD_NORM_REL = 2e-2


def assert_grad_parity(got, ref, what=""):
    """bf16 gradients: max |got - ref| <= 2e-2 * max |ref| over the tensor
    (normwise: the gradient entries span orders of magnitude, so an absolute
    bound would be meaningless at one scale and loose at another)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite gradient"
    scale = float(np.abs(ref).max()) if ref.size else 0.0
    err = float(np.abs(got - ref).max()) if ref.size else 0.0
    assert err <= GRAD_NORM_REL * max(scale, 1e-30), f"{what}: max abs error {err:.3e} > 2e-2 * {scale:.3e}"
    return err / max(scale, 1e-30)
