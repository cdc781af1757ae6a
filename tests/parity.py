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


# Gradients (bf16 storage and products, fp32 accumulation), row-normwise per
# row of the last axis (a (b, h, n) row of dQ, a key row of dK / dV), scaled
# by the row's term magnitude T (oracle.backward_terms: per entry, the sum of
# the absolute values of the terms the entry sums):
#     max_r ||got_r - ref_r||_inf / max(||T_r||_inf, GRAD_FLOOR * max T)
# Rounding each term to bf16 (the weights dS and P are rounded before their
# products) moves an entry by up to 2^-8 of its term magnitude whatever the
# terms' cancellation, so that is the scale; a row whose terms cancel (several
# equal keys, one key taking all the weight) is still held to its own terms,
# not to the tensor's largest entry.  The floor only covers rows whose every
# term is exactly zero.
GRAD_ROW_REL = 2e-2
GRAD_FLOOR = 1e-3


def grad_row_err(got, ref, terms):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    terms = np.asarray(terms, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    d = ref.shape[-1]
    g = got.reshape(-1, d)
    r = ref.reshape(-1, d)
    t = terms.reshape(-1, d)
    den = np.maximum(t.max(axis=1), GRAD_FLOOR * max(float(t.max()), 1e-30))
    return float((np.abs(g - r).max(axis=1) / den).max())


def assert_grad_parity(got, ref, terms, what=""):
    """bf16 gradients: row-normwise error relative to the rows' term
    magnitudes (see GRAD_ROW_REL) within GRAD_ROW_REL; returns the error."""
    got = np.asarray(got, dtype=np.float64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite gradient"
    assert np.all(np.asarray(terms) >= np.abs(np.asarray(ref)) * (1 - 1e-12) - 1e-300), f"{what}: |ref| > terms"
    err = grad_row_err(got, ref, terms)
    assert err <= GRAD_ROW_REL, f"{what}: row-normwise error {err:.3e} > {GRAD_ROW_REL} (of the rows' term magnitudes)"
    return err
