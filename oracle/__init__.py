"""EVA oracle: fp64 CPU reference (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import
this package.  It wraps oracle/eva_oracle.c through ctypes and shares no code
with the HIP library.  Every array handed in is converted to contiguous
float64 numpy first, so callers may pass torch tensors (any dtype, any device
already copied to the host) or numpy arrays.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None

_dp = ctypes.POINTER(ctypes.c_double)
_lp = ctypes.POINTER(ctypes.c_long)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_build.LIB):
        _build.build()
    lib = ctypes.CDLL(_build.LIB)
    lib.eva_ref_visible_summaries.restype = ctypes.c_long
    lib.eva_ref_visible_summaries.argtypes = [ctypes.c_long, ctypes.c_long, ctypes.c_long]
    lib.eva_ref_summaries.restype = None
    lib.eva_ref_summaries.argtypes = [_dp, _dp, ctypes.c_long, ctypes.c_int, ctypes.c_long, _dp, _dp]
    lib.eva_ref_summaries_rf.restype = None
    lib.eva_ref_summaries_rf.argtypes = [_dp, _dp, _dp, ctypes.c_long, ctypes.c_int, ctypes.c_long, ctypes.c_double,
                                         _dp, _dp]
    lib.eva_ref_attend_row.restype = None
    lib.eva_ref_attend_row.argtypes = [_dp, _dp, _dp, _dp, _dp, ctypes.c_long, ctypes.c_int,
                                       ctypes.c_long, ctypes.c_long, _dp]
    lib.eva_ref_attend_rows.restype = None
    lib.eva_ref_attend_rows.argtypes = [_dp, _lp, ctypes.c_long, _dp, _dp, _dp, _dp, ctypes.c_int,
                                        ctypes.c_long, ctypes.c_long, _dp]
    lib.eva_ref_attend_rows_variant.restype = None
    lib.eva_ref_attend_rows_variant.argtypes = [_dp, _lp, ctypes.c_long, _dp, _dp, _dp, _dp, ctypes.c_long,
                                                ctypes.c_int, ctypes.c_long, ctypes.c_long, ctypes.c_int, _dp]
    lib.eva_ref_prefill_variant.restype = None
    lib.eva_ref_prefill_variant.argtypes = [_dp, _dp, _dp, _dp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                            ctypes.c_long, ctypes.c_int, ctypes.c_long, ctypes.c_long, ctypes.c_int,
                                            _dp, _dp]
    lib.eva_ref_prefill.restype = None
    lib.eva_ref_prefill.argtypes = [_dp, _dp, _dp, _dp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_long, ctypes.c_int, ctypes.c_long, ctypes.c_long, _dp, _dp]
    lib.eva_ref_backward_group.restype = None
    lib.eva_ref_backward_group.argtypes = [_dp, _dp, _dp, _dp, ctypes.c_int, ctypes.c_long, ctypes.c_int,
                                           ctypes.c_long, ctypes.c_long, _dp, _dp, _dp]
    lib.eva_ref_backward_group_variant.restype = None
    lib.eva_ref_backward_group_variant.argtypes = [_dp, _dp, _dp, _dp, ctypes.c_int, ctypes.c_long, ctypes.c_int,
                                                   ctypes.c_long, ctypes.c_long, ctypes.c_int, _dp, _dp, _dp]
    lib.eva_ref_backward_terms_variant.restype = None
    lib.eva_ref_backward_terms_variant.argtypes = [_dp, _dp, _dp, _dp, ctypes.c_int, ctypes.c_long, ctypes.c_int,
                                                   ctypes.c_long, ctypes.c_long, ctypes.c_int, _dp, _dp, _dp]
    lib.eva_ref_backward_terms.restype = None
    lib.eva_ref_backward_terms.argtypes = [_dp, _dp, _dp, _dp, ctypes.c_int, ctypes.c_long, ctypes.c_int,
                                           ctypes.c_long, ctypes.c_long, _dp, _dp, _dp]
    lib.eva_ref_philox4x32_10.restype = None
    lib.eva_ref_philox4x32_10.argtypes = [ctypes.POINTER(ctypes.c_uint), ctypes.POINTER(ctypes.c_uint),
                                          ctypes.POINTER(ctypes.c_uint)]
    lib.eva_ref_rf_noise.restype = None
    lib.eva_ref_rf_noise.argtypes = [_dp, ctypes.c_long, ctypes.c_long, ctypes.c_int, ctypes.c_ulonglong]
    lib.eva_ref_num_threads.restype = ctypes.c_int
    lib.eva_ref_num_threads.argtypes = []
    lib.eva_ref_set_num_threads.restype = None
    lib.eva_ref_set_num_threads.argtypes = [ctypes.c_int]
    _lib = lib
    return lib


def _f64(x):
    if hasattr(x, "detach"):  # torch tensor
        x = x.detach().to("cpu").double().numpy()
    return np.ascontiguousarray(x, dtype=np.float64)


def _ptr(a):
    return a.ctypes.data_as(_dp)


def num_threads() -> int:
    return int(_load().eva_ref_num_threads())


def set_num_threads(n: int) -> None:
    """Threads of the oracle's parallel loops from now on."""
    _load().eva_ref_set_num_threads(int(n))


def visible_summaries(n: int, W: int, C: int) -> int:
    """s(n): number of chunk summaries the query at position n attends."""
    return int(_load().eva_ref_visible_summaries(n, W, C))


def summaries(K, V, C: int):
    """Chunk summaries of one sequence. K, V: [L, d] -> (Ksum, Vsum): [L // C, d]."""
    K, V = _f64(K), _f64(V)
    L, d = K.shape
    n_chunks = L // C
    Ks = np.zeros((n_chunks, d))
    Vs = np.zeros((n_chunks, d))
    _load().eva_ref_summaries(_ptr(K), _ptr(V), L, d, C, _ptr(Ks), _ptr(Vs))
    return Ks, Vs


def summaries_rf(K, V, eps, C: int, lam: float = 0.1):
    """Stochastic random-feature summaries of one sequence: K, V [L, d], eps
    [L // C, d] (one N(0, I) draw per chunk) -> (Ksum, Vsum) [L // C, d]."""
    K, V, eps = _f64(K), _f64(V), _f64(eps)
    L, d = K.shape
    n_chunks = L // C
    assert eps.shape == (n_chunks, d)
    Ks = np.zeros((n_chunks, d))
    Vs = np.zeros((n_chunks, d))
    if n_chunks:
        _load().eva_ref_summaries_rf(_ptr(K), _ptr(V), _ptr(eps), L, d, C, float(lam), _ptr(Ks), _ptr(Vs))
    return Ks, Vs


def attend_rows(Qrows, rows, K, V, Ksum, Vsum, W: int, C: int):
    """Rows `rows` (positions) of one sequence; Qrows[r] is the query at rows[r]."""
    Qrows, K, V = _f64(Qrows), _f64(K), _f64(V)
    Ksum, Vsum = _f64(Ksum), _f64(Vsum)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    d = K.shape[1]
    assert Qrows.shape == (rows.shape[0], d)
    if Ksum.shape[0] == 0:  # keep a valid pointer for empty summary sets
        Ksum = np.zeros((1, d))
        Vsum = np.zeros((1, d))
    out = np.zeros((rows.shape[0], d))
    _load().eva_ref_attend_rows(_ptr(Qrows), rows.ctypes.data_as(_lp), rows.shape[0], _ptr(K), _ptr(V),
                                _ptr(Ksum), _ptr(Vsum), d, W, C, _ptr(out))
    return out


def prefill(Q, K, V, W: int, C: int, return_summaries: bool = False):
    """Whole EVA prefill. Q: [B, H, L, d]; K, V: [B, Hkv, L, d] -> O: [B, H, L, d] (fp64)."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    B, H, L, d = Q.shape
    Hkv = K.shape[1]
    assert K.shape == (B, Hkv, L, d) and V.shape == K.shape and H % Hkv == 0
    n_chunks = L // C
    O = np.zeros_like(Q)
    Ks = np.zeros((B, Hkv, max(n_chunks, 1), d))
    Vs = np.zeros((B, Hkv, max(n_chunks, 1), d))
    _load().eva_ref_prefill(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), B, H, Hkv, L, d, W, C,
                            _ptr(Ks), _ptr(Vs))
    if return_summaries:
        return O, Ks[:, :, :n_chunks], Vs[:, :, :n_chunks]
    return O


# Window variants (eva_ref_attend_row_variant): 0 sliding, 1 chunk-aligned,
# 2 blocked, 3 non-causal blocked.
SLIDING, CHUNK_ALIGNED, BLOCKED, NONCAUSAL = 0, 1, 2, 3


def attend_rows_variant(Qrows, rows, K, V, Ksum, Vsum, W: int, C: int, variant: int):
    """Rows of one sequence under a window variant; K, V hold the whole
    sequence (L = K.shape[0]) and Ksum, Vsum all its L // C summaries."""
    Qrows, K, V = _f64(Qrows), _f64(K), _f64(V)
    Ksum, Vsum = _f64(Ksum), _f64(Vsum)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    L, d = K.shape
    assert Ksum.shape[0] == L // C
    if Ksum.shape[0] == 0:
        Ksum = np.zeros((1, d))
        Vsum = np.zeros((1, d))
    out = np.zeros((rows.shape[0], d))
    _load().eva_ref_attend_rows_variant(_ptr(Qrows), rows.ctypes.data_as(_lp), rows.shape[0], _ptr(K), _ptr(V),
                                        _ptr(Ksum), _ptr(Vsum), L, d, W, C, int(variant), _ptr(out))
    return out


def prefill_variant(Q, K, V, W: int, C: int, variant: int):
    """Whole prefill under a window variant: Q [B, H, L, d]; K, V [B, Hkv, L, d]."""
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    B, H, L, d = Q.shape
    Hkv = K.shape[1]
    n_chunks = L // C
    O = np.zeros_like(Q)
    Ks = np.zeros((B, Hkv, max(n_chunks, 1), d))
    Vs = np.zeros((B, Hkv, max(n_chunks, 1), d))
    _load().eva_ref_prefill_variant(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), B, H, Hkv, L, d, W, C, int(variant),
                                    _ptr(Ks), _ptr(Vs))
    return O


def backward(Q, K, V, dO, W: int, C: int, variant: int = SLIDING):
    """Gradients of the EVA prefill (window variant `variant`, default the
    sliding window): Q, dO [B, H, L, d]; K, V [B, Hkv, L, d] -> (dQ, dK, dV)
    in fp64, for the loss whose gradient with respect to O is dO."""
    Q, K, V, dO = _f64(Q), _f64(K), _f64(V), _f64(dO)
    B, H, L, d = Q.shape
    Hkv = K.shape[1]
    G = H // Hkv
    dQ = np.zeros_like(Q)
    dK = np.zeros_like(K)
    dV = np.zeros_like(V)
    lib = _load()
    for b in range(B):
        for g in range(Hkv):
            q = np.ascontiguousarray(Q[b, g * G:(g + 1) * G])
            go = np.ascontiguousarray(dO[b, g * G:(g + 1) * G])
            dq = np.zeros_like(q)
            dk = np.zeros((L, d))
            dv = np.zeros((L, d))
            lib.eva_ref_backward_group_variant(_ptr(q), _ptr(np.ascontiguousarray(K[b, g])),
                                               _ptr(np.ascontiguousarray(V[b, g])), _ptr(go), G, L, d, W, C,
                                               int(variant), _ptr(dq), _ptr(dk), _ptr(dv))
            dQ[b, g * G:(g + 1) * G] = dq
            dK[b, g] = dk
            dV[b, g] = dv
    return dQ, dK, dV


def backward_terms(Q, K, V, dO, W: int, C: int, variant: int = SLIDING):
    """Term magnitudes of backward() (rounding-error scales, not part of the
    method): for every gradient entry the sum of the absolute values of the
    terms it sums, carried through the same steps.  Same shapes as
    backward(); returns (Tq, Tk, Tv)."""
    Q, K, V, dO = _f64(Q), _f64(K), _f64(V), _f64(dO)
    B, H, L, d = Q.shape
    Hkv = K.shape[1]
    G = H // Hkv
    Tq = np.zeros_like(Q)
    Tk = np.zeros_like(K)
    Tv = np.zeros_like(V)
    lib = _load()
    for b in range(B):
        for g in range(Hkv):
            q = np.ascontiguousarray(Q[b, g * G:(g + 1) * G])
            go = np.ascontiguousarray(dO[b, g * G:(g + 1) * G])
            tq = np.zeros_like(q)
            tk = np.zeros((L, d))
            tv = np.zeros((L, d))
            lib.eva_ref_backward_terms_variant(_ptr(q), _ptr(np.ascontiguousarray(K[b, g])),
                                               _ptr(np.ascontiguousarray(V[b, g])), _ptr(go), G, L, d, W, C,
                                               int(variant), _ptr(tq), _ptr(tk), _ptr(tv))
            Tq[b, g * G:(g + 1) * G] = tq
            Tk[b, g] = tk
            Tv[b, g] = tv
    return Tq, Tk, Tv


def philox4x32_10(counter, key):
    """One Philox4x32-10 block: counter (4 words), key (2 words) -> 4 words."""
    c = (ctypes.c_uint * 4)(*[int(x) & 0xffffffff for x in counter])
    k = (ctypes.c_uint * 2)(*[int(x) & 0xffffffff for x in key])
    out = (ctypes.c_uint * 4)()
    _load().eva_ref_philox4x32_10(c, k, out)
    return [int(x) for x in out]


def rf_noise(n_seq: int, n_chunks: int, d: int, seed: int):
    """Counter-based standard normal draws [n_seq, n_chunks, d] (see
    eva_ref_rf_noise): the noise of chunk c of sequence-head s = b * H_kv + g."""
    eps = np.zeros((n_seq, n_chunks, d))
    if eps.size:
        _load().eva_ref_rf_noise(_ptr(eps), n_seq, n_chunks, d, int(seed) & 0xffffffffffffffff)
    return eps
