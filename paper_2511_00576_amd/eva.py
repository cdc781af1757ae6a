"""Torch-facing binding of libeva: marshals device tensors and the current HIP
stream into the C ABI.  Every computation runs in the library's HIP kernels;
this module only checks shapes, allocates outputs with torch and forwards
pointers.  Tensors must live on a ROCm device; there is no CPU path.
"""
import ctypes

import torch

from . import _lib

_DTYPES = {torch.bfloat16: _lib.EVA_BF16, torch.float32: _lib.EVA_F32}


def _dtype_code(t: torch.Tensor) -> int:
    try:
        return _DTYPES[t.dtype]
    except KeyError:
        raise TypeError(f"unsupported dtype {t.dtype}; use bfloat16 or float32") from None


def _require_device(*ts):
    for t in ts:
        if not t.is_cuda:
            raise RuntimeError("EVA kernels run on the GPU only: tensors must be on a ROCm device")
        if not t.is_contiguous():
            raise ValueError("tensors must be contiguous")


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def build_summaries(K: torch.Tensor, V: torch.Tensor, C: int, out=None):
    """Chunk summaries. K, V: [B, Hkv, L, d] -> (Ksum, Vsum): [B, Hkv, L // C, d].
    `out` = (Ksum, Vsum) preallocated, else allocated here."""
    _require_device(K, V)
    B, Hkv, L, d = K.shape
    if out is None:
        Ks = torch.empty(B, Hkv, L // C, d, dtype=K.dtype, device=K.device)
        Vs = torch.empty_like(Ks)
    else:
        Ks, Vs = out
        _require_device(Ks, Vs)
        if tuple(Ks.shape) != (B, Hkv, L // C, d) or Vs.shape != Ks.shape or Ks.dtype != K.dtype:
            raise ValueError("summary buffers must be [B, Hkv, L // C, d] in the input dtype")
    lib = _lib.load()
    _lib.check("eva_build_summaries",
               lib.eva_build_summaries(_ptr(K), _ptr(V), _ptr(Ks), _ptr(Vs), B, Hkv, L, d, C, _dtype_code(K),
                                       _stream()))
    return Ks, Vs


def build_summaries_rf(K: torch.Tensor, V: torch.Tensor, eps: torch.Tensor, C: int, lam: float = 0.1, out=None):
    """Stochastic random-feature summaries.  K, V: [B, Hkv, L, d]; eps: fp32
    [B, Hkv, L // C, d] standard normal draws (one per chunk) -> (Ksum, Vsum)."""
    _require_device(K, V, eps)
    B, Hkv, L, d = K.shape
    if eps.dtype != torch.float32 or tuple(eps.shape) != (B, Hkv, L // C, d):
        raise ValueError("eps must be float32 [B, Hkv, L // C, d]")
    if out is None:
        Ks = torch.empty(B, Hkv, L // C, d, dtype=K.dtype, device=K.device)
        Vs = torch.empty_like(Ks)
    else:
        Ks, Vs = out
    lib = _lib.load()
    _lib.check("eva_build_summaries_rf",
               lib.eva_build_summaries_rf(_ptr(K), _ptr(V), _ptr(eps), float(lam), _ptr(Ks), _ptr(Vs), B, Hkv, L, d,
                                          C, _dtype_code(K), _stream()))
    return Ks, Vs


def rf_noise(B, Hkv, n_chunks, d, seed, device="cuda"):
    """Counter-based standard normal draws for the stochastic summaries:
    fp32 [B, Hkv, n_chunks, d], chunk c of (b, g) depending only on
    (seed, b * Hkv + g, c) (eva_rf_noise); the draws a cache with the same
    seed uses for the chunks its appends complete."""
    eps = torch.empty(B, Hkv, n_chunks, d, dtype=torch.float32, device=device)
    _require_device(eps)
    _lib.check("eva_rf_noise", _lib.load().eva_rf_noise(_ptr(eps), B, Hkv, n_chunks, d, int(seed), _stream()))
    return eps


class Cache:
    """Window + summary decode cache in device memory (see eva_cache in eva.h).

    k_ring [B, Hkv, R, d], vt_ring [B, Hkv, R // 8, d, 8] (values transposed
    per 8-slot tile), k_sum [B, Hkv, S_max, d], vt_sum [B, Hkv, S_max // 8, d, 8].
    The ring holds the
    last R positions (R >= W + C - 1, a multiple of 32); S_max bounds the number
    of chunk summaries, i.e. the tokens the cache can ever absorb.
    """

    def __init__(self, B, H, Hkv, d, W, C, max_tokens, dtype=torch.bfloat16, device="cuda", R=None,
                 fill=None, window=_lib.EVA_WINDOW_SLIDING, rf_lambda=None, rf_seed=0):
        if R is None:
            R = -(-(W + C - 1) // 32) * 32
        S_max = max(32, -(-(max_tokens // C + 1) // 32) * 32)
        mk = (lambda *s: torch.full(s, fill, dtype=dtype, device=device)) if fill is not None else \
            (lambda *s: torch.empty(*s, dtype=dtype, device=device))
        self.k_ring = mk(B, Hkv, R, d)
        self.vt_ring = mk(B, Hkv, R // 8, d, 8)
        self.k_sum = mk(B, Hkv, S_max, d)
        self.vt_sum = mk(B, Hkv, S_max // 8, d, 8)
        self.dtype = dtype
        self.struct = _lib.EvaCacheStruct(B=B, H=H, H_kv=Hkv, d=d, W=W, C=C, dtype=_DTYPES[dtype], window=window,
                                          R=R, S_max=S_max, n_tok=0, k_ring=self.k_ring.data_ptr(),
                                          vt_ring=self.vt_ring.data_ptr(), k_sum=self.k_sum.data_ptr(),
                                          vt_sum=self.vt_sum.data_ptr(), rf=int(rf_lambda is not None),
                                          rf_lambda=float(rf_lambda or 0.0), rf_seed=int(rf_seed))
        self._ws = None

    @property
    def n_tok(self) -> int:
        return int(self.struct.n_tok)

    @property
    def R(self) -> int:
        return int(self.struct.R)

    @property
    def S_max(self) -> int:
        return int(self.struct.S_max)

    def workspace(self):
        """Decode split workspace for the current length (cached, grown on demand)."""
        n = _lib.load().eva_decode_workspace_bytes(ctypes.byref(self.struct))
        if n == 0:
            return None
        if self._ws is None or self._ws.numel() * 4 < n:
            self._ws = torch.empty((n + 3) // 4, dtype=torch.float32, device=self.k_ring.device)
        return self._ws


def prefill(Q, K, V, W: int, C: int, cache: Cache = None, return_summaries: bool = False,
            window: int = _lib.EVA_WINDOW_SLIDING, out=None, summaries=None):
    """EVA prefill. Q [B, H, L, d]; K, V [B, Hkv, L, d] -> O [B, H, L, d].
    `window`: one of the EVA_WINDOW_* variants.  `out` (O) and `summaries`
    ((Ks, Vs), [B, Hkv, L // C, d]) may be preallocated."""
    _require_device(Q, K, V)
    B, H, L, d = Q.shape
    Hkv = K.shape[1]
    if K.shape != (B, Hkv, L, d) or V.shape != K.shape or Q.dtype != K.dtype or V.dtype != K.dtype:
        raise ValueError("Q [B,H,L,d], K and V [B,Hkv,L,d] of one dtype expected")
    n_chunks = L // C
    if out is None:
        O = torch.empty_like(Q)
    else:
        O = out
        _require_device(O)
        if O.shape != Q.shape or O.dtype != Q.dtype:
            raise ValueError("out must be [B, H, L, d] in the dtype of Q")
    if summaries is None:
        Ks = torch.empty(B, Hkv, n_chunks, d, dtype=Q.dtype, device=Q.device)
        Vs = torch.empty_like(Ks)
    else:
        Ks, Vs = summaries
        _require_device(Ks, Vs)
        if tuple(Ks.shape) != (B, Hkv, n_chunks, d) or Vs.shape != Ks.shape or Ks.dtype != Q.dtype:
            raise ValueError("summaries must be [B, Hkv, L // C, d] in the dtype of Q")
    lib = _lib.load()
    cref = ctypes.byref(cache.struct) if cache is not None else None
    _lib.check("eva_prefill_ex",
               lib.eva_prefill_ex(_ptr(Q), _ptr(K), _ptr(V), _ptr(O), B, H, Hkv, L, d, W, C, _dtype_code(Q), window,
                                  _ptr(Ks) if n_chunks else None, _ptr(Vs) if n_chunks else None, cref, _stream()))
    if return_summaries:
        return O, Ks, Vs
    return O


def prefill_attention(Q, K, V, Ks, Vs, W: int, C: int, out=None, window: int = _lib.EVA_WINDOW_SLIDING):
    """The fused window + summary attention alone, given summaries from
    build_summaries(K, V, C). Q [B, H, L, d] -> O [B, H, L, d]."""
    _require_device(Q, K, V)
    B, H, L, d = Q.shape
    Hkv = K.shape[1]
    if K.shape != (B, Hkv, L, d) or V.shape != K.shape or Q.dtype != K.dtype or V.dtype != K.dtype:
        raise ValueError("Q [B,H,L,d], K and V [B,Hkv,L,d] of one dtype expected")
    if Ks is not None and (tuple(Ks.shape) != (B, Hkv, L // C, d) or Vs.shape != Ks.shape):
        raise ValueError("summaries must be [B, Hkv, L // C, d]")
    O = torch.empty_like(Q) if out is None else out
    _require_device(O)
    _lib.check("eva_prefill_attention_ex",
               _lib.load().eva_prefill_attention_ex(_ptr(Q), _ptr(K), _ptr(V), _ptr(Ks), _ptr(Vs), _ptr(O), B, H,
                                                    Hkv, L, d, W, C, _dtype_code(Q), window, _stream()))
    return O


def cache_fill(cache: Cache, K, V, Ks, Vs):
    """Load the cache from a prefilled sequence (K, V [B, Hkv, L, d] and its
    summaries); n_tok becomes L."""
    _require_device(K, V)
    s = cache.struct
    B, Hkv, L, d = K.shape
    if (B, Hkv, d) != (s.B, s.H_kv, s.d) or K.dtype != cache.dtype or V.shape != K.shape:
        raise ValueError("K, V must be [B, Hkv, L, d] matching the cache")
    _lib.check("eva_cache_fill",
               _lib.load().eva_cache_fill(ctypes.byref(s), _ptr(K), _ptr(V), _ptr(Ks), _ptr(Vs), L, _stream()))


def cache_append(cache: Cache, k_new, v_new):
    """Append one token per sequence: k_new, v_new [B, Hkv, d]."""
    _require_device(k_new, v_new)
    s = cache.struct
    if tuple(k_new.shape) != (s.B, s.H_kv, s.d) or v_new.shape != k_new.shape or k_new.dtype != cache.dtype:
        raise ValueError("k_new, v_new must be [B, Hkv, d] in the cache dtype")
    _lib.check("eva_cache_append",
               _lib.load().eva_cache_append(ctypes.byref(s), _ptr(k_new), _ptr(v_new), _stream()))


def append_decode(cache: Cache, q, k_new, v_new, use_workspace: bool = True, out=None):
    """Fused cache_append(k_new, v_new) + decode_step(q) in one launch."""
    _require_device(q, k_new, v_new)
    s = cache.struct
    if tuple(q.shape) != (s.B, s.H, s.d) or q.dtype != cache.dtype:
        raise ValueError("q must be [B, H, d] in the cache dtype")
    if tuple(k_new.shape) != (s.B, s.H_kv, s.d) or v_new.shape != k_new.shape or k_new.dtype != cache.dtype:
        raise ValueError("k_new, v_new must be [B, Hkv, d] in the cache dtype")
    o = torch.empty_like(q) if out is None else out
    ws = cache.workspace() if use_workspace else None
    nbytes = ws.numel() * 4 if ws is not None else 0
    _lib.check("eva_append_decode",
               _lib.load().eva_append_decode(ctypes.byref(s), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(o), _ptr(ws),
                                             nbytes, _stream()))
    return o


def append_decode_noalloc(cache: Cache, q, k_new, v_new, out=None):
    """append_decode without a workspace: split partials go to the library's
    fixed device array (eva_append_decode_noalloc).  With `out` given the
    call allocates nothing."""
    _require_device(q, k_new, v_new)
    s = cache.struct
    if tuple(q.shape) != (s.B, s.H, s.d) or q.dtype != cache.dtype:
        raise ValueError("q must be [B, H, d] in the cache dtype")
    if tuple(k_new.shape) != (s.B, s.H_kv, s.d) or v_new.shape != k_new.shape or k_new.dtype != cache.dtype:
        raise ValueError("k_new, v_new must be [B, Hkv, d] in the cache dtype")
    o = torch.empty_like(q) if out is None else out
    _require_device(o)
    _lib.check("eva_append_decode_noalloc",
               _lib.load().eva_append_decode_noalloc(ctypes.byref(s), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(o),
                                                     _stream()))
    return o


def decode_step(cache: Cache, q, use_workspace: bool = True, out=None):
    """Attention output of the last appended position: q [B, H, d] -> o [B, H, d]."""
    _require_device(q)
    s = cache.struct
    if tuple(q.shape) != (s.B, s.H, s.d) or q.dtype != cache.dtype:
        raise ValueError("q must be [B, H, d] in the cache dtype")
    o = torch.empty_like(q) if out is None else out
    ws = cache.workspace() if use_workspace else None
    nbytes = ws.numel() * 4 if ws is not None else 0
    _lib.check("eva_decode_step",
               _lib.load().eva_decode_step(ctypes.byref(s), _ptr(q), _ptr(o), _ptr(ws), nbytes, _stream()))
    return o


class RaggedCache:
    """Decode cache whose sequences hold different numbers of tokens (see
    eva_rcache in eva.h).  Same arrays as Cache; the per-sequence token counts
    `n_tok` [B] (int32) and the library's arrival counters live on the device,
    so steps need no host-side state.  `max_tokens` bounds every sequence."""

    def __init__(self, B, H, Hkv, d, W, C, max_tokens, dtype=torch.bfloat16, device="cuda", R=None, fill=None,
                 window=_lib.EVA_WINDOW_SLIDING, rf_lambda=None, rf_seed=0):
        if R is None:
            R = -(-(W + C - 1) // 32) * 32
        S_max = max(32, -(-(max_tokens // C + 1) // 32) * 32)
        mk = (lambda *s: torch.full(s, fill, dtype=dtype, device=device)) if fill is not None else \
            (lambda *s: torch.empty(*s, dtype=dtype, device=device))
        self.k_ring = mk(B, Hkv, R, d)
        self.vt_ring = mk(B, Hkv, R // 8, d, 8)
        self.k_sum = mk(B, Hkv, S_max, d)
        self.vt_sum = mk(B, Hkv, S_max // 8, d, 8)
        self.n_tok = torch.zeros(B, dtype=torch.int32, device=device)
        self.arrive = torch.zeros(B, dtype=torch.int32, device=device)
        self.dtype = dtype
        self.struct = _lib.EvaRCacheStruct(B=B, H=H, H_kv=Hkv, d=d, W=W, C=C, dtype=_DTYPES[dtype], window=window,
                                           R=R, S_max=S_max, max_tok=max_tokens, n_tok=self.n_tok.data_ptr(),
                                           arrive=self.arrive.data_ptr(), k_ring=self.k_ring.data_ptr(),
                                           vt_ring=self.vt_ring.data_ptr(), k_sum=self.k_sum.data_ptr(),
                                           vt_sum=self.vt_sum.data_ptr(), rf=int(rf_lambda is not None),
                                           rf_lambda=float(rf_lambda or 0.0), rf_seed=int(rf_seed))
        n = _lib.load().eva_rdecode_workspace_bytes(ctypes.byref(self.struct))
        self.ws = torch.empty((n + 3) // 4, dtype=torch.float32, device=device) if n else None

    @property
    def R(self) -> int:
        return int(self.struct.R)

    @property
    def S_max(self) -> int:
        return int(self.struct.S_max)

    def _ws_args(self, use_workspace):
        if use_workspace and self.ws is not None:
            return _ptr(self.ws), self.ws.numel() * 4
        return ctypes.c_void_p(0), 0


def _active_ptr(active):
    if active is None:
        return ctypes.c_void_p(0)
    _require_device(active)
    if active.dtype != torch.int32:
        raise ValueError("active must be an int32 device tensor [B]")
    return _ptr(active)


def rcache_fill(cache: RaggedCache, K, V, Ks, Vs, lens):
    """Load a ragged cache from a right-padded prefill: K, V [B, Hkv, L, d] and
    their summaries; lens (int32 device [B]) are the valid lengths."""
    _require_device(K, V, lens)
    s = cache.struct
    B, Hkv, L, d = K.shape
    if (B, Hkv, d) != (s.B, s.H_kv, s.d) or K.dtype != cache.dtype or V.shape != K.shape:
        raise ValueError("K, V must be [B, Hkv, L, d] matching the cache")
    if lens.dtype != torch.int32 or tuple(lens.shape) != (B,):
        raise ValueError("lens must be an int32 device tensor [B]")
    _lib.check("eva_rcache_fill",
               _lib.load().eva_rcache_fill(ctypes.byref(s), _ptr(K), _ptr(V), _ptr(Ks), _ptr(Vs), L, _ptr(lens),
                                           _stream()))


def rcache_append(cache: RaggedCache, k_new, v_new, active=None):
    """Append one token to each active sequence: k_new, v_new [B, Hkv, d]."""
    _require_device(k_new, v_new)
    s = cache.struct
    if tuple(k_new.shape) != (s.B, s.H_kv, s.d) or v_new.shape != k_new.shape or k_new.dtype != cache.dtype:
        raise ValueError("k_new, v_new must be [B, Hkv, d] in the cache dtype")
    _lib.check("eva_rcache_append",
               _lib.load().eva_rcache_append(ctypes.byref(s), _ptr(k_new), _ptr(v_new), _active_ptr(active),
                                             _stream()))


def rdecode_step(cache: RaggedCache, q, active=None, out=None, use_workspace=True):
    """Output of each active sequence's last appended position: q [B, H, d].
    Rows of inactive or empty sequences keep the contents of `out`."""
    _require_device(q)
    s = cache.struct
    if tuple(q.shape) != (s.B, s.H, s.d) or q.dtype != cache.dtype:
        raise ValueError("q must be [B, H, d] in the cache dtype")
    o = torch.zeros_like(q) if out is None else out
    ws, nbytes = cache._ws_args(use_workspace)
    _lib.check("eva_rdecode_step",
               _lib.load().eva_rdecode_step(ctypes.byref(s), _ptr(q), _ptr(o), _active_ptr(active), ws, nbytes,
                                            _stream()))
    return o


def rappend_decode(cache: RaggedCache, q, k_new, v_new, active=None, out=None, use_workspace=True):
    """Fused rcache_append + rdecode_step of every active sequence in one launch."""
    _require_device(q, k_new, v_new)
    s = cache.struct
    if tuple(q.shape) != (s.B, s.H, s.d) or q.dtype != cache.dtype:
        raise ValueError("q must be [B, H, d] in the cache dtype")
    if tuple(k_new.shape) != (s.B, s.H_kv, s.d) or v_new.shape != k_new.shape or k_new.dtype != cache.dtype:
        raise ValueError("k_new, v_new must be [B, Hkv, d] in the cache dtype")
    o = torch.zeros_like(q) if out is None else out
    ws, nbytes = cache._ws_args(use_workspace)
    _lib.check("eva_rappend_decode",
               _lib.load().eva_rappend_decode(ctypes.byref(s), _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(o),
                                              _active_ptr(active), ws, nbytes, _stream()))
    return o


def generate(cache: RaggedCache, q, k, v, active=None, out=None, use_workspace=True):
    """T generation steps: q [T, B, H, d], k, v [T, B, Hkv, d] -> o [T, B, H, d]
    (token t of every active sequence appended, then decoded)."""
    _require_device(q, k, v)
    s = cache.struct
    T = q.shape[0]
    if tuple(q.shape) != (T, s.B, s.H, s.d) or tuple(k.shape) != (T, s.B, s.H_kv, s.d) or v.shape != k.shape:
        raise ValueError("q [T, B, H, d], k and v [T, B, Hkv, d] expected")
    if q.dtype != cache.dtype or k.dtype != cache.dtype or v.dtype != cache.dtype:
        raise ValueError("q, k, v must be in the cache dtype")
    o = torch.zeros_like(q) if out is None else out
    ws, nbytes = cache._ws_args(use_workspace)
    _lib.check("eva_generate",
               _lib.load().eva_generate(ctypes.byref(s), _ptr(q), _ptr(k), _ptr(v), _ptr(o), T, _active_ptr(active),
                                        ws, nbytes, _stream()))
    return o


def prefill_forward(Q, K, V, W: int, C: int, residual: bool = False, window: int = _lib.EVA_WINDOW_SLIDING):
    """Training forward under window variant `window` (EVA_WINDOW_*):
    summaries, O and the per-row log-sum-exp.  Returns (O, lse, Ks, Vs); lse
    is fp32 [B, H, L].  With `residual` (bf16) also the output's rounding
    residual O_lo: (O, lse, Ks, Vs, O_lo)."""
    _require_device(Q, K, V)
    B, H, L, d = Q.shape
    Hkv = K.shape[1]
    Ks, Vs = build_summaries(K, V, C)
    O = torch.empty_like(Q)
    O_lo = torch.empty_like(Q) if residual else None
    lse = torch.empty(B, H, L, dtype=torch.float32, device=Q.device)
    n_chunks = L // C
    _lib.check("eva_prefill_forward_ex",
               _lib.load().eva_prefill_forward_ex(_ptr(Q), _ptr(K), _ptr(V), _ptr(Ks) if n_chunks else None,
                                                  _ptr(Vs) if n_chunks else None, _ptr(O), _ptr(lse), _ptr(O_lo), B, H,
                                                  Hkv, L, d, W, C, _dtype_code(Q), window, _stream()))
    if residual:
        return O, lse, Ks, Vs, O_lo
    return O, lse, Ks, Vs


def prefill_backward(Q, K, V, Ks, Vs, O, lse, dO, W: int, C: int, workspace=None, O_lo=None,
                     window: int = _lib.EVA_WINDOW_SLIDING):
    """Gradients (dQ, dK, dV) of the EVA prefill for the output gradient dO
    (bf16, window variant `window`), from the training forward's O, lse and
    summaries under the same variant (and, if it kept one, its output
    residual O_lo)."""
    _require_device(Q, K, V, O, lse, dO)
    if O_lo is not None:
        _require_device(O_lo)
        if O_lo.shape != O.shape or O_lo.dtype != O.dtype:
            raise ValueError("O_lo must match O")
    B, H, L, d = Q.shape
    Hkv = K.shape[1]
    if dO.shape != Q.shape or O.shape != Q.shape or tuple(lse.shape) != (B, H, L) or lse.dtype != torch.float32:
        raise ValueError("O, dO [B, H, L, d] and fp32 lse [B, H, L] expected")
    lib = _lib.load()
    need = lib.eva_prefill_backward_workspace_bytes(B, H, Hkv, L, d, C)
    ws = workspace
    if ws is None or ws.numel() * ws.element_size() < need:
        ws = torch.empty((need + 3) // 4, dtype=torch.float32, device=Q.device)
    dQ = torch.empty_like(Q)
    dK = torch.empty_like(K)
    dV = torch.empty_like(V)
    n_chunks = L // C
    _lib.check("eva_prefill_backward_ex",
               lib.eva_prefill_backward_ex(_ptr(Q), _ptr(K), _ptr(V), _ptr(Ks) if n_chunks else None,
                                           _ptr(Vs) if n_chunks else None, _ptr(O), _ptr(O_lo), _ptr(dO), _ptr(lse),
                                           _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(ws), ws.numel() * ws.element_size(), B,
                                           H, Hkv, L, d, W, C, _dtype_code(Q), window, _stream()))
    return dQ, dK, dV
