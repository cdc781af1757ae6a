"""The C ABI library loads, exports every symbol include/eva.h declares, and
rejects bad arguments with the documented status codes before touching the
GPU (no compute call is made here)."""
import ctypes
import os
import re

import pytest

from paper_2511_00576_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    return _lib.load()


def header_functions():
    with open(os.path.join(ROOT, "include", "eva.h")) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(eva_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = header_functions()
    for fn in ("eva_build_summaries", "eva_prefill", "eva_decode_step", "eva_cache_append"):
        assert fn in names
    assert sorted(_lib.SYMBOLS) == names


def test_library_exports_every_declared_symbol(lib):
    for name in header_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    assert lib.eva_status_string(0) == b"ok"
    for code in (-1, -2, -3, -4):
        assert lib.eva_status_string(code) not in (b"ok", b"unknown status")
    assert lib.eva_status_string(7) == b"unknown status"


FAKE = ctypes.c_void_p(0x10000)  # aligned, never dereferenced: validation fails first


def prefill_call(lib, **kw):
    a = dict(Q=FAKE, K=FAKE, V=FAKE, O=FAKE, B=1, H=4, H_kv=2, L=64, d=64, W=8, C=4, dtype=_lib.EVA_BF16,
             Ks=FAKE, Vs=FAKE, cache=None)
    a.update(kw)
    return lib.eva_prefill(a["Q"], a["K"], a["V"], a["O"], a["B"], a["H"], a["H_kv"], a["L"], a["d"], a["W"],
                           a["C"], a["dtype"], a["Ks"], a["Vs"], a["cache"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(H=3, H_kv=2), _lib.EVA_ERR_INVALID),
    (dict(W=0), _lib.EVA_ERR_INVALID),
    (dict(C=0), _lib.EVA_ERR_INVALID),
    (dict(L=0), _lib.EVA_ERR_INVALID),
    (dict(B=0), _lib.EVA_ERR_INVALID),
    (dict(Q=None), _lib.EVA_ERR_INVALID),
    (dict(Ks=None), _lib.EVA_ERR_INVALID),
    (dict(Q=ctypes.c_void_p(0x10008)), _lib.EVA_ERR_INVALID),
    (dict(d=96), _lib.EVA_ERR_UNSUPPORTED),
    (dict(d=256), _lib.EVA_ERR_UNSUPPORTED),
    (dict(dtype=5), _lib.EVA_ERR_UNSUPPORTED),
    (dict(C=100000), _lib.EVA_ERR_UNSUPPORTED),
])
def test_prefill_rejects(lib, kw, code):
    assert prefill_call(lib, **kw) == code


def make_cache(**kw):
    a = dict(B=1, H=4, H_kv=2, d=64, W=8, C=4, dtype=_lib.EVA_BF16, window=0, R=32, S_max=32, n_tok=0,
             k_ring=0x10000, vt_ring=0x20000, k_sum=0x30000, vt_sum=0x40000)
    a.update(kw)
    return _lib.EvaCacheStruct(**a)


@pytest.mark.parametrize("kw,code", [
    (dict(R=16), _lib.EVA_ERR_INVALID),          # not a multiple of 32
    (dict(R=40), _lib.EVA_ERR_INVALID),
    (dict(W=30, C=4), _lib.EVA_ERR_CAPACITY),     # R = 32 < W + C - 1 = 33
    (dict(S_max=0), _lib.EVA_ERR_INVALID),
    (dict(k_ring=0), _lib.EVA_ERR_INVALID),
    (dict(vt_sum=0x40004), _lib.EVA_ERR_INVALID),  # misaligned
    (dict(H=3), _lib.EVA_ERR_INVALID),
    (dict(d=80), _lib.EVA_ERR_UNSUPPORTED),
    (dict(rf=2), _lib.EVA_ERR_INVALID),           # rf is 0 or 1
    (dict(rf=1, rf_lambda=float("nan")), _lib.EVA_ERR_INVALID),
    (dict(rf=1, rf_lambda=-0.1), _lib.EVA_ERR_INVALID),
])
def test_cache_validation(lib, kw, code):
    c = make_cache(**kw)
    assert lib.eva_cache_append(ctypes.byref(c), FAKE, FAKE, None) == code
    assert c.n_tok == 0


def test_decode_needs_a_token(lib):
    c = make_cache()
    assert lib.eva_decode_step(ctypes.byref(c), FAKE, FAKE, None, 0, None) == _lib.EVA_ERR_INVALID
    assert lib.eva_decode_workspace_bytes(ctypes.byref(c)) == 0


def test_decode_fp32_cache_validates_before_launch(lib):
    # fp32 caches decode too (their own kernel); malformed calls are still
    # refused before anything is enqueued
    c = make_cache(dtype=_lib.EVA_F32, n_tok=0)
    assert lib.eva_decode_step(ctypes.byref(c), FAKE, FAKE, None, 0, None) == _lib.EVA_ERR_INVALID
    c = make_cache(dtype=_lib.EVA_F32, n_tok=5)
    assert lib.eva_decode_step(ctypes.byref(c), None, FAKE, None, 0, None) == _lib.EVA_ERR_INVALID
    assert lib.eva_append_decode(ctypes.byref(c), FAKE, None, FAKE, FAKE, None, 0, None) == _lib.EVA_ERR_INVALID
    assert c.n_tok == 5


def test_append_capacity(lib):
    # C = 4: the token at p = 4k + 3 completes chunk k, whose summary is built
    # by that append; with S_max = 32 chunks 32 (p = 131) and 33 (p = 135) do
    # not fit.
    for p in (131, 135):
        c = make_cache(n_tok=p)
        assert lib.eva_cache_append(ctypes.byref(c), FAKE, FAKE, None) == _lib.EVA_ERR_CAPACITY
        assert c.n_tok == p
        assert lib.eva_append_decode(ctypes.byref(c), FAKE, FAKE, FAKE, FAKE, None, 0, None) == \
            _lib.EVA_ERR_CAPACITY
        assert c.n_tok == p


def test_append_decode_rejects(lib):
    c = make_cache(n_tok=5)
    f = lib.eva_append_decode
    assert f(ctypes.byref(c), FAKE, None, FAKE, FAKE, None, 0, None) == _lib.EVA_ERR_INVALID
    assert f(ctypes.byref(c), FAKE, FAKE, FAKE, None, None, 0, None) == _lib.EVA_ERR_INVALID
    c = make_cache(n_tok=5, dtype=_lib.EVA_F32)
    assert f(ctypes.byref(c), FAKE, FAKE, None, FAKE, None, 0, None) == _lib.EVA_ERR_INVALID
    assert c.n_tok == 5


def test_prefill_cache_mismatch(lib):
    c = make_cache(W=16)
    assert prefill_call(lib, cache=ctypes.byref(c)) == _lib.EVA_ERR_INVALID
    c = make_cache(S_max=32)
    assert prefill_call(lib, L=4 * 33, cache=ctypes.byref(c)) == _lib.EVA_ERR_CAPACITY


def test_prefill_validates_before_filling(lib):
    # the attention stage's limit on its tile count (B * H_kv * position
    # tiles < 2^31) is checked before the summaries and the cache fill are
    # launched: the call fails and the cache is left as it was
    B, L, C, W = 65535, 2 ** 30, 256, 8
    c = make_cache(B=B, H=1, H_kv=1, W=W, C=C, R=288, S_max=(L // C + 31) // 32 * 32)
    assert prefill_call(lib, B=B, H=1, H_kv=1, L=L, W=W, C=C, cache=ctypes.byref(c)) == _lib.EVA_ERR_UNSUPPORTED
    assert c.n_tok == 0


def test_length_limits(lib):
    # sequence lengths above 2^30 are refused before any launch; so is a
    # cache that already holds 2^30 tokens
    f = lib.eva_build_summaries
    assert f(FAKE, FAKE, FAKE, FAKE, 1, 1, 2 ** 30 + 1, 64, 4, 0, None) == _lib.EVA_ERR_UNSUPPORTED
    assert prefill_call(lib, L=2 ** 30 + 1) == _lib.EVA_ERR_UNSUPPORTED
    c = make_cache(n_tok=2 ** 30)
    assert lib.eva_cache_append(ctypes.byref(c), FAKE, FAKE, None) == _lib.EVA_ERR_CAPACITY
    assert c.n_tok == 2 ** 30
    r = make_rcache(max_tok=2 ** 30 + 1)
    assert lib.eva_rcache_append(ctypes.byref(r), FAKE, FAKE, None, None) == _lib.EVA_ERR_UNSUPPORTED


def test_summaries_rejects(lib):
    f = lib.eva_build_summaries
    assert f(FAKE, FAKE, FAKE, FAKE, 1, 1, 64, 64, 0, 0, None) == _lib.EVA_ERR_INVALID
    assert f(None, FAKE, FAKE, FAKE, 1, 1, 64, 64, 4, 0, None) == _lib.EVA_ERR_INVALID
    assert f(FAKE, FAKE, FAKE, FAKE, 1, 1, 64, 32, 4, 0, None) == _lib.EVA_ERR_UNSUPPORTED
    # fewer tokens than one chunk: nothing to do, no pointer needed
    assert f(None, None, None, None, 1, 1, 3, 64, 4, 0, None) == _lib.EVA_OK


def make_rcache(**kw):
    a = dict(B=2, H=4, H_kv=2, d=64, W=8, C=4, dtype=_lib.EVA_BF16, window=0, R=32, S_max=32, max_tok=100,
             n_tok=0x50000, arrive=0x60000, k_ring=0x10000, vt_ring=0x20000, k_sum=0x30000, vt_sum=0x40000)
    a.update(kw)
    return _lib.EvaRCacheStruct(**a)


@pytest.mark.parametrize("kw,code", [
    (dict(n_tok=0), _lib.EVA_ERR_INVALID),        # per-sequence counts are required
    (dict(arrive=0), _lib.EVA_ERR_INVALID),
    (dict(max_tok=0), _lib.EVA_ERR_INVALID),
    (dict(R=48), _lib.EVA_ERR_INVALID),
    (dict(W=30, C=4), _lib.EVA_ERR_CAPACITY),     # R = 32 < W + C - 1
    # C = 4: a sequence of 132 tokens completes 33 chunks > S_max = 32
    (dict(max_tok=132), _lib.EVA_ERR_CAPACITY),
    (dict(H=5), _lib.EVA_ERR_INVALID),
    (dict(d=96), _lib.EVA_ERR_UNSUPPORTED),
    (dict(rf=3), _lib.EVA_ERR_INVALID),
    (dict(rf=1, rf_lambda=float("inf")), _lib.EVA_ERR_INVALID),
])
def test_rcache_validation(lib, kw, code):
    c = make_rcache(**kw)
    assert lib.eva_rcache_append(ctypes.byref(c), FAKE, FAKE, None, None) == code
    assert lib.eva_rdecode_step(ctypes.byref(c), FAKE, FAKE, None, None, 0, None) == code
    assert lib.eva_rappend_decode(ctypes.byref(c), FAKE, FAKE, FAKE, FAKE, None, None, 0, None) == code
    assert lib.eva_rdecode_workspace_bytes(ctypes.byref(c)) == 0


def test_rcache_capacity_boundary(lib):
    # C = 4: 131 tokens complete 32 chunks = S_max, which fits
    c = make_rcache(max_tok=131)
    assert lib.eva_rcache_append(ctypes.byref(c), None, FAKE, None, None) == _lib.EVA_ERR_INVALID
    assert lib.eva_rappend_decode(ctypes.byref(c), FAKE, None, FAKE, FAKE, None, None, 0, None) == \
        _lib.EVA_ERR_INVALID


def test_cache_fill_rejects_misaligned(lib):
    c = make_cache()
    odd = ctypes.c_void_p(0x10008)
    f = lib.eva_cache_fill
    assert f(ctypes.byref(c), odd, FAKE, FAKE, FAKE, 64, None) == _lib.EVA_ERR_INVALID
    assert f(ctypes.byref(c), FAKE, odd, FAKE, FAKE, 64, None) == _lib.EVA_ERR_INVALID
    assert f(ctypes.byref(c), FAKE, FAKE, odd, FAKE, 64, None) == _lib.EVA_ERR_INVALID
    assert f(ctypes.byref(c), FAKE, FAKE, FAKE, odd, 64, None) == _lib.EVA_ERR_INVALID
    assert c.n_tok == 0
    r = make_rcache()
    assert lib.eva_rcache_fill(ctypes.byref(r), FAKE, FAKE, odd, FAKE, 64, FAKE, None) == _lib.EVA_ERR_INVALID


def test_rcache_fill_rejects(lib):
    c = make_rcache()
    f = lib.eva_rcache_fill
    assert f(ctypes.byref(c), FAKE, FAKE, FAKE, FAKE, 64, None, None) == _lib.EVA_ERR_INVALID  # no lens
    assert f(ctypes.byref(c), FAKE, FAKE, FAKE, FAKE, 0, FAKE, None) == _lib.EVA_ERR_INVALID
    assert f(ctypes.byref(c), FAKE, FAKE, None, FAKE, 64, FAKE, None) == _lib.EVA_ERR_INVALID
    # 33 complete chunks of a sequence that may keep all of them: S_max = 32 is short
    big = make_rcache(max_tok=4 * 33, W=8 + 4 * 33, R=160)
    assert f(ctypes.byref(big), FAKE, FAKE, FAKE, FAKE, 4 * 33, FAKE, None) == _lib.EVA_ERR_CAPACITY


def test_rdecode_and_generate_reject(lib):
    c = make_rcache(dtype=_lib.EVA_F32)
    assert lib.eva_rdecode_step(ctypes.byref(c), None, FAKE, None, None, 0, None) == _lib.EVA_ERR_INVALID
    c = make_rcache()
    g = lib.eva_generate
    assert g(ctypes.byref(c), FAKE, FAKE, FAKE, FAKE, 0, None, None, 0, None) == _lib.EVA_ERR_INVALID
    assert g(ctypes.byref(c), FAKE, None, FAKE, FAKE, 4, None, None, 0, None) == _lib.EVA_ERR_INVALID
    assert g(ctypes.byref(c), ctypes.c_void_p(0x10008), FAKE, FAKE, FAKE, 4, None, None, 0,
             None) == _lib.EVA_ERR_INVALID


def test_summaries_rf_rejects(lib):
    f = lib.eva_build_summaries_rf
    ok = dict(K=FAKE, V=FAKE, eps=FAKE, lam=0.1, Ks=FAKE, Vs=FAKE, B=1, H_kv=1, L=64, d=64, C=4, dtype=0)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(a["K"], a["V"], a["eps"], a["lam"], a["Ks"], a["Vs"], a["B"], a["H_kv"], a["L"], a["d"], a["C"],
                 a["dtype"], None)

    assert call(eps=None) == _lib.EVA_ERR_INVALID
    assert call(eps=ctypes.c_void_p(0x10004)) == _lib.EVA_ERR_INVALID  # misaligned
    assert call(lam=-0.5) == _lib.EVA_ERR_INVALID
    assert call(lam=float("nan")) == _lib.EVA_ERR_INVALID
    assert call(lam=float("inf")) == _lib.EVA_ERR_INVALID
    assert call(d=96) == _lib.EVA_ERR_UNSUPPORTED
    assert call(C=0) == _lib.EVA_ERR_INVALID
    # fewer tokens than one chunk: nothing to do, no pointer needed
    assert call(K=None, V=None, eps=None, Ks=None, Vs=None, L=3) == _lib.EVA_OK


@pytest.mark.parametrize("window,code", [(4, _lib.EVA_ERR_INVALID), (-1, _lib.EVA_ERR_INVALID)])
def test_prefill_rejects_unknown_window(lib, window, code):
    f = lib.eva_prefill_attention_ex
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1, 4, 2, 64, 64, 8, 4, 0, window, None) == code


@pytest.mark.parametrize("window", [4, -1])
def test_training_calls_reject_unknown_window(lib, window):
    f = lib.eva_prefill_forward_ex
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, 1, 4, 2, 64, 64, 8, 4, 0, window,
             None) == _lib.EVA_ERR_INVALID
    g = lib.eva_prefill_backward_ex
    assert g(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, 1, 4, 2, 64, 64,
             8, 4, 0, window, None) == _lib.EVA_ERR_INVALID


def test_noncausal_takes_no_cache(lib):
    c = make_cache(window=_lib.EVA_WINDOW_NONCAUSAL)
    assert lib.eva_cache_append(ctypes.byref(c), FAKE, FAKE, None) == _lib.EVA_ERR_INVALID
    c = make_cache()
    assert lib.eva_prefill_ex(FAKE, FAKE, FAKE, FAKE, 1, 4, 2, 64, 64, 8, 4, 0, _lib.EVA_WINDOW_NONCAUSAL, FAKE, FAKE,
                              ctypes.byref(c), None) == _lib.EVA_ERR_INVALID
    # a cache of another window variant
    c = make_cache(window=_lib.EVA_WINDOW_BLOCKED)
    assert lib.eva_prefill_ex(FAKE, FAKE, FAKE, FAKE, 1, 4, 2, 64, 64, 8, 4, 0, _lib.EVA_WINDOW_SLIDING, FAKE, FAKE,
                              ctypes.byref(c), None) == _lib.EVA_ERR_INVALID
    r = make_rcache(window=_lib.EVA_WINDOW_NONCAUSAL)
    assert lib.eva_rcache_append(ctypes.byref(r), FAKE, FAKE, None, None) == _lib.EVA_ERR_INVALID


def test_rf_noise_and_rf_cache_validation(lib):
    f = lib.eva_rf_noise
    assert f(FAKE, 0, 2, 4, 64, 1, None) == _lib.EVA_ERR_INVALID
    assert f(FAKE, 1, 2, -1, 64, 1, None) == _lib.EVA_ERR_INVALID
    assert f(FAKE, 1, 2, 4, 96, 1, None) == _lib.EVA_ERR_UNSUPPORTED
    assert f(None, 1, 2, 4, 64, 1, None) == _lib.EVA_ERR_INVALID
    assert f(ctypes.c_void_p(0x10004), 1, 2, 4, 64, 1, None) == _lib.EVA_ERR_INVALID
    assert f(None, 1, 2, 0, 64, 1, None) == _lib.EVA_OK  # nothing to draw
    # eva_prefill builds deterministic summaries: a cache of stochastic ones is refused
    c = make_cache(rf=1, rf_lambda=0.1, rf_seed=5)
    assert prefill_call(lib, cache=ctypes.byref(c)) == _lib.EVA_ERR_INVALID
    assert c.n_tok == 0
