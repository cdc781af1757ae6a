"""ctypes declarations of libeva.so (the C ABI in include/eva.h).

The library is loaded from this package's directory.  There is no fallback:
if libeva.so is missing or lacks a symbol, loading raises.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libeva.so")

EVA_OK = 0
EVA_ERR_INVALID = -1
EVA_ERR_UNSUPPORTED = -2
EVA_ERR_CAPACITY = -3
EVA_ERR_HIP = -4
EVA_BF16 = 0
EVA_F32 = 1
EVA_WINDOW_SLIDING = 0
EVA_WINDOW_CHUNK_ALIGNED = 1
EVA_WINDOW_BLOCKED = 2
EVA_WINDOW_NONCAUSAL = 3

# Every entry point include/eva.h declares.
SYMBOLS = (
    "eva_build_summaries",
    "eva_build_summaries_rf",
    "eva_rf_noise",
    "eva_prefill",
    "eva_prefill_attention",
    "eva_prefill_attention_ex",
    "eva_prefill_ex",
    "eva_prefill_forward",
    "eva_prefill_forward_ex",
    "eva_prefill_backward",
    "eva_prefill_backward_ex",
    "eva_prefill_backward_workspace_bytes",
    "eva_cache_fill",
    "eva_cache_append",
    "eva_decode_step",
    "eva_decode_workspace_bytes",
    "eva_append_decode",
    "eva_append_decode_noalloc",
    "eva_rcache_fill",
    "eva_rcache_append",
    "eva_rdecode_step",
    "eva_rdecode_workspace_bytes",
    "eva_rappend_decode",
    "eva_generate",
    "eva_status_string",
)


class EvaCacheStruct(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int), ("H", ctypes.c_int), ("H_kv", ctypes.c_int), ("d", ctypes.c_int),
        ("W", ctypes.c_int), ("C", ctypes.c_int), ("dtype", ctypes.c_int), ("window", ctypes.c_int),
        ("R", ctypes.c_int), ("S_max", ctypes.c_int), ("n_tok", ctypes.c_longlong),
        ("k_ring", ctypes.c_void_p), ("vt_ring", ctypes.c_void_p),
        ("k_sum", ctypes.c_void_p), ("vt_sum", ctypes.c_void_p),
        ("rf", ctypes.c_int), ("rf_lambda", ctypes.c_float), ("rf_seed", ctypes.c_ulonglong),
    ]


class EvaRCacheStruct(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int), ("H", ctypes.c_int), ("H_kv", ctypes.c_int), ("d", ctypes.c_int),
        ("W", ctypes.c_int), ("C", ctypes.c_int), ("dtype", ctypes.c_int), ("window", ctypes.c_int),
        ("R", ctypes.c_int), ("S_max", ctypes.c_int), ("max_tok", ctypes.c_int),
        ("n_tok", ctypes.c_void_p), ("arrive", ctypes.c_void_p),
        ("k_ring", ctypes.c_void_p), ("vt_ring", ctypes.c_void_p),
        ("k_sum", ctypes.c_void_p), ("vt_sum", ctypes.c_void_p),
        ("rf", ctypes.c_int), ("rf_lambda", ctypes.c_float), ("rf_seed", ctypes.c_ulonglong),
    ]


_lib = None


def load():
    """Load libeva.so and declare its signatures (raises if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built: run __graft_entry__.build() or "
                           "python paper_2511_00576_amd/build.py")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
    cp = ctypes.POINTER(EvaCacheStruct)
    lib.eva_build_summaries.restype = i
    lib.eva_build_summaries.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, vp]
    lib.eva_build_summaries_rf.restype = i
    lib.eva_build_summaries_rf.argtypes = [vp, vp, vp, ctypes.c_float, vp, vp, i, i, i, i, i, i, vp]
    lib.eva_rf_noise.restype = i
    lib.eva_rf_noise.argtypes = [vp, i, i, i, i, ctypes.c_ulonglong, vp]
    lib.eva_prefill.restype = i
    lib.eva_prefill.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, i, vp, vp, cp, vp]
    lib.eva_prefill_attention.restype = i
    lib.eva_prefill_attention.argtypes = [vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, i, vp]
    lib.eva_prefill_attention_ex.restype = i
    lib.eva_prefill_attention_ex.argtypes = [vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, i, i, vp]
    lib.eva_prefill_ex.restype = i
    lib.eva_prefill_ex.argtypes = [vp, vp, vp, vp, i, i, i, i, i, i, i, i, i, vp, vp, cp, vp]
    lib.eva_prefill_forward.restype = i
    lib.eva_prefill_forward.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, i, vp]
    lib.eva_prefill_forward_ex.restype = i
    lib.eva_prefill_forward_ex.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i, i, i, i, i, i, i, i, i, vp]
    lib.eva_prefill_backward.restype = i
    lib.eva_prefill_backward.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, i, i, i, i, i, i, i,
                                         i, vp]
    lib.eva_prefill_backward_ex.restype = i
    lib.eva_prefill_backward_ex.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, i, i, i, i, i, i,
                                            i, i, i, vp]
    lib.eva_prefill_backward_workspace_bytes.restype = sz
    lib.eva_prefill_backward_workspace_bytes.argtypes = [i, i, i, i, i, i]
    lib.eva_cache_fill.restype = i
    lib.eva_cache_fill.argtypes = [cp, vp, vp, vp, vp, i, vp]
    lib.eva_cache_append.restype = i
    lib.eva_cache_append.argtypes = [cp, vp, vp, vp]
    lib.eva_decode_step.restype = i
    lib.eva_decode_step.argtypes = [cp, vp, vp, vp, sz, vp]
    lib.eva_append_decode.restype = i
    lib.eva_append_decode.argtypes = [cp, vp, vp, vp, vp, vp, sz, vp]
    lib.eva_append_decode_noalloc.restype = i
    lib.eva_append_decode_noalloc.argtypes = [cp, vp, vp, vp, vp, vp]
    lib.eva_decode_workspace_bytes.restype = sz
    lib.eva_decode_workspace_bytes.argtypes = [cp]
    rp = ctypes.POINTER(EvaRCacheStruct)
    lib.eva_rcache_fill.restype = i
    lib.eva_rcache_fill.argtypes = [rp, vp, vp, vp, vp, i, vp, vp]
    lib.eva_rcache_append.restype = i
    lib.eva_rcache_append.argtypes = [rp, vp, vp, vp, vp]
    lib.eva_rdecode_step.restype = i
    lib.eva_rdecode_step.argtypes = [rp, vp, vp, vp, vp, sz, vp]
    lib.eva_rappend_decode.restype = i
    lib.eva_rappend_decode.argtypes = [rp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.eva_rdecode_workspace_bytes.restype = sz
    lib.eva_rdecode_workspace_bytes.argtypes = [rp]
    lib.eva_generate.restype = i
    lib.eva_generate.argtypes = [rp, vp, vp, vp, vp, i, vp, vp, sz, vp]
    lib.eva_status_string.restype = ctypes.c_char_p
    lib.eva_status_string.argtypes = [i]
    _lib = lib
    return lib


class EvaError(RuntimeError):
    def __init__(self, fn: str, status: int):
        msg = load().eva_status_string(status).decode()
        super().__init__(f"{fn} failed: {msg} ({status})")
        self.status = status


def check(fn: str, status: int) -> None:
    if status != EVA_OK:
        raise EvaError(fn, status)
