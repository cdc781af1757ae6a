"""MI355X-native EVA attention (FlashEVA's fused window + summary attention).

The compute lives in libeva.so (hand-written HIP for gfx950 behind the C ABI
in include/eva.h); `eva` is the torch-facing binding, `inputs` the seeded
synthetic workloads.  Importing the package does not load the library; the
first call does, and raises if it is not built.
"""
from .eva import (Cache, build_summaries, cache_append, cache_fill, decode_step, prefill,  # noqa: F401
                  prefill_attention)
