"""MI355X (gfx950) MOD-DiT hot path: mask predictor + block-sparse attention.

The compute lives in libmoddit.so (HIP kernels behind the C ABI declared in
include/moddit.h); this package only binds it.
"""
from ._capi import *  # noqa: F401,F403
from ._capi import (EXPORTED, LIB_PATH, ModError, Stats, make_budget, make_params,  # noqa: F401
                    make_shape, raw_lib)
