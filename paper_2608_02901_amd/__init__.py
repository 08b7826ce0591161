"""AnchorKV on AMD MI355X (gfx950): anchor-residual KV-cache compression and
decode attention over the compressed cache (arXiv 2608.02901).

The compute lives in libanchorkv.so (HIP kernels behind the C ABI of
include/anchorkv.h); this package only binds it.  Build it with
``python -m paper_2608_02901_amd.build``.
"""
from ._native import (BF16, BUDGET_COUNT, BUDGET_FRACTION, BUDGET_THETA, F32, SCALE_ABSMAX_LITERAL,  # noqa: F401
                      SCALE_ABSMAX_OUTER, SCALE_RMS, SCALE_NAIVE, RANK_UTILITY, RANK_COSINE, RANK_RESNORM,
                      RANK_ATTENTION, RANK_RANDOM, APPEND_ENCODED, APPEND_DENSE, AnchorKVError, Config, Plan, append, decode_attn, decode_step,
                      decode_step_noalloc, encode, export, last_error, lib, reconstruct, LIB_PATH)
