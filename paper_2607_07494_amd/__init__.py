"""GIFT gradient codec for AMD Instinct MI355X (gfx950).

The HIP library ``libgift.so`` (C ABI in ``include/gift.h``) holds the whole
hot path; :mod:`paper_2607_07494_amd.gift` is its thin Python binding.
"""

from .gift import (  # noqa: F401
    BF16, F32, KERNELS, SCALE_LOCAL, SCALE_SHARED, SIDE_BOTH, SIDE_INPUT, SIDE_OUTPUT,
    CholFactor, Context, Factor, GiftError, decode, decode_batch, encode, encode_mxfp4, encode_noalloc,
    factor_update_batch, reduce_local, reduce_local_mxfp4, scale_grid, statistics,
)
