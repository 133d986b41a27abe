"""Seeded synthetic inputs shared by the tests, the bench and the reference checks.

Input generation only: configurations, block-mask generators, bit packing and
Q/K/V tensors.  Holds none of the attention arithmetic, so it can serve both
the HIP library and the CPU reference without coupling them.
"""

from .configs import (  # noqa: F401
    Workload, TINY, WAN13B_480P, WAN14B_480P, WAN14B_720P, sweep_point,
    SWEEP_RHOS, SWEEP_BLKS, SWEEP_KINDS, NAMED, SHORT,
)
from .masks import make_masks, pack_rows, structured_head, uniform_head, block_centres  # noqa: F401
from .tensors import head_scales, masks_for, qkv_for, bf16_to_bits, sample_items  # noqa: F401
from .thresholds import threshold_maps, p_for_density, stratified_rows  # noqa: F401
