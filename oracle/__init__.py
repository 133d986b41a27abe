"""CPU reference ("oracle") for the block-sparse attention forward pass.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import or call
this package: only the tests, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code, constants or
helpers with the HIP library under ``paper_2606_23019_amd/``; both sides
receive the same seeded inputs from ``workloads/`` and nothing else.

Everything here is plain NumPy in float64 (or Python integers for the bit
work), written to be checked against the paper by eye:

* ``bits``       -- bf16 decoding, the Compressed Row Mask (CRM) bit layout of
                   Sec. 4.3.2 and the ascending active-block enumeration of the
                   CRM forward iterator (Appendix, "CRM Forward Iterator").
* ``masks``      -- mask instantiation M_p = 1[T <= p] from a threshold map
                   (Sec. 4.1.2) and CRM packing.
* ``fidelity``   -- Hellinger distance and Fidelity Score (Sec. 4.2.1, Eq. 3-4)
                   of threshold-map masks on sampled rows (Sec. 4.2.3).
* ``resize``     -- conservative bilinear-ceiling resize of masks and threshold
                   maps between resolutions (Sec. 4.3.1, Eq. 7).
* ``attention``  -- softmax attention restricted to the key blocks a query
                   block's CRM row enables (Sec. 4.3.2; mask instantiation
                   M_p = 1[T <= p] of Sec. 4.1.2 supplies the masks).

Pins (tests/test_oracle_pins.py) tie every function to facts fixed by the
paper or by mathematics: dense attention from a library routine for the
all-ones mask, brute force on tiny inputs, closed forms, invariances and the
paper's "64 uint32 loads for 256k tokens" layout figure.
"""

from .bits import (  # noqa: F401
    bf16_bits_to_f64,
    mask_bit,
    block_mask,
    active_blocks,
    crm_walk,
    n_words_u64,
)
from .masks import instantiate, instantiate_packed, pack_crm  # noqa: F401
from .fidelity import hellinger, fidelity_score, profile  # noqa: F401
from .resize import bilinear_ceil, resize_mask, resize_threshold_map  # noqa: F401
from .attention import (  # noqa: F401
    attention_block,
    attention,
    attention_sampled,
)
