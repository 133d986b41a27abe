"""MI355X (gfx950) block-sparse video attention forward.

The compute lives in the HIP library ``libsa_bsattn.so`` (C ABI in
include/sa_bsattn.h); ``binding`` marshals torch tensors into it.
"""

__all__ = ["binding", "build"]
