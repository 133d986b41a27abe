"""Reference mask instantiation from a threshold map (paper Sec. 4.1.2).

Test infrastructure only (see ``oracle/__init__``).

WEST stores, for every block (u, v) of a head, the smallest sparsity
threshold p at which the block joins the active set: the threshold map T
(Sec. 4.1.2, Eq. 2).  A binary mask for a target p is then one comparison per
block, M_p = 1[T <= p]; FAST picks p per layer, timestep and head
(Sec. 4.2.2), so a head's map is compared against one p per (layer, step).
The result is stored in the CRM layout of ``oracle.bits`` (LSB-first uint64
words, bits past the last key block zero).

Everything is float32 comparison (the map and the thresholds are float32
inputs, compared exactly as given) and plain bit packing.
"""

import numpy as np

from .bits import n_words_u64


def instantiate(T, p):
    """M[i, h, u, v] = 1[T[h, u, v] <= p[i, h]] as bool ``[n_p][H][n_qb][n_kb]``.

    ``T``: float32 ``[H][n_qb][n_kb]``; ``p``: float32 ``[n_p][H]``.  A NaN in
    either compares false (the block stays off).
    """
    T = np.asarray(T, dtype=np.float32)
    p = np.asarray(p, dtype=np.float32)
    if T.ndim != 3 or p.ndim != 2 or p.shape[1] != T.shape[0]:
        raise ValueError("T must be [H][n_qb][n_kb] and p [n_p][H]")
    return T[None, :, :, :] <= p[:, :, None, None]


def pack_crm(mask):
    """bool ``[..., n_kb]`` -> uint64 ``[..., W]``: block v at bit v % 64 of word v // 64.

    Written from the definition, one bit at a time (slow, obviously right).
    """
    mask = np.asarray(mask, dtype=bool)
    n_kb = mask.shape[-1]
    W = n_words_u64(n_kb)
    out = np.zeros(mask.shape[:-1] + (W,), dtype=np.uint64)
    for v in range(n_kb):
        bit = mask[..., v].astype(np.uint64) << np.uint64(v % 64)
        out[..., v // 64] |= bit
    return out


def instantiate_packed(T, p):
    """Instantiated masks in CRM form: uint64 ``[n_p][H][n_qb][W]``."""
    return pack_crm(instantiate(T, p))
