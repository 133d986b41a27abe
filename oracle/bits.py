"""Bit-level reference: bf16 decoding and the Compressed Row Mask (CRM).

Test infrastructure only (see ``oracle/__init__``).

CRM layout (paper Sec. 4.3.2, "CRM Kernel: Bit-wise Block-Sparse Attention
Execution"): every block row of the attention matrix is a bitmask with one bit
per key/value block, stored in aligned unsigned words.  The paper uses
``uint32`` segments; the enumeration order fixed by its forward iterator
(Appendix, "CRM Forward Iterator") is: segment by segment, and inside a
segment lowest set bit first, the block index being ``32 * segment + bit``.
Bit b of word w therefore stands for block ``32 w + b`` (LSB-first).

This library stores the same bits as little-endian ``uint64`` words: word w of
a row holds blocks ``64 w .. 64 w + 63`` with block ``64 w + b`` at bit b.  On
a little-endian machine the bytes are identical to the paper's ``uint32``
layout whenever a row holds an even number of 32-bit segments (the tests pin
this equivalence).  Mask shape: ``[H][n_qb][W]`` with ``W = ceil(n_kb / 64)``;
a head's mask is shared by every batch entry.  Bits at positions ``>= n_kb``
in the last word carry no block and are ignored (reading recorded in the
design notes).
"""

import numpy as np


def n_words_u64(n_kb):
    """Number of uint64 words in one CRM row covering ``n_kb`` key blocks."""
    return (int(n_kb) + 63) // 64


def bf16_bits_to_f64(bits):
    """Decode IEEE bfloat16 bit patterns (uint16) to float64.

    bfloat16 is the top half of an IEEE binary32 value, so the value is the
    binary32 number whose high 16 bits are ``bits`` and whose low 16 bits are
    zero; every bf16 value is exact in float64.
    """
    b = np.asarray(bits)
    if b.dtype != np.uint16:
        raise TypeError("expected uint16 bf16 bit patterns, got %s" % b.dtype)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def mask_bit(mask_bits, h, u, v):
    """1 if key block ``v`` is enabled for query block ``u`` of head ``h``."""
    word = int(mask_bits[h, u, v // 64])
    return (word >> (v % 64)) & 1


def block_mask(mask_bits, n_kb):
    """Decode a ``[H][n_qb][W]`` uint64 CRM array to bool ``[H][n_qb][n_kb]``.

    Straight from the definition: entry (h, u, v) is bit ``v mod 64`` of word
    ``v // 64`` of row (h, u).
    """
    mb = np.asarray(mask_bits, dtype=np.uint64)
    if mb.ndim != 3:
        raise ValueError("mask_bits must be [H][n_qb][W]")
    if mb.shape[2] != n_words_u64(n_kb):
        raise ValueError("row length %d words does not match n_kb=%d" % (mb.shape[2], n_kb))
    v = np.arange(n_kb)
    words = mb[:, :, v // 64]
    shifts = (v % 64).astype(np.uint64)
    return ((words >> shifts) & np.uint64(1)).astype(bool)


def active_blocks(mask_bits, h, u, n_kb):
    """Ascending list of enabled key blocks of CRM row (h, u): plain definition."""
    return [v for v in range(n_kb) if mask_bit(mask_bits, h, u, v)]


def crm_walk(segments_u32, n_kb=None):
    """Enumerate a CRM row the way the paper's forward iterator does.

    ``segments_u32`` is one row as 32-bit segments.  Empty segments are
    skipped; inside a segment the lowest set bit is reported first and then
    cleared, and the block index is the segment's base (32 per segment) plus
    the bit's position (count of trailing zeros).  The walk ends when the
    segments are exhausted (the iterator's end-of-row sentinel).  ``n_kb``, if
    given, drops positions past the last real block.
    """
    out = []
    for s, seg in enumerate(segments_u32):
        val = int(seg) & 0xFFFFFFFF
        while val:
            lowest = val & -val
            idx = 32 * s + lowest.bit_length() - 1
            if n_kb is None or idx < n_kb:
                out.append(idx)
            val ^= lowest
    return out
