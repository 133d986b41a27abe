"""Reference conservative resize of block masks and threshold maps (paper Sec. 4.3.1, Eq. 7).

Test infrastructure only (see ``oracle/__init__``).

Masks are built once at a base resolution and reused at others (Sec. 4.3.1):
the block map is resampled with bilinear interpolation and a ceiling,

    R_target(u, v) = ceil( Phi(R_base, u / s_h, v / s_w) ),

with s_h = n_q_target / n_q_base and s_w = n_k_target / n_k_base, so target
block (u, v) samples the base map at x = u * n_q_base / n_q_target,
y = v * n_k_base / n_k_target.  Phi is bilinear interpolation between the
four base blocks around (x, y) (indices past the last block repeat the last
one).  Readings:

* For a 0/1 mask, ceil(Phi) is 1 exactly when some base block with a
  positive interpolation weight is 1: the resize keeps every block that any
  neighbour keeps, which is the conservative property Eq. 7 is meant to have
  (no active region of the base map is lost at the target resolution).
* The paper resizes the threshold map.  A ceiling of interpolated thresholds
  would send every value in (0, 1] to 1, so the reading taken is the operator
  that commutes with instantiation: T_target(u, v) is the minimum of T_base
  over the same positively weighted neighbours.  Then for every p,
  1[T_target <= p] is exactly the ceil-resize of 1[T_base <= p].
* The sample points are exact rationals; all arithmetic here is in integers
  (weights over the denominators n_q_target and n_k_target), so there is no
  rounding.  With a target smaller than the base the formula samples only
  some base rows and can drop blocks: the operation is meant for upscaling.
"""

import numpy as np


def _axis(n_base, n_target):
    """Per target index t: base index i0 = floor(t n_b / n_t), its weight
    numerator n_t - r and the next index's numerator r, over denominator n_t."""
    t = np.arange(n_target, dtype=np.int64)
    num = t * n_base
    i0 = num // n_target
    r = num % n_target
    i1 = np.minimum(i0 + 1, n_base - 1)
    return i0, i1, n_target - r, r


def bilinear_ceil(R, n_q_target, n_k_target):
    """Eq. 7 on a non-negative integer map R [H][n_q][n_k]: ceil of bilinear
    interpolation at the exact sample points, computed as integer fractions."""
    R = np.asarray(R).astype(np.int64)
    H, nq, nk = R.shape
    i0, i1, wi0, wi1 = _axis(nq, n_q_target)
    j0, j1, wj0, wj1 = _axis(nk, n_k_target)
    num = (wi0[:, None] * wj0[None, :] * R[:, i0][:, :, j0]
           + wi0[:, None] * wj1[None, :] * R[:, i0][:, :, j1]
           + wi1[:, None] * wj0[None, :] * R[:, i1][:, :, j0]
           + wi1[:, None] * wj1[None, :] * R[:, i1][:, :, j1])
    den = np.int64(n_q_target) * np.int64(n_k_target)
    return (num + den - 1) // den


def resize_mask(M, n_q_target, n_k_target):
    """Eq. 7 on a bool block mask [H][n_q][n_k]; result bool [H][n_q_t][n_k_t]."""
    return bilinear_ceil(np.asarray(M, dtype=bool), n_q_target, n_k_target) > 0


def resize_threshold_map(T, n_q_target, n_k_target):
    """Minimum of T over the positively weighted bilinear neighbours (float32).

    NaN entries are skipped (numpy fmin); a cell whose neighbours are all NaN
    stays NaN.
    """
    T = np.asarray(T, dtype=np.float32)
    H, nq, nk = T.shape
    i0, i1, _, wi1 = _axis(nq, n_q_target)
    j0, j1, _, wj1 = _axis(nk, n_k_target)
    out = T[:, i0][:, :, j0]
    use_i1 = (wi1 > 0)[:, None]
    use_j1 = (wj1 > 0)[None, :]
    out = np.where(use_j1, np.fmin(out, T[:, i0][:, :, j1]), out)
    out = np.where(use_i1, np.fmin(out, T[:, i1][:, :, j0]), out)
    out = np.where(use_i1 & use_j1, np.fmin(out, T[:, i1][:, :, j1]), out)
    return out.astype(np.float32)
