"""Pins for the Hellinger fidelity reference (oracle/fidelity.py), CPU only.

Tied to facts other than the code itself: scipy's Euclidean distance (Eq. 3
is the Euclidean distance of square-root vectors over sqrt 2), the closed form
H = sqrt(1 - sqrt(m)) for a distribution restricted to a subset of mass m and
renormalised (sum_j sqrt(p_j q_j) = sqrt(m) when q = p / m on the subset), the
metric's identity/symmetry/bounds, and a pure-Python brute force of the
profile on a tiny input.  Planted mistakes must each fail one pin.
"""

import math

import numpy as np
import pytest
from scipy.spatial import distance

from oracle import fidelity as ofid


def _dist(n, seed, sharp=1.0):
    x = np.random.default_rng(seed).normal(size=n) * sharp
    e = np.exp(x - x.max())
    return e / e.sum()


def _tiny_problem(seed=3):
    rng = np.random.default_rng(seed)
    B, H, N, d, blk = 1, 2, 24, 4, 4
    q = rng.normal(size=(B, H, N, d))
    k = rng.normal(size=(B, H, N, d))
    n = N // blk
    T = rng.random((H, n, n)).astype(np.float32)
    T[:, np.arange(n), np.arange(n)] = 0.0
    T[0, 2, 4] = np.float32(0.5)            # exactly equal to a candidate: included
    rows = np.array([[1, 9, 22], [0, 13, 17]])
    p = np.array([0.0, 0.25, 0.5, 1.0], dtype=np.float32)
    return q, k, rows, T, p, blk, 0.7


def _brute_profile(q, k, rows, T, p, blk, scale):
    B, H, N, _ = q.shape
    R, K = rows.shape[1], len(p)
    Hd = [[[[0.0] * K for _ in range(R)] for _ in range(H)] for _ in range(B)]
    for b in range(B):
        for h in range(H):
            for i in range(R):
                r = int(rows[h, i])
                s = [scale * sum(float(q[b, h, r, c]) * float(k[b, h, j, c]) for c in range(q.shape[3]))
                     for j in range(N)]
                z = sum(math.exp(x) for x in s)
                P = [math.exp(x) / z for x in s]
                for c in range(K):
                    allowed = [float(T[h, r // blk, j // blk]) <= float(p[c]) for j in range(N)]
                    zs = sum(math.exp(x) for x, a in zip(s, allowed) if a)
                    Q = [math.exp(x) / zs if a else 0.0 for x, a in zip(s, allowed)]
                    Hd[b][h][i][c] = math.sqrt(sum((math.sqrt(a) - math.sqrt(bq)) ** 2
                                                   for a, bq in zip(P, Q)) / 2.0)
    return np.array(Hd)


def pin_scipy_euclidean(hel, prof):
    for seed in range(5):
        P, Q = _dist(50, seed), _dist(50, seed + 100)
        ref = distance.euclidean(np.sqrt(P), np.sqrt(Q)) / math.sqrt(2.0)
        if abs(hel(P, Q) - ref) > 1e-14:
            return False
    return True


def pin_restriction_closed_form(hel, prof):
    rng = np.random.default_rng(7)
    for seed in range(6):
        P = _dist(64, seed, sharp=2.0)
        keep = rng.random(64) < 0.4
        keep[0] = True
        m = P[keep].sum()
        Q = np.where(keep, P / m, 0.0)
        if abs(hel(P, Q) - math.sqrt(1.0 - math.sqrt(m))) > 1e-12:
            return False
    return True


def pin_metric_facts(hel, prof):
    P, Q = _dist(30, 1), _dist(30, 2)
    A = np.zeros(30); A[:10] = 0.1
    Bv = np.zeros(30); Bv[10:20] = 0.1
    return (abs(hel(P, P)) < 1e-15 and abs(hel(P, Q) - hel(Q, P)) < 1e-15
            and 0.0 <= hel(P, Q) <= 1.0 and abs(hel(A, Bv) - 1.0) < 1e-15)


def pin_profile_brute_force(hel, prof):
    q, k, rows, T, p, blk, scale = _tiny_problem()
    Hd, F = prof(q, k, rows, T, p, blk, scale)
    ref = _brute_profile(q, k, rows, T, p, blk, scale)
    return np.allclose(Hd, ref, atol=1e-12) and np.allclose(F, 1.0 - ref.mean(axis=2), atol=1e-12)


def pin_profile_extremes_and_monotone(hel, prof):
    q, k, rows, T, p, blk, scale = _tiny_problem(5)
    Hd, F = prof(q, k, rows, T, p, blk, scale)
    full = p == 1.0
    return (np.allclose(Hd[..., full], 0.0, atol=1e-12) and np.allclose(F[..., full], 1.0)
            and np.all(np.diff(F, axis=-1) >= -1e-12))


PINS = [pin_scipy_euclidean, pin_restriction_closed_form, pin_metric_facts,
        pin_profile_brute_force, pin_profile_extremes_and_monotone]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_fidelity_reference_pins(pin):
    assert pin(ofid.hellinger, ofid.profile)


def test_fidelity_score_is_one_minus_distance():
    P, Q = _dist(20, 4), _dist(20, 5)
    assert ofid.fidelity_score(P, Q) == 1.0 - ofid.hellinger(P, Q)


def test_empty_mask_row_has_distance_one():
    q, k, rows, T, p, blk, scale = _tiny_problem()
    T = T.copy()
    T[0, rows[0, 0] // blk, :] = 2.0      # nothing reaches this row below p = 2
    Hd, _ = ofid.profile(q, k, rows, T, p, blk, scale)
    assert np.all(Hd[0, 0, 0, :] == 1.0)


# -------------------------------------------------------- planted mistakes ---

def _hel_no_root2(P, Q):
    return ofid.hellinger(P, Q) * math.sqrt(2.0)


def _hel_squared(P, Q):
    return ofid.hellinger(P, Q) ** 2


def _prof_unnormalised(q, k, rows, T, p, blk, scale):
    orig = ofid._softmax_over

    def unnorm(s, allowed=None):
        full = orig(s)
        if allowed is None:
            return full
        return np.where(allowed, full, 0.0) if allowed.any() else None
    ofid._softmax_over = unnorm
    try:
        return ofid.profile(q, k, rows, T, p, blk, scale)
    finally:
        ofid._softmax_over = orig


def _prof_strict(q, k, rows, T, p, blk, scale):
    return ofid.profile(q, k, rows, T, np.nextafter(np.asarray(p, np.float32), np.float32(-1)),
                        blk, scale)


def _prof_max(q, k, rows, T, p, blk, scale):
    Hd, _ = ofid.profile(q, k, rows, T, p, blk, scale)
    return Hd, 1.0 - Hd.max(axis=2)


def _prof_key_block_of_query(q, k, rows, T, p, blk, scale):
    # map row looked up by the key block index instead of the query block
    return ofid.profile(q, k, rows, np.swapaxes(T, 1, 2), p, blk, scale)


MUTANTS = {
    "missing_one_over_root2": (_hel_no_root2, ofid.profile),
    "squared_distance": (_hel_squared, ofid.profile),
    "unnormalised_sparse_row": (ofid.hellinger, _prof_unnormalised),
    "strict_threshold": (ofid.hellinger, _prof_strict),
    "max_instead_of_mean": (ofid.hellinger, _prof_max),
    "transposed_map": (ofid.hellinger, _prof_key_block_of_query),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name):
    hel, prof = MUTANTS[name]
    failed = []
    for pin in PINS:
        try:
            ok = pin(hel, prof)
        except Exception:
            ok = False
        if not ok:
            failed.append(pin.__name__)
    assert failed, "planted mistake %s passed every pin" % name


def test_block_log_mass_sums_to_dense_row_blocks():
    rng = np.random.default_rng(9)
    q_row, k = rng.normal(size=8), rng.normal(size=(70, 8))
    blm = ofid.block_log_mass(q_row, k, 16, 0.5)
    P = ofid.dense_row(q_row, k, 0.5)
    total = np.log(np.exp(blm - blm.max()).sum()) + blm.max()
    masses = np.exp(blm - total)
    ref = np.array([P[v * 16:(v + 1) * 16].sum() for v in range(5)])   # last block holds 6 keys
    assert np.allclose(masses, ref, atol=1e-15) and abs(masses.sum() - 1.0) < 1e-14
    s = 0.5 * (k @ q_row)
    assert abs(total - math.log(sum(math.exp(x) for x in s))) < 1e-12
