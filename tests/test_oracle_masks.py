"""Pins for the mask-instantiation reference (oracle/masks.py), CPU only.

Each pin ties the reference to something other than itself: a hand-worked
example, numpy's own bit packing, the decoding already pinned in
test_oracle_pins.py, the empirical distribution function of the map, and
order/tie/NaN facts of the comparison M_p = 1[T <= p] (paper Sec. 4.1.2).
Planted mistakes at the end must each fail one of them.
"""

import numpy as np
import pytest

import oracle
from oracle import bits as obits
from oracle import masks as omasks
from workloads import threshold_maps, p_for_density


def _rand_T(H, n_qb, n_kb, seed):
    return np.random.default_rng(seed).random((H, n_qb, n_kb)).astype(np.float32)


def pin_hand_example(inst, pack):
    # one head, two query rows, three key blocks, p = 0.5
    T = np.array([[[0.1, 0.5, 0.9], [0.7, 0.2, 0.5]]], dtype=np.float32)
    p = np.array([[0.5]], dtype=np.float32)
    m = inst(T, p)
    ok = m.shape == (1, 1, 2, 3) and m[0, 0].tolist() == [[True, True, False], [False, True, True]]
    words = pack(m)
    return ok and words.shape == (1, 1, 2, 1) and words[0, 0, :, 0].tolist() == [0b011, 0b110]


def pin_pack_matches_numpy_packbits(inst, pack):
    rng = np.random.default_rng(5)
    for n_kb in (1, 7, 63, 64, 65, 130, 591):
        m = rng.random((2, 3, n_kb)) < 0.4
        W = obits.n_words_u64(n_kb)
        padded = np.zeros((2, 3, 64 * W), dtype=bool)
        padded[..., :n_kb] = m
        ref = np.packbits(padded, axis=-1, bitorder="little").view("<u8")
        if not np.array_equal(pack(m), ref):
            return False
    return True


def pin_pack_roundtrips_through_decoder(inst, pack):
    rng = np.random.default_rng(6)
    for n_kb in (1, 64, 65, 200):
        m = rng.random((3, 4, n_kb)) < 0.5
        if not np.array_equal(obits.block_mask(pack(m), n_kb), m):
            return False
    return True


def pin_density_is_empirical_cdf(inst, pack):
    T = _rand_T(3, 17, 29, 7)
    ps = np.array([[0.0, 0.25, 0.5], [0.9, 0.1, 1.0]], dtype=np.float32)
    m = inst(T, ps)
    for i in range(ps.shape[0]):
        for h in range(3):
            srt = np.sort(T[h].ravel())
            cdf = np.searchsorted(srt, ps[i, h], side="right")
            if m[i, h].sum() != cdf:
                return False
    return True


def pin_monotone_and_extremes(inst, pack):
    T = _rand_T(2, 9, 11, 8)
    lo = np.array([[T.min() - 1e-3] * 2], dtype=np.float32)
    hi = np.array([[T.max()] * 2], dtype=np.float32)
    a = np.array([[0.3, 0.6]], dtype=np.float32)
    b = np.array([[0.4, 0.6]], dtype=np.float32)
    ma, mb = inst(T, a), inst(T, b)
    return (not inst(T, lo).any()) and inst(T, hi).all() and np.all(ma <= mb)


def pin_ties_included_and_nan_off(inst, pack):
    T = np.array([[[0.25, 0.5, np.nan, 0.75]]], dtype=np.float32)
    m = inst(T, np.array([[0.5]], dtype=np.float32))
    m_nan = inst(T, np.array([[np.nan]], dtype=np.float32))
    return m[0, 0, 0].tolist() == [True, True, False, False] and not m_nan.any()


def pin_per_head_thresholds(inst, pack):
    # head h is compared with its own p[i, h] only
    T = np.zeros((3, 2, 2), dtype=np.float32) + np.array([0.1, 0.5, 0.9], dtype=np.float32)[:, None, None]
    m = inst(T, np.array([[0.2, 0.2, 0.95]], dtype=np.float32))
    return m[0, 0].all() and not m[0, 1].any() and m[0, 2].all()


PINS = [pin_hand_example, pin_pack_matches_numpy_packbits, pin_pack_roundtrips_through_decoder,
        pin_density_is_empirical_cdf, pin_monotone_and_extremes, pin_ties_included_and_nan_off,
        pin_per_head_thresholds]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_mask_reference_pins(pin):
    assert pin(omasks.instantiate, omasks.pack_crm)


def test_instantiate_packed_is_composition():
    T = _rand_T(2, 5, 70, 9)
    p = np.array([[0.3, 0.7], [0.5, 0.1]], dtype=np.float32)
    assert np.array_equal(oracle.instantiate_packed(T, p), omasks.pack_crm(omasks.instantiate(T, p)))


def test_synthetic_maps_and_density_helper():
    T = threshold_maps(4, 40, 40, 128, (5, 30, 52), seed=11)
    assert T.shape == (4, 40, 40) and T.dtype == np.float32
    assert np.all((T >= 0) & (T <= 1))
    assert np.all(T[:, np.arange(40), np.arange(40)] == 0.0)  # the diagonal enters first
    for rho in (0.05, 0.25, 0.6):
        p = p_for_density(T, rho)
        m = omasks.instantiate(T, p[None])
        dens = m[0].reshape(4, -1).mean(axis=1)
        assert np.all(dens >= rho - 1e-9) and np.all(dens <= rho + 0.05)


# -------------------------------------------------------- planted mistakes ---

def _strict(T, p):
    return np.asarray(T, np.float32)[None] < np.asarray(p, np.float32)[:, :, None, None]


def _msb_pack(mask):
    mask = np.asarray(mask, dtype=bool)
    n_kb = mask.shape[-1]
    W = obits.n_words_u64(n_kb)
    out = np.zeros(mask.shape[:-1] + (W,), dtype=np.uint64)
    for v in range(n_kb):
        out[..., v // 64] |= mask[..., v].astype(np.uint64) << np.uint64(63 - v % 64)
    return out


def _transposed(T, p):
    return omasks.instantiate(np.swapaxes(np.asarray(T), 1, 2), p)


def _shared_p(T, p):
    p = np.asarray(p, np.float32)
    return omasks.instantiate(T, np.repeat(p[:, :1], p.shape[1], axis=1))


def _ge(T, p):
    return np.asarray(T, np.float32)[None] >= np.asarray(p, np.float32)[:, :, None, None]


MUTANTS = {
    "strict_less": (_strict, omasks.pack_crm),
    "msb_first_pack": (omasks.instantiate, _msb_pack),
    "transposed_map": (_transposed, omasks.pack_crm),
    "first_head_threshold_for_all": (_shared_p, omasks.pack_crm),
    "inverted_comparison": (_ge, omasks.pack_crm),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name):
    inst, pack = MUTANTS[name]
    failed = [pin.__name__ for pin in PINS if not _safe(pin, inst, pack)]
    assert failed, "planted mistake %s passed every pin" % name


def _safe(pin, inst, pack):
    try:
        return bool(pin(inst, pack))
    except Exception:
        return False
