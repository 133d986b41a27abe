"""Pins of the CPU reference against facts it does not compute itself.

Each pin is a function taking an attention callable with the reference's
signature, so the same pins can be run against deliberately broken copies of
the reference (``test_planted_mistakes_are_caught``): every plausible slip
(bit order, block size mix-up, dropped scale, log base, transposed mask,
wrong normalisation set, swapped operands) must fail at least one pin.
"""

import importlib
import math
import os

import numpy as np
import pytest
import torch

import oracle
from workloads import pack_rows

oracle_attention_mod = importlib.import_module("oracle.attention")
oracle_bits = importlib.import_module("oracle.bits")
_ORIG_ATTENTION_BLOCK = oracle_attention_mod.attention_block

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------- inputs ---

def _rand(shape, seed, lo=-1.0, hi=1.0):
    return np.random.default_rng(seed).uniform(lo, hi, size=shape)


def _rand_mask(H, n_qb, n_kb, seed, p=0.4, diag=True, empty_rows=()):
    rng = np.random.default_rng(seed)
    m = rng.random((H, n_qb, n_kb)) < p
    if diag:
        for u in range(min(n_qb, n_kb)):
            m[:, u, u] = True
    for (h, u) in empty_rows:
        m[h, u, :] = False
    return m


def _torch_sdpa_f64(q, k, v, scale, token_mask=None):
    """Library routine: torch's scaled_dot_product_attention in float64 (CPU)."""
    tq, tk, tv = (torch.from_numpy(np.ascontiguousarray(x)) for x in (q, k, v))
    am = None if token_mask is None else torch.from_numpy(token_mask)
    return torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, attn_mask=am, scale=scale).numpy()


# ------------------------------------------------------------------- pins ---

def pin_dense_equals_library(attn):
    """All-ones mask == textbook dense attention (torch SDPA, float64)."""
    B, H, N, d, blk = 2, 2, 200, 16, 64
    q, k, v = (_rand((B, H, N, d), s, -2, 2) for s in (1, 2, 3))
    n = -(-N // blk)
    mask = pack_rows(np.ones((H, n, n), dtype=bool))
    scale = 0.37
    out, lse = attn(q, k, v, mask, blk, blk, scale)
    ref = _torch_sdpa_f64(q, k, v, scale)
    s = scale * np.einsum("bhid,bhjd->bhij", q, k)
    ref_lse = torch.logsumexp(torch.from_numpy(s), dim=-1).numpy()
    return np.allclose(out, ref, atol=1e-12) and np.allclose(lse, ref_lse, atol=1e-12)


def pin_diagonal_equals_blockwise(attn):
    """Diagonal-only mask == dense attention inside each block (ragged tail too)."""
    B, H, N, d, blk = 1, 2, 150, 8, 32
    q, k, v = (_rand((B, H, N, d), s, -2, 2) for s in (4, 5, 6))
    n = -(-N // blk)
    mask = pack_rows(np.broadcast_to(np.eye(n, dtype=bool), (H, n, n)))
    scale = 0.5
    out, _ = attn(q, k, v, mask, blk, blk, scale)
    ok = True
    for u in range(n):
        sl = slice(u * blk, min((u + 1) * blk, N))
        ref = _torch_sdpa_f64(q[:, :, sl], k[:, :, sl], v[:, :, sl], scale)
        ok &= np.allclose(out[:, :, sl], ref, atol=1e-12)
    return bool(ok)


def _brute(q, k, v, bm, blk_q, blk_k, scale):
    """Pure-Python loops over tokens; bm is the decoded bool block mask."""
    B, H, N, d = q.shape
    out = [[[[0.0] * d for _ in range(N)] for _ in range(H)] for _ in range(B)]
    lse = [[[-math.inf] * N for _ in range(H)] for _ in range(B)]
    for b in range(B):
        for h in range(H):
            for i in range(N):
                keys = [j for j in range(N) if bm[h][i // blk_q][j // blk_k]]
                if not keys:
                    continue
                s = {j: scale * sum(float(q[b, h, i, c]) * float(k[b, h, j, c]) for c in range(d))
                     for j in keys}
                mx = max(s.values())
                tot = sum(math.exp(s[j] - mx) for j in keys)
                lse[b][h][i] = mx + math.log(tot)
                for c in range(d):
                    out[b][h][i][c] = sum(math.exp(s[j] - lse[b][h][i]) * float(v[b, h, j, c])
                                          for j in keys)
    return np.array(out), np.array(lse)


def pin_brute_force(attn):
    """Pure-Python brute force, blk_q != blk_k, non-symmetric mask, empty rows."""
    B, H, N, d, bq, bk = 1, 2, 40, 3, 8, 16
    q, k, v = (_rand((B, H, N, d), s, -2, 2) for s in (7, 8, 9))
    n_qb, n_kb = -(-N // bq), -(-N // bk)
    bm = np.zeros((H, n_qb, n_kb), dtype=bool)
    rng = np.random.default_rng(10)
    bm[:] = rng.random((H, n_qb, n_kb)) < 0.5
    bm[0, 1, :] = False                 # an empty row
    bm[1, 2, :] = [True, False, False]  # only the first key block
    bm[1, 4, :] = [False, False, True]  # only the short last key block
    scale = 0.8
    out, lse = attn(q, k, v, pack_rows(bm), bq, bk, scale)
    rout, rlse = _brute(q, k, v, bm.tolist(), bq, bk, scale)
    fin = np.isfinite(rlse)
    return (np.allclose(out, rout, atol=1e-12) and np.array_equal(np.isfinite(lse), fin)
            and np.allclose(lse[fin], rlse[fin], atol=1e-12))


def pin_q_zero_closed_form(attn):
    """q = 0: uniform weights, lse = ln |K_i|, out = mean of the allowed v."""
    B, H, N, d, blk = 1, 1, 96, 4, 32
    q = np.zeros((B, H, N, d))
    k = _rand((B, H, N, d), 11, -3, 3)
    v = _rand((B, H, N, d), 12, -3, 3)
    bm = np.array([[[True, False, True], [False, True, False], [True, True, True]]])
    out, lse = attn(q, k, v, pack_rows(bm), blk, blk, 1.0)
    ok = True
    for u in range(3):
        keys = np.concatenate([np.arange(c * blk, (c + 1) * blk) for c in range(3) if bm[0, u, c]])
        sl = slice(u * blk, (u + 1) * blk)
        ok &= np.allclose(lse[0, 0, sl], np.log(len(keys)), atol=1e-13)
        ok &= np.allclose(out[0, 0, sl], v[0, 0, keys].mean(axis=0), atol=1e-13)
    return bool(ok)


def pin_key_shift(attn):
    """k_j += c for every key: lse_i += scale q_i.c, out unchanged."""
    B, H, N, d, blk = 1, 2, 64, 5, 16
    q, k, v = (_rand((B, H, N, d), s) for s in (13, 14, 15))
    c = _rand((d,), 16, -2, 2)
    mask = pack_rows(_rand_mask(H, 4, 4, 17))
    scale = 0.6
    o1, l1 = attn(q, k, v, mask, blk, blk, scale)
    o2, l2 = attn(q, k + c, v, mask, blk, blk, scale)
    return np.allclose(o1, o2, atol=1e-12) and np.allclose(l2 - l1, scale * (q @ c), atol=1e-12)


def pin_permutation(attn):
    """Joint K/V permutations among a query block's allowed keys change nothing
    for that block; moving an allowed key into a disallowed block does."""
    B, H, N, d, blk = 1, 1, 64, 4, 16
    q, k, v = (_rand((B, H, N, d), s, -2, 2) for s in (18, 19, 20))
    bm = np.array([[[True, False, True, False]] * 4])
    mask = pack_rows(bm)
    o1, l1 = attn(q, k, v, mask, blk, blk, 1.0)
    allowed = np.r_[0:16, 32:48]
    perm = np.arange(N)
    perm[allowed] = np.random.default_rng(21).permutation(allowed)   # within and across
    o2, l2 = attn(q, k[:, :, perm], v[:, :, perm], mask, blk, blk, 1.0)
    same = np.allclose(o1, o2, atol=1e-12) and np.allclose(l1, l2, atol=1e-12)
    swap = np.arange(N)
    swap[[3, 20]] = [20, 3]            # key 3 (allowed block 0) <-> key 20 (disallowed block 1)
    o3, _ = attn(q, k[:, :, swap], v[:, :, swap], mask, blk, blk, 1.0)
    return same and not np.allclose(o1, o3, atol=1e-6)


def pin_rows_sum_to_one(attn):
    """v = 1 gives out = 1 exactly where a row has any allowed key."""
    B, H, N, d, blk = 2, 2, 70, 3, 32
    q, k = (_rand((B, H, N, d), s, -4, 4) for s in (22, 23))
    v = np.ones((B, H, N, d))
    mask = pack_rows(_rand_mask(H, 3, 3, 24))
    out, _ = attn(q, k, v, mask, blk, blk, 1.3)
    return np.allclose(out, 1.0, atol=1e-13)


def pin_empty_row(attn):
    """A query block with no enabled key block: out = 0, lse = -inf."""
    B, H, N, d, blk = 1, 1, 48, 2, 16
    q, k, v = (_rand((B, H, N, d), s) for s in (25, 26, 27))
    bm = np.array([[[True, True, False], [False, False, False], [False, True, True]]])
    out, lse = attn(q, k, v, pack_rows(bm), blk, blk, 1.0)
    return (np.all(out[0, 0, 16:32] == 0.0) and np.all(np.isneginf(lse[0, 0, 16:32]))
            and np.all(np.isfinite(lse[0, 0, :16])) and np.all(np.isfinite(lse[0, 0, 32:])))


PINS = [pin_dense_equals_library, pin_diagonal_equals_blockwise, pin_brute_force,
        pin_q_zero_closed_form, pin_key_shift, pin_permutation, pin_rows_sum_to_one,
        pin_empty_row]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_reference_meets_pin(pin):
    assert pin(oracle.attention)


def test_sampled_matches_full():
    B, H, N, d, blk = 2, 3, 100, 8, 32
    q, k, v = (_rand((B, H, N, d), s) for s in (30, 31, 32))
    mask = pack_rows(_rand_mask(H, 4, 4, 33))
    out, lse = oracle.attention(q, k, v, mask, blk, blk, 0.4)
    items = [(1, 2, 3), (0, 0, 0), (1, 1, 2)]
    for (b, h, u), (o, l) in zip(items, oracle.attention_sampled(q, k, v, mask, blk, blk, 0.4, items)):
        sl = slice(u * blk, min((u + 1) * blk, N))
        assert np.array_equal(o, out[b, h, sl]) and np.array_equal(l, lse[b, h, sl])


# ---------------------------------------------------------- bit-level pins ---

def test_bf16_decode_known_patterns():
    # IEEE binary32 values whose low half is zero.
    cases = {0x3F80: 1.0, 0xC000: -2.0, 0x3F81: 1.0078125, 0x0000: 0.0, 0x8000: -0.0,
             0x7F80: np.inf, 0xFF80: -np.inf, 0x4049: 3.140625, 0x0001: 2.0 ** -133}
    got = oracle.bf16_bits_to_f64(np.array(list(cases), dtype=np.uint16))
    assert np.array_equal(got, np.array(list(cases.values())))
    assert np.isnan(oracle.bf16_bits_to_f64(np.array([0x7FC0], dtype=np.uint16)))[0]


def test_mask_decode_is_lsb_first():
    words = np.zeros((1, 3, 2), dtype=np.uint64)
    words[0, 0, 0] = 1                      # block 0
    words[0, 1, 0] = np.uint64(1) << np.uint64(63)   # block 63
    words[0, 2, 1] = 1 | (1 << 5)           # blocks 64 and 69
    bm = oracle.block_mask(words, 70)
    assert [list(np.flatnonzero(r)) for r in bm[0]] == [[0], [63], [64, 69]]
    assert oracle.active_blocks(words, 0, 2, 70) == [64, 69]
    assert oracle.mask_bit(words, 0, 1, 63) == 1 and oracle.mask_bit(words, 0, 1, 62) == 0


@pytest.mark.parametrize("n_kb", [1, 8, 63, 64, 65, 256, 591, 2048])
def test_crm_walk_matches_library_unpack(n_kb):
    rng = np.random.default_rng(n_kb)
    bm = rng.random((2, 5, n_kb)) < 0.3
    bm[0, 0] = False                        # empty row
    bm[1, 1] = True                         # full row
    if n_kb > 70:
        bm[1, 2, :64] = False               # a leading all-zero word
    packed = pack_rows(bm)
    dec = oracle.block_mask(packed, n_kb)
    assert np.array_equal(dec, bm)
    for h in range(2):
        for u in range(5):
            row = packed[h, u]
            ref = np.flatnonzero(np.unpackbits(row.view(np.uint8), bitorder="little"))
            ref = [int(x) for x in ref if x < n_kb]
            segs = row.view("<u4")          # the paper's uint32 segments, same bytes
            assert oracle.crm_walk(segs, n_kb) == ref
            assert oracle.active_blocks(packed, h, u, n_kb) == ref


def test_crm_segments_are_byte_identical_to_u64_words():
    rng = np.random.default_rng(5)
    words = rng.integers(0, 2 ** 63, size=(1, 3, 4), dtype=np.int64).astype(np.uint64)
    for u in range(3):
        segs = words[0, u].view("<u4")
        for w in range(4):
            assert int(words[0, u, w]) == int(segs[2 * w]) | (int(segs[2 * w + 1]) << 32)


def test_golden_crm_layout_figure():
    kv = {}
    with open(os.path.join(GOLDEN, "crm_layout.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                a, b = line.split()
                kv[a] = int(b)
    n_kb = kv["tokens"] // kv["block"]
    assert -(-n_kb // kv["bits_per_segment"]) == kv["segments_per_row"]
    assert oracle.n_words_u64(n_kb) * 2 == kv["segments_per_row"]
    full = pack_rows(np.ones((1, 1, n_kb), dtype=bool))
    assert full.shape[2] * 2 == kv["segments_per_row"]
    assert oracle.crm_walk(full[0, 0].view("<u4"), n_kb) == list(range(n_kb))


# --------------------------------------------------------- planted mistakes ---

def _msb_first_block_mask(mask_bits, n_kb):
    mb = np.asarray(mask_bits, dtype=np.uint64)
    v = np.arange(n_kb)
    return ((mb[:, :, v // 64] >> (63 - (v % 64)).astype(np.uint64)) & np.uint64(1)).astype(bool)


def _transposed_block_mask(mask_bits, n_kb):
    bm = oracle_bits.block_mask(mask_bits, n_kb)
    n_qb = bm.shape[1]
    if n_qb != n_kb:
        return bm
    return np.ascontiguousarray(np.swapaxes(bm, 1, 2))


def _wrong_norm_attention_block(q_rows, k, v, allowed_kb, blk_k, scale):
    # softmax over every key, then masked: normalised over the wrong set
    q_rows, k, v = (np.asarray(x, dtype=np.float64) for x in (q_rows, k, v))
    keys = np.asarray(allowed_kb)[np.arange(k.shape[0]) // blk_k]
    s = scale * (q_rows @ k.T)
    lse = np.log(np.exp(s).sum(axis=1))
    p = np.exp(s - lse[:, None]) * keys
    if not keys.any():
        return np.zeros((q_rows.shape[0], v.shape[1])), np.full(q_rows.shape[0], -np.inf)
    return p @ v, lse


def _swapped_qk_attention_block(q_rows, k, v, allowed_kb, blk_k, scale):
    # logits taken against the value vectors instead of the keys
    return _ORIG_ATTENTION_BLOCK(q_rows, v, v, allowed_kb, blk_k, scale)


MUTANTS = {
    "msb_first_bits": ("patch", "block_mask", _msb_first_block_mask),
    "transposed_mask": ("patch", "block_mask", _transposed_block_mask),
    "wrong_normalisation": ("patch", "attention_block", _wrong_norm_attention_block),
    "logits_against_v": ("patch", "attention_block", _swapped_qk_attention_block),
    "scale_dropped": ("wrap", lambda q, k, v, m, bq, bk, s: oracle.attention(q, k, v, m, bq, bk, 1.0)),
    "key_block_uses_blk_q": ("wrap", lambda q, k, v, m, bq, bk, s: oracle.attention(q, k, v, m, bq, bq, s)),
    "lse_in_log2": ("wrap", lambda q, k, v, m, bq, bk, s: (lambda r: (r[0], r[1] / np.log(2.0)))(
        oracle.attention(q, k, v, m, bq, bk, s))),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name, monkeypatch):
    spec = MUTANTS[name]
    if spec[0] == "patch":
        monkeypatch.setattr(oracle_attention_mod, spec[1], spec[2])
        attn = oracle_attention_mod.attention
    else:
        attn = spec[1]
    failed = []
    for pin in PINS:
        try:
            ok = pin(attn)
        except Exception:
            ok = False
        if not ok:
            failed.append(pin.__name__)
    assert failed, "planted mistake %s passed every pin" % name


def test_crm_walk_mutant_is_caught():
    def msb_walk(segs, n_kb=None):
        out = []
        for s, seg in enumerate(segs):
            for b in range(32):
                if (int(seg) >> (31 - b)) & 1:
                    out.append(32 * s + b)
        return [x for x in out if n_kb is None or x < n_kb]
    row = pack_rows(np.array([[[True, False, False, True, True] + [False] * 40]]))[0, 0]
    ref = [int(x) for x in np.flatnonzero(np.unpackbits(row.view(np.uint8), bitorder="little"))]
    assert oracle.crm_walk(row.view("<u4"), 45) == ref
    assert msb_walk(row.view("<u4"), 45) != ref
