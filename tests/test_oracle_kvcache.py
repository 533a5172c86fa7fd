"""Pins of the KV-cache state reference (Section 4.4: logical validity mask,
Eq. 8; rollback and physical truncation, Eq. 9)."""

import numpy as np
import pytest

import oracle
from oracle import kvcache


def _cache(rng, B, Hkv, L_cap, D):
    k = rng.integers(0, 1 << 15, (B, Hkv, L_cap, D)).astype(np.uint16)
    v = rng.integers(0, 1 << 15, (B, Hkv, L_cap, D)).astype(np.uint16)
    return k, v


def _bf16(rng, shape):
    x = rng.normal(0, 1, shape).astype(np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


def test_append_writes_rows_at_the_cursor_and_nothing_else():
    rng = np.random.default_rng(0)
    B, Hkv, L_cap, D, gmax = 4, 2, 40, 8, 3
    k, v = _cache(rng, B, Hkv, L_cap, D)
    mask = (rng.random((B, L_cap)) < 0.7).astype(np.uint8)
    kv_len = np.array([5, 0, 37, 12], np.int32)
    gamma = np.array([3, 0, 3, 1], np.int32)
    kn, vn = _cache(rng, B, gmax + 1, Hkv, D)
    k2, v2, m2, l2, st = kvcache.append(k, v, mask, kv_len, kn, vn, gamma)
    assert st == kvcache.ST_KVLEN  # sequence 2: 37 + 4 > 40
    for b in range(B):
        if b == 2:
            assert (k2[b] == k[b]).all() and l2[b] == kv_len[b] and (m2[b] == mask[b]).all()
            continue
        n = gamma[b] + 1
        c = kv_len[b]
        assert l2[b] == c + n
        for i in range(n):
            assert (k2[b, :, c + i] == kn[b, i]).all() and (v2[b, :, c + i] == vn[b, i]).all()
        assert (m2[b, c:c + n] == 1).all()
        other = np.ones(L_cap, bool)
        other[c:c + n] = False
        assert (k2[b][:, other] == k[b][:, other]).all() and (m2[b, other] == mask[b, other]).all()


def test_append_at_a_shared_length_keeps_holes():
    rng = np.random.default_rng(1)
    B, Hkv, L_cap, D = 3, 1, 30, 4
    k, v = _cache(rng, B, Hkv, L_cap, D)
    mask = np.zeros((B, L_cap), np.uint8)
    kv_len = np.array([10, 7, 9], np.int32)
    for b in range(B):
        mask[b, : kv_len[b]] = 1
    kn, vn = _cache(rng, B, 3, Hkv, D)
    k2, v2, m2, l2, st = kvcache.append(k, v, mask, kv_len, kn, vn, np.array([2, 2, 2]), phys_len=10)
    assert st == 0 and list(l2) == [13, 13, 13]
    assert (m2[1, 7:10] == 0).all() and (m2[2, 9:10] == 0).all() and (m2[:, 10:13] == 1).all()


@pytest.mark.parametrize("seed", [2, 3])
def test_attention_over_holes_equals_attention_over_the_compacted_cache(seed):
    """Eq. 8: masked entries are ignored whatever they hold, so the attention
    of a holed cache equals that of its compaction."""
    rng = np.random.default_rng(seed)
    B, G1, Hq, Hkv, D, L_cap = 3, 3, 4, 2, 16, 64
    kv_len = np.array([40, 64, 20], np.int32)
    gamma = np.array([2, 1, 0], np.int32)
    k, v = _bf16(rng, (B, Hkv, L_cap, D)), _bf16(rng, (B, Hkv, L_cap, D))
    mask = (rng.random((B, L_cap)) < 0.6).astype(np.uint8)
    for b in range(B):  # this step's rows are valid
        mask[b, kv_len[b] - gamma[b] - 1: kv_len[b]] = 1
    q = _bf16(rng, (B, G1, Hq, D))
    scale = 1 / np.sqrt(D)
    a, st = oracle.verify_attention(q, k, v, kv_len, gamma, scale, mask)
    kc, vc, mc, lc, stc = kvcache.compact(k, v, mask, kv_len)
    assert st == stc == 0
    assert list(lc) == [int(mask[b, : kv_len[b]].sum()) for b in range(B)]
    ac, _ = oracle.verify_attention(q, kc, vc, lc, gamma, scale, mc)
    np.testing.assert_allclose(a, ac, rtol=1e-12, atol=1e-12)


def test_paper_layout_cycle_tracks_every_sequence():
    """Shared physical length L (the paper's layout): append at L, roll back
    each sequence to its accepted prefix (mask holes), cut the common tail
    (Eq. 9); the valid rows of every sequence are always its own tokens in
    order, and compaction makes them contiguous."""
    rng = np.random.default_rng(4)
    B, Hkv, L_cap, D, g = 5, 1, 200, 2, 4
    k = np.zeros((B, Hkv, L_cap, D), np.uint16)
    v = np.zeros_like(k)
    mask = np.zeros((B, L_cap), np.uint8)
    L = 6
    mask[:, :L] = 1
    seqs = [[1000 * b + i for i in range(L)] for b in range(B)]
    for b in range(B):
        k[b, 0, :L, 0] = seqs[b]
    kv_len = np.full(B, L, np.int32)
    next_tok = [L] * B
    for step in range(12):
        toks = np.zeros((B, g + 1, Hkv, D), np.uint16)
        for b in range(B):
            for i in range(g + 1):
                toks[b, i, 0, 0] = 1000 * b + next_tok[b] + i
        k, v, mask, kv_len, st = kvcache.append(k, v, mask, kv_len, toks, toks, np.full(B, g), phys_len=L)
        assert st == 0 and (kv_len == L + g + 1).all()
        keep = rng.integers(1, g + 2, B)  # accepted prefix incl. the pending row: 1 .. g + 1
        new_len = L + keep
        kv_r, mask, phys, st = oracle.rollback(kv_len, mask, new_len, cap=L_cap)
        rb = (L + g + 1) - new_len
        assert st == 0 and phys == kvcache.physical_truncation(L + g + 1, rb)[0]
        for b in range(B):
            seqs[b] += [1000 * b + next_tok[b] + i for i in range(keep[b])]
            next_tok[b] += keep[b]
        kv_len = np.full(B, phys, np.int32)  # every sequence's physical length is the shared one
        L = phys
        for b in range(B):
            assert list(k[b, 0, : L, 0][mask[b, :L] == 1]) == seqs[b]
    kc, vc, mc, lc, st = kvcache.compact(k, v, mask, kv_len)
    for b in range(B):
        assert lc[b] == len(seqs[b]) and list(kc[b, 0, : lc[b], 0]) == seqs[b] and (mc[b, : lc[b]] == 1).all()


def test_physical_truncation_eq9():
    assert kvcache.physical_truncation(50, [3, 1, 4]) == (49, 1)
    assert kvcache.physical_truncation(50, [0, 2]) == (50, 0)
