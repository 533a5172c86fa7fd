"""Pins for the rollback reference (CPU only): idempotence, Eq. 9's common
physical length, the exact span of cleared validity bits (Section 4.4), and
the data-error rules."""

import numpy as np
import pytest

from oracle.rollback import rollback


@pytest.mark.parametrize("seed", range(5))
def test_idempotent(seed):
    rng = np.random.default_rng(seed)
    B, cap = 9, 64
    kv = rng.integers(10, cap + 1, B)
    mask = (rng.random((B, cap)) < 0.9).astype(np.uint8)
    new = kv - rng.integers(0, 8, B)
    kv1, m1, p1, s1 = rollback(kv, mask, new)
    kv2, m2, p2, s2 = rollback(kv1, m1, new)
    np.testing.assert_array_equal(kv1, kv2)
    np.testing.assert_array_equal(m1, m2)
    assert p1 == p2 and s1 == s2 == 0


@pytest.mark.parametrize("seed", range(5))
def test_eq9_common_physical_length(seed):
    """All sequences at L; rolling back r_b leaves L - min_b r_b (Eq. 9)."""
    rng = np.random.default_rng(seed)
    B, L = 7, 50
    r = rng.integers(0, 9, B)
    kv, _, phys, st = rollback(np.full(B, L), None, L - r)
    assert st == 0
    assert phys == L - r.min()
    np.testing.assert_array_equal(kv, L - r)


def test_clears_exactly_the_rolled_back_entries():
    cap = 20
    mask = np.ones((2, cap), np.uint8)
    mask[0, 3] = 0
    kv, m, phys, st = rollback(np.array([15, 12]), mask, np.array([10, 12]))
    want = np.ones((2, cap), np.uint8)
    want[0, 3] = 0
    want[0, 10:15] = 0
    np.testing.assert_array_equal(m, want)
    assert list(kv) == [10, 12] and phys == 12 and st == 0


def test_grow_is_noop_and_flagged():
    mask = np.ones((1, 8), np.uint8)
    kv, m, phys, st = rollback(np.array([5]), mask, np.array([7]))
    assert kv[0] == 5 and (m == 1).all() and st == 16


def test_negative_or_out_of_range_lengths_are_errors():
    mask = np.ones((2, 8), np.uint8)
    kv, m, phys, st = rollback(np.array([5, 9]), mask, np.array([-1, 3]))
    assert list(kv) == [5, 9] and (m == 1).all() and st == 2
