"""Pins of the oracle's Prefix Forgetting Score (Eq. (5); scoring caps and
the 32-token minimum from Appendix B): exact constant differences, the cap,
the minimum, masked tokens, symmetry, and an exact rational mean."""
from fractions import Fraction

import numpy as np
import pytest

import oracle

U = 2.0 ** -53


def test_prefix_constant_difference_is_exact():
    for delta in (0.0, 0.5, 0.25, 1.75, 3.0):
        for m in (32, 33, 100, 1024):
            a = np.full(m, -2.0, np.float32)
            b = (a - np.float32(delta)).astype(np.float32)
            s = oracle.prefix_score(a, b, np.array([0, m]), cap=1024, min_tokens=32)
            assert s[0] == delta


def test_prefix_minimum_tokens_and_empty():
    a = np.zeros(40, np.float32)
    b = np.ones(40, np.float32)
    s = oracle.prefix_score(a, b, np.array([0, 31, 31, 40]), cap=1024, min_tokens=32)
    assert np.isnan(s[0]) and np.isnan(s[1]) and np.isnan(s[2])
    s = oracle.prefix_score(a, b, np.array([0, 32, 40]), cap=1024, min_tokens=32)
    assert s[0] == 1.0 and np.isnan(s[1])
    s = oracle.prefix_score(a, b, np.array([0, 9, 40]), cap=1024, min_tokens=0)
    assert s[0] == 1.0 and s[1] == 1.0


def test_prefix_cap_counts_only_the_first_eligible_tokens():
    rng = np.random.default_rng(51)
    m, cap = 3000, 1024
    a = rng.normal(-1, 0.5, m).astype(np.float32)
    b = rng.normal(-1, 0.5, m).astype(np.float32)
    s1 = oracle.prefix_score(a, b, np.array([0, m]), cap=cap)
    a2, b2 = a.copy(), b.copy()
    a2[cap:] = 1e6                      # beyond the cap: must not matter
    s2 = oracle.prefix_score(a2, b2, np.array([0, m]), cap=cap)
    assert s1[0] == s2[0]
    exact = sum((abs(Fraction(float(x)) - Fraction(float(y))) for x, y in zip(a[:cap], b[:cap])), Fraction(0)) / cap
    assert abs(Fraction(float(s1[0])) - exact) <= Fraction(cap * U) * exact


def test_prefix_masked_tokens_are_skipped():
    rng = np.random.default_rng(52)
    m = 500
    a = rng.normal(-1, 0.5, m).astype(np.float32)
    b = rng.normal(-1, 0.5, m).astype(np.float32)
    tags = rng.integers(0, 50, m).astype(np.int32)
    mask = rng.random(m) < 0.3
    tags[mask] = -1
    a_m = a.copy()
    a_m[mask] = 1e6                     # masked tokens: must not matter
    s1 = oracle.prefix_score(a, b, np.array([0, m]), tags=tags, cap=200)
    s2 = oracle.prefix_score(a_m, b, np.array([0, m]), tags=tags, cap=200)
    assert s1[0] == s2[0]
    keep = np.flatnonzero(~mask)[:200]
    ref = oracle.prefix_score(a[keep], b[keep], np.array([0, len(keep)]), cap=200)
    assert s1[0] == ref[0]


def test_prefix_symmetric_and_within_rounding_of_exact():
    rng = np.random.default_rng(53)
    for _ in range(12):
        n = int(rng.integers(1, 12))
        lens = rng.integers(0, 2500, n)
        po = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        a = rng.normal(-3, 2, po[-1]).astype(np.float32)
        b = (a + rng.normal(0, 0.1, po[-1])).astype(np.float32)
        cap = int(rng.choice([1024, 2048]))
        s = oracle.prefix_score(a, b, po, cap=cap)
        s_sw = oracle.prefix_score(b, a, po, cap=cap)
        assert np.array_equal(s.view(np.uint64), s_sw.view(np.uint64))
        for i in range(n):
            m = min(int(lens[i]), cap)
            if m < 32:
                assert np.isnan(s[i])
                continue
            lo = po[i]
            exact = sum((abs(Fraction(float(x)) - Fraction(float(y)))
                         for x, y in zip(a[lo:lo + m], b[lo:lo + m])), Fraction(0)) / m
            assert abs(Fraction(float(s[i])) - exact) <= Fraction((m + 2) * U) * exact


def test_prefix_offsets_preconditions():
    a = np.zeros(10, np.float32)
    for po in ([1, 10], [0, 9], [0, 6, 5, 10]):
        with pytest.raises(oracle.OracleError):
            oracle.prefix_score(a, a, np.array(po, np.int64))
