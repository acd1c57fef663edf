"""Pins of the oracle's Stale-k admission (Eq. (1) lag <= k) and admission
diagnostics (kept/rejected staleness histograms): closed forms for
single-version trajectories, exact rational lags from the tags, Lemma 1's
identity, and numpy's binning and sums."""
from fractions import Fraction

import numpy as np

import oracle
import poolgen


def _pool_arrays(lens, rng, V=100, mask_frac=0.0):
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    comp = rng.integers(V - 8, V + 1, len(lens)).astype(np.int32)
    tags = np.empty(int(off[-1]), np.int32)
    for i in range(len(lens)):
        tags[off[i]:off[i + 1]] = rng.integers(max(comp[i] - 12, 0), comp[i] + 1, lens[i])
    if mask_frac:
        tags[rng.random(len(tags)) < mask_frac] = -1
    return tags, off, comp


def test_stale_k_single_version_closed_form():
    V = 50
    for v in range(30, 51):
        tags = np.full(10, v, np.int32)
        for k in (0, 3, 8, 20):
            keep, lag = oracle.stale_k(tags, np.array([0, 10]), np.array([v], np.int32), V, k)
            assert lag[0] == V - v and keep[0] == (V - v <= k)


def test_stale_k_exact_lag_and_boundary():
    rng = np.random.default_rng(71)
    for _ in range(30):
        lens = rng.integers(0, 200, 40)
        tags, off, comp = _pool_arrays(lens, rng, mask_frac=0.2)
        V = 100
        k = int(rng.integers(0, 16))
        keep, lag = oracle.stale_k(tags, off, comp, V, k)
        for i in range(len(lens)):
            t = tags[off[i]:off[i + 1]]
            t = t[t != -1]
            if len(t) == 0:
                exact = Fraction(V - int(comp[i]))
            else:
                exact = Fraction(int((V - t.astype(np.int64)).sum()), len(t))
            assert keep[i] == (exact <= k), i
            assert lag[i] == float(exact) or abs(Fraction(lag[i]) - exact) <= Fraction(2.0 ** -52) * exact


def test_stale_k_lemma_identity():
    pool = poolgen.make_pool("multiturn")
    keep, lag = oracle.stale_k(pool.tags, pool.offsets, pool.completion, pool.V, 8)
    sc, S, T = oracle.score(pool.tags, pool.offsets, pool.completion, pool.V)
    num = S + (pool.V - pool.completion.astype(np.int64)) * T
    has = T > 0
    assert np.array_equal(keep[has], (num[has] <= 8 * T[has]).astype(np.uint8))
    assert np.array_equal(keep[~has], ((pool.V - pool.completion[~has]) <= 8).astype(np.uint8))


def test_stale_k_masked_tokens_do_not_count():
    tags = np.array([10, -1, -1, 10], np.int32)
    keep, lag = oracle.stale_k(tags, np.array([0, 4]), np.array([10], np.int32), 12, 2)
    assert lag[0] == 2.0 and keep[0] == 1
    keep, lag = oracle.stale_k(tags, np.array([0, 4]), np.array([10], np.int32), 12, 1)
    assert keep[0] == 0


def test_diagnostics_match_numpy_binning_and_sums():
    rng = np.random.default_rng(72)
    for _ in range(20):
        lens = rng.integers(0, 300, int(rng.integers(1, 80)))
        tags, off, comp = _pool_arrays(lens, rng, mask_frac=float(rng.choice([0.0, 0.3])))
        V = 100
        sc, S, T = oracle.score(tags, off, comp, V)
        keep = (rng.random(len(lens)) < 0.5).astype(np.uint8)
        nb = int(rng.integers(1, 12))
        edges = np.sort(rng.uniform(-1, 14, (3, nb + 1)), axis=1)
        hist, tot = oracle.diagnostics(tags, off, comp, V, sc, keep, edges)
        # independent metric values
        kw = (V - comp.astype(np.int64)).astype(np.float64)
        S2 = np.array([int((comp[i] - tags[off[i]:off[i + 1]][tags[off[i]:off[i + 1]] != -1].astype(np.int64)).sum())
                       for i in range(len(lens))])
        T2 = np.array([int((tags[off[i]:off[i + 1]] != -1).sum()) for i in range(len(lens))])
        kg = np.where(T2 > 0, S2 / np.maximum(T2, 1), 0.0)
        for q, x in enumerate((kw, kg, sc)):
            b = np.searchsorted(edges[q], x, side="right")          # 0 = below, nb+1 = at/above the top
            for cls in (0, 1):
                ref = np.bincount(b[keep == cls], minlength=nb + 2)
                assert np.array_equal(hist[q, cls], ref), (q, cls)
        for cls in (0, 1):
            sel = keep == cls
            assert list(tot[cls]) == [int(sel.sum()), int((V - comp[sel].astype(np.int64)).sum()),
                                      int(S2[sel].sum()), int(T2[sel].sum())]


def test_diagnostics_values_on_edges_go_right():
    """K_wait is an integer: with integer edges every value sits on an edge,
    and [e_b, e_b+1) puts it in the bin that starts there."""
    rng = np.random.default_rng(73)
    lens = rng.integers(1, 50, 200)
    tags, off, comp = _pool_arrays(lens, rng)
    V = 100
    sc, S, T = oracle.score(tags, off, comp, V)
    keep = np.ones(len(lens), np.uint8)
    edges = np.array([np.arange(0, 10, dtype=np.float64)] * 3)      # 9 bins [0,1), ..., [8,9)
    hist, tot = oracle.diagnostics(tags, off, comp, V, sc, keep, edges)
    kw = V - comp.astype(np.int64)
    ref = np.bincount(np.minimum(kw + 1, 10), minlength=11)          # value w lands in bin w + 1; >= 9 overflow
    assert np.array_equal(hist[0, 1], ref)
    assert hist[0, 0].sum() == 0
