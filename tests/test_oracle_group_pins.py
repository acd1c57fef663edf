"""Pins of the oracle's group-level admission (Appendix B: mean aggregation
within prompt groups; groups as the admission unit). Each check rests on
something other than the oracle's own arithmetic: singleton groups reduce
to trajectory mode, exact rational means, numpy repeats and concatenations,
and a brute-force ordering of exactly computed means."""
from fractions import Fraction

import numpy as np
import pytest

import oracle
import poolgen

U = 2.0 ** -53


def _groups(rng, n, max_size=12, empty_frac=0.1):
    sizes = []
    left = n
    while left > 0:
        s = 0 if rng.random() < empty_frac else int(rng.integers(1, max_size + 1))
        s = min(s, left)
        sizes.append(s)
        left -= s
    sizes.append(0) if rng.random() < 0.5 else None
    return np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64), np.array(sizes, np.int64)


def test_group_singletons_reduce_to_trajectory_mode():
    pool = poolgen.make_pool("math")
    go = np.arange(pool.n + 1, dtype=np.int64)
    t = oracle.filter_step(pool)
    g = oracle.group_filter_step(pool, go, pool.occupancy, pool.capacity)
    assert np.array_equal(g["group_score"].view(np.uint64), t["score"].view(np.uint64))
    assert np.array_equal(g["keep"], t["keep"]) and np.array_equal(g["reject_group_ids"], t["reject_ids"])
    assert np.array_equal(g["offsets_out"], t["offsets_out"]) and np.array_equal(g["packed"][0], t["packed"][0])


def test_group_mean_of_equal_members_is_exact():
    for x in (0.0, 1.5, 3.0, 7.25, 1e6, 4097.0):
        for k in range(1, 17):
            s = np.full(k, x)
            assert oracle.group_score(s, np.array([0, k]))[0] == x


def test_group_mean_within_rounding_of_exact_mean():
    rng = np.random.default_rng(5)
    for _ in range(40):
        n = int(rng.integers(1, 300))
        s = rng.normal(50.0, 30.0, n) * rng.choice([1.0, 1e-3, 1e4])
        go, sizes = _groups(rng, n)
        gs = oracle.group_score(s, go)
        for g in range(len(sizes)):
            lo, hi = go[g], go[g + 1]
            if hi == lo:
                assert gs[g] == 0.0
                continue
            exact = sum((Fraction(float(v)) for v in s[lo:hi]), Fraction(0)) / (hi - lo)
            k = int(hi - lo)
            bound = k * U * float(np.max(np.abs(s[lo:hi]))) * 2 + U * abs(float(exact))
            assert abs(Fraction(float(gs[g])) - exact) <= Fraction(bound), (g, k)


def test_group_empty_groups_score_zero_and_keep_nothing():
    go = np.array([0, 0, 3, 3, 5, 5], np.int64)
    s = np.array([2.0, 4.0, 6.0, 1.0, 3.0])
    assert list(oracle.group_score(s, go)) == [0.0, 4.0, 0.0, 2.0, 0.0]
    keep = oracle.group_expand(go, np.array([1, 0, 1, 1, 0], np.uint8), 5)
    assert list(keep) == [0, 0, 0, 1, 1]


def test_group_expand_matches_repeat():
    rng = np.random.default_rng(6)
    for _ in range(50):
        n = int(rng.integers(0, 200))
        go, sizes = _groups(rng, n)
        gk = (rng.random(len(sizes)) < 0.5).astype(np.uint8)
        assert np.array_equal(oracle.group_expand(go, gk, n), np.repeat(gk, sizes))


def test_group_selection_is_top_b_by_mean_then_id():
    """Equal group sizes and integer member scores: every mean is an exact
    rational; the oracle must reject the b groups first in (mean desc, id asc)."""
    rng = np.random.default_rng(7)
    for _ in range(60):
        k = int(rng.integers(1, 9))
        ng = int(rng.integers(1, 40))
        s = rng.integers(0, 6, ng * k).astype(np.float64)      # many exact ties
        go = np.arange(0, ng * k + 1, k, dtype=np.int64)
        gs = oracle.group_score(s, go)
        means = [Fraction(int(s[g * k:(g + 1) * k].sum()), k) for g in range(ng)]
        order = sorted(range(ng), key=lambda g: (-means[g], g))
        b = int(rng.integers(0, ng + 1))
        keep, rej = oracle.select(gs, b)
        assert sorted(order[:b]) == list(rej)
        assert all(keep[g] == (g not in order[:b]) for g in range(ng))


def test_group_step_compacts_kept_groups_members():
    pool = poolgen.make_pool("math")
    go = pool.group_offsets
    ng = len(go) - 1
    occ, cap = ng, (pool.capacity + 7) // 8
    r = oracle.group_filter_step(pool, go, occ, cap)
    # the budget counts groups
    assert r["budget"] == min(occ - cap, int(np.rint(0.9 * occ)))
    assert len(r["reject_group_ids"]) == r["budget"]
    kept_groups = [g for g in range(ng) if r["group_keep"][g]]
    members = [i for g in kept_groups for i in range(go[g], go[g + 1])]
    assert list(r["kept_ids"]) == members
    ref = np.concatenate([pool.tags[pool.offsets[i]:pool.offsets[i + 1]] for i in members])
    assert np.array_equal(r["packed"][0], ref)
    # every rejected group's mean is at least every kept group's mean
    gs = r["group_score"]
    rej = set(int(g) for g in r["reject_group_ids"])
    if rej and len(rej) < ng:
        assert min(gs[g] for g in rej) >= max(gs[g] for g in range(ng) if g not in rej)


def test_group_offsets_preconditions():
    s = np.zeros(4)
    for go in ([1, 2, 4], [0, 2, 3], [0, 3, 2, 4]):
        with pytest.raises(oracle.OracleError) as e:
            oracle.group_score(s, np.array(go, np.int64))
        assert e.value.code == oracle.ERR_PRECONDITION
        with pytest.raises(oracle.OracleError):
            oracle.group_expand(np.array(go, np.int64), np.ones(len(go) - 1, np.uint8), 4)
