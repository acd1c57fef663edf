"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these checks re-types the oracle's own arithmetic: each pins it to an
independent route (Eq. (1) computed directly in exact rationals against the
oracle's Lemma 1 route, closed forms the paper states, Python's own sort for
selection, numpy slicing for compaction, brute force on tiny pools).
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

import oracle
import poolgen

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "closed_forms.json")


def rel_close(x: float, exact: Fraction, tol=1e-12) -> bool:
    if exact == 0:
        return x == 0.0
    return abs(Fraction(x) - exact) <= abs(exact) * Fraction(tol)


# --------------------------------------------------------------------------
# Golden hand-derived cases (tests/golden/closed_forms.json)
# --------------------------------------------------------------------------
def test_golden_scores():
    g = json.load(open(GOLDEN))
    for case in g["score_cases"]:
        sc, S, T = oracle.score(np.array(case["tags"], np.int32), np.array(case["offsets"], np.int64),
                                np.array(case["completion"], np.int32), case["V"])
        assert S.tolist() == case["S"], case["name"]
        assert T.tolist() == case["T"], case["name"]
        for x, (num, den) in zip(sc, case["raw"]):
            assert rel_close(x, Fraction(num, den)), case["name"]


def test_golden_weights():
    """F of Eq. (9) isolated: a trajectory whose Generation Staleness is exactly
    1 (all tokens one version below c) scored with w_wait = 0 has M = F."""
    g = json.load(open(GOLDEN))
    for case in g["weight_cases"]:
        for gam, (num, den) in zip(case["gamma"], case["F"]):
            sc, _, _ = oracle.score(np.array([4, 4], np.int32), np.array([0, 2], np.int64),
                                    np.array([5], np.int32), 5,
                                    prefix=np.array([case["s"]]), window=np.array(case["window"], float),
                                    w_wait=0.0, gamma=gam, window_min=1)
            assert rel_close(sc[0], Fraction(num, den), 1e-15), (case["name"], gam)


def test_golden_budgets():
    g = json.load(open(GOLDEN))
    for case in g["budget_cases"]:
        b, _ = oracle.budget(case["N"], case["N_tar"], 0.0, case["beta"], 0.9)
        assert b == case["budget"], case["cite"]


# --------------------------------------------------------------------------
# Eq. (1) and Lemma 1
# --------------------------------------------------------------------------
def _random_valid_pool(rng, n, max_len=300, mask_frac=0.2, V=50):
    lens = rng.integers(0, max_len, size=n)
    return poolgen.make_custom_pool(lens, V=V, seed=int(rng.integers(1 << 30)),
                                    max_breaks=5, mask_frac=mask_frac)


def test_single_version_closed_form():
    """A trajectory generated under one version v: K_gen = c - v, S = T (c - v),
    and the Raw score equals j - v (Eq. (1), the sentence after it)."""
    rng = np.random.default_rng(1)
    for trial in range(50):
        n = int(rng.integers(1, 40))
        lens = rng.integers(1, 500, size=n)
        V = int(rng.integers(10, 10_000))
        c = V - rng.integers(0, 9, size=n)
        v = c - rng.integers(0, 9, size=n)
        v = np.maximum(v, 0)
        tags = np.repeat(v.astype(np.int32), lens)
        # sprinkle masked (non-generated) tokens; they must not matter
        m = rng.random(tags.size) < 0.3
        tags[m] = -1
        offsets = np.concatenate(([0], np.cumsum(lens))).astype(np.int64)
        sc, S, T = oracle.score(tags, offsets, c.astype(np.int32), V)
        T_ref = np.add.reduceat((~m).astype(np.int64), offsets[:-1])
        assert np.array_equal(T, T_ref)
        assert np.array_equal(S, T_ref * (c - v))
        for i in range(n):
            expect = Fraction(V - int(v[i])) if T_ref[i] > 0 else Fraction(V - int(c[i]))
            assert rel_close(sc[i], expect)


def test_raw_score_equals_eq1_lag_exactly():
    """Raw score (F = 1, w = 1) is Eq. (1)'s mean lag (1/T) sum_t (j - v_t),
    computed here directly in exact rationals from the tags alone -- a route
    that never forms K_gen or K_wait (Lemma 1)."""
    rng = np.random.default_rng(2)
    for trial in range(20):
        p = _random_valid_pool(rng, int(rng.integers(1, 60)), V=int(rng.integers(20, 100000)))
        sc, S, T = oracle.score(p.tags, p.offsets, p.completion, p.V)
        for i in range(p.n):
            seg = p.tags[p.offsets[i]:p.offsets[i + 1]]
            gen = seg[seg != -1].astype(np.int64)
            if gen.size == 0:
                exact = Fraction(p.V - int(p.completion[i]))   # reading: K_gen = 0
            else:
                exact = Fraction(int((p.V - gen).sum()), gen.size)
            assert rel_close(sc[i], exact), (trial, i)
            # integer identity from the proof of Lemma 1
            assert int(S[i]) + (p.V - int(p.completion[i])) * int(T[i]) == int((p.V - gen).sum())
            assert S[i] >= 0 and T[i] == gen.size


def test_components_nonnegative_on_paper_pools():
    """v_t <= c <= j implies both components are nonnegative (Lemma 1)."""
    for name in ("tiny", "math", "multiturn"):
        p = poolgen.make_pool(name)
        sc, S, T = oracle.score(p.tags, p.offsets, p.completion, p.V)
        assert (S >= 0).all() and (T >= 0).all()
        assert (sc >= p.V - p.completion).all()


def test_masked_tokens_do_not_change_scores():
    rng = np.random.default_rng(3)
    p = _random_valid_pool(rng, 30, mask_frac=0.0)
    base = oracle.score(p.tags, p.offsets, p.completion, p.V, p.prefix_score, p.window, gamma=4)
    # insert masked runs inside every trajectory
    tags, offs = [], [0]
    for i in range(p.n):
        seg = p.tags[p.offsets[i]:p.offsets[i + 1]]
        k = int(rng.integers(0, seg.size + 1))
        ins = np.full(int(rng.integers(0, 50)), -1, np.int32)
        tags.append(np.concatenate((seg[:k], ins, seg[k:])))
        offs.append(offs[-1] + tags[-1].size)
    t2 = np.concatenate(tags).astype(np.int32)
    o2 = np.array(offs, np.int64)
    alt = oracle.score(t2, o2, p.completion, p.V, p.prefix_score, p.window, gamma=4)
    for a, b in zip(base, alt):
        assert np.array_equal(a, b)


# --------------------------------------------------------------------------
# Eq. (7)-(9)
# --------------------------------------------------------------------------
def _F_via_gen_only(s, window, gamma, window_min=1):
    sc, _, _ = oracle.score(np.array([4], np.int32), np.array([0, 1], np.int64), np.array([5], np.int32), 5,
                            prefix=np.array([s], float), window=np.asarray(window, float),
                            w_wait=0.0, gamma=gamma, window_min=window_min)
    return sc[0]


def test_phi_matches_paper_form_in_exact_arithmetic():
    """F equals q^g / (q^g + (1-q)^g) with q = #{w <= s}/W (np.searchsorted,
    side='right' is that count), evaluated in Fractions in the paper's form."""
    rng = np.random.default_rng(4)
    for trial in range(200):
        W = int(rng.integers(1, 700))
        window = np.sort(rng.lognormal(np.log(0.02), 1.0, size=W))
        s = float(rng.lognormal(np.log(0.02), 1.2))
        if trial % 5 == 0:
            s = float(window[int(rng.integers(0, W))])   # exact hit: <= must count it
        gam = int(rng.integers(1, 5))
        q = Fraction(int(np.searchsorted(window, s, side="right")), W)
        exact = q ** gam / (q ** gam + (1 - q) ** gam)
        assert rel_close(_F_via_gen_only(s, window, gam), exact, 1e-15)


def test_phi_symmetry_and_monotonicity():
    window = np.arange(1, 513, dtype=float)
    for gam in (1, 2, 3, 4):
        Fs = [_F_via_gen_only(float(a) + 0.5, window, gam) for a in range(0, 513)]
        assert all(x <= y for x, y in zip(Fs, Fs[1:]))          # nondecreasing (Eq. (7))
        assert Fs[0] == 0.0 and Fs[-1] == 1.0                  # F maps into [0, 1]
        for a in range(0, 513):                                # phi(q) + phi(1-q) = 1
            assert abs(Fs[a] + Fs[512 - a] - 1.0) <= 2.0 ** -52
        assert Fs[256] == 0.5


def test_missing_prefix_or_short_window_gives_full_penalty():
    window = np.arange(1, 31, dtype=float)     # 30 < 32 observations
    assert _F_via_gen_only(10.0, window, 4, window_min=32) == 1.0
    assert _F_via_gen_only(float("nan"), np.arange(1, 600, dtype=float), 4, window_min=32) == 1.0


# Largest window W with W^gamma < 2^53 for each integer gamma (worked out by
# hand: 94906265^2 = 9007199136250225, 208063^3 = 9007091372906047 and
# 9741^4 = 9003558140700561 lie below 2^53 = 9007199254740992; the next W
# does not). Up to that size every a^gamma, (W - a)^gamma and their sum is an
# exact integer in binary64, so Eq. (9) is one correctly rounded division.
WINDOW_POWER_BOUNDS = {2: 94906265, 3: 208063, 4: 9741}


def _score_rc(W, gamma, prefix=None):
    """Return code of oracle.score on a one-trajectory pool with a window of
    W equal entries (sorted); the zero-filled window costs no memory until
    read."""
    return oracle.score(np.array([4], np.int32), np.array([0, 1], np.int64), np.array([5], np.int32), 5,
                        prefix=prefix, window=np.zeros(W), w_wait=0.0, gamma=gamma, window_min=1, check=False)


def test_window_power_bound_per_gamma():
    """The exact form of Eq. (9) needs W^gamma < 2^53: the oracle accepts the
    largest such W for every gamma and rejects the next one, without the
    power overflowing on the way."""
    for gam, W in WINDOW_POWER_BOUNDS.items():
        ok = _score_rc(W, gam)
        assert not isinstance(ok, int), (gam, W, ok)
        assert _score_rc(W + 1, gam) == oracle.ERR_ARG, (gam, W + 1)
    # gamma = 4 past the point where W^4 no longer fits in 63 bits (55109^4 >
    # 2^63): a power computed without a check would wrap and pass the test
    for W in (55108, 55109, 55110, 65536, 100000):
        assert _score_rc(W, 4) == oracle.ERR_ARG, W
    assert not isinstance(_score_rc(4096, 4), int)


def test_phi_exact_at_the_largest_window():
    """At W = 9741, gamma = 4 (the largest window for gamma 4), F is the
    correctly rounded q^4 / (q^4 + (1-q)^4) of Eq. (9) and lies in [0, 1]
    (Eq. (7)); s runs over ranks 0, 1, W/2, W-1 and W."""
    W = WINDOW_POWER_BOUNDS[4]
    window = np.arange(1, W + 1, dtype=float)
    for a in (0, 1, W // 2, W // 2 + 1, W - 1, W):
        F = _F_via_gen_only(float(a) + 0.5, window, 4)
        q = Fraction(a, W)
        exact = q ** 4 / (q ** 4 + (1 - q) ** 4)
        assert F == float(exact), (a, F, float(exact))
        assert 0.0 <= F <= 1.0


def test_effective_and_gen_only_variants():
    """Eq. (7): K_eff = K_wait + F K_gen; generation-only variant: w_wait = 0."""
    rng = np.random.default_rng(5)
    p = _random_valid_pool(rng, 80)
    W = p.window.size
    eff, S, T = oracle.score(p.tags, p.offsets, p.completion, p.V, p.prefix_score, p.window, gamma=4)
    gen, _, _ = oracle.score(p.tags, p.offsets, p.completion, p.V, p.prefix_score, p.window, w_wait=0.0, gamma=4)
    for i in range(p.n):
        kg = Fraction(int(S[i]), int(T[i])) if T[i] else Fraction(0)
        s = p.prefix_score[i]
        if math.isnan(s):
            F = Fraction(1)
        else:
            q = Fraction(int(np.searchsorted(p.window, s, side="right")), W)
            F = q ** 4 / (q ** 4 + (1 - q) ** 4)
        assert rel_close(eff[i], (p.V - int(p.completion[i])) + F * kg)
        assert rel_close(gen[i], F * kg)


# --------------------------------------------------------------------------
# Eq. (3)-(4) budget
# --------------------------------------------------------------------------
def test_budget_zero_at_or_below_target():
    rng = np.random.default_rng(6)
    for _ in range(2000):
        Ntar = int(rng.integers(0, 10 ** 6))
        N = int(rng.integers(0, Ntar + 1))
        b, rh = oracle.budget(N, Ntar, float(rng.random()), float(rng.uniform(0.5, 0.99)), 0.9)
        assert b == 0


def test_budget_beta0_is_surplus_until_cap():
    for N in range(1, 3000, 7):
        for Ntar in range(0, N + 1, max(1, N // 13)):
            b, rh = oracle.budget(N, Ntar, 0.0, 0.0, 0.9)
            surplus = N - Ntar
            if Fraction(surplus, N) <= Fraction(9, 10):
                assert b == surplus, (N, Ntar)
            else:
                assert b == round(Fraction(9, 10) * N) or b == math.floor(Fraction(9, 10) * N + Fraction(1, 2)), (N, Ntar)
                assert b <= surplus


def test_budget_ema_closed_form():
    """Constant r from r_hat_0 = 0: r_hat_s = r (1 - beta^s) (Eq. (4))."""
    for beta in (0.5, 0.9, 0.99):
        for N, Ntar in ((300, 100), (4096, 1365), (1000, 999)):
            r = Fraction(N - Ntar, N)
            rh = 0.0
            for s in range(1, 60):
                b, rh = oracle.budget(N, Ntar, rh, beta, 0.9)
                exact = r * (1 - Fraction(beta) ** s)
                assert abs(Fraction(rh) - exact) <= Fraction(1, 10 ** 12)
                assert 0 <= b <= N - Ntar


def test_budget_falling_backlog_keeps_target_buffer():
    """With smoothing (beta > 0) r_hat lags a falling backlog. The budget never
    removes more than the surplus N - N^tar (the target is the buffer of ready
    trajectories kept for training, Sec. 3.1), and is 0 once N <= N^tar even
    though r_hat is still positive."""
    rh = 0.0
    for _ in range(40):                      # long backlog: r = 0.75
        b, rh = oracle.budget(4000, 1000, rh, 0.9, 0.9)
    assert rh > 0.7
    b, rh2 = oracle.budget(1100, 1000, rh, 0.9, 0.9)
    assert b == 100 and rh2 > 0.6
    b, rh3 = oracle.budget(1000, 1000, rh2, 0.9, 0.9)
    assert b == 0 and rh3 > 0.5
    b, _ = oracle.budget(900, 1000, rh3, 0.9, 0.9)
    assert b == 0


# --------------------------------------------------------------------------
# Selection: exact top-b, ties to the lower id
# --------------------------------------------------------------------------
def _brute(score, b):
    order = sorted(range(len(score)), key=lambda i: (-score[i], i))
    return sorted(order[:b])


def test_select_brute_force_all_small_pools():
    rng = np.random.default_rng(7)
    for n in range(0, 17):
        for trial in range(30):
            kind = trial % 3
            if kind == 0:
                sc = rng.random(n)
            elif kind == 1:
                sc = np.full(n, 2.5)                           # all equal
            else:
                sc = rng.integers(0, 3, size=n).astype(float)  # two/three-level ties
                if n:
                    sc[rng.random(n) < 0.2] = -0.0
            for b in sorted({0, 1, n - 1, n, n // 2}):
                if b < 0 or b > n:
                    continue
                keep, rej = oracle.select(sc, b)
                assert rej.tolist() == _brute(sc.tolist(), b)
                assert int((keep == 0).sum()) == b
                if 0 < b < n:
                    assert sc[keep == 0].min() >= sc[keep == 1].max()


def test_select_every_subset_tiny():
    """Exhaustive over all score patterns in {0,1,2}^6 and every budget."""
    for pat in itertools.product((0.0, 1.0, 2.0), repeat=6):
        sc = np.array(pat)
        for b in range(0, 7):
            _, rej = oracle.select(sc, b)
            assert rej.tolist() == _brute(list(pat), b)


def test_select_errors():
    with pytest.raises(oracle.OracleError):
        oracle.select(np.array([1.0, np.nan]), 1)
    assert oracle.select(np.array([1.0, 2.0]), 3, check=False) == oracle.ERR_ARG


# --------------------------------------------------------------------------
# Compaction
# --------------------------------------------------------------------------
def test_compact_matches_numpy_concatenation():
    rng = np.random.default_rng(8)
    for trial in range(40):
        n = int(rng.integers(0, 50))
        lens = rng.integers(0, 200, size=n)
        lens[rng.random(n) < 0.2] = 0
        offsets = np.concatenate(([0], np.cumsum(lens))).astype(np.int64)
        N = int(offsets[-1])
        keep = (rng.random(n) < 0.6).astype(np.uint8)
        cols = [rng.integers(-5, 5, size=N).astype(np.int32),
                rng.integers(0, 255, size=N).astype(np.uint8),
                rng.integers(-300, 300, size=N).astype(np.int16),
                rng.random(N).astype(np.float64)]
        off_out, ids, packed = oracle.compact(offsets, keep, cols)
        kept = np.flatnonzero(keep)
        assert ids.tolist() == kept.tolist()
        assert off_out.tolist() == [0] + np.cumsum(lens[kept]).tolist()
        assert int(off_out[-1]) + int(lens[keep == 0].sum()) == N
        for c, pk in zip(cols, packed):
            ref = np.concatenate([c[offsets[i]:offsets[i + 1]] for i in kept]) if kept.size else c[:0]
            assert np.array_equal(ref, pk)


# --------------------------------------------------------------------------
# Preconditions (Lemma 1)
# --------------------------------------------------------------------------
def test_validate_rejects_broken_preconditions():
    tags = np.array([1, 2, 2, 3], np.int32)
    off = np.array([0, 2, 4], np.int64)
    comp = np.array([2, 3], np.int32)
    assert oracle.validate(tags, off, comp, 5) == oracle.OK
    assert oracle.validate(np.array([1, 3, 2, 3], np.int32), off, comp, 5) == oracle.ERR_PRECONDITION  # v > c
    assert oracle.validate(tags, off, np.array([2, 6], np.int32), 5) == oracle.ERR_PRECONDITION      # c > j
    assert oracle.validate(tags, np.array([0, 3, 2], np.int64), comp, 5) == oracle.ERR_PRECONDITION  # offsets
    assert oracle.validate(np.array([1, -2, 2, 3], np.int32), off, comp, 5) == oracle.ERR_PRECONDITION
    with pytest.raises(oracle.OracleError):
        oracle.score(np.array([1, 3, 2, 3], np.int32), off, comp, 5)


# --------------------------------------------------------------------------
# A planted mistake must fail a pin (checks the pins themselves, on the CPU)
# --------------------------------------------------------------------------
@settings(max_examples=60, deadline=None)
@given(st.lists(st.tuples(st.integers(0, 6), st.integers(0, 3), st.integers(1, 40)), min_size=1, max_size=12),
       st.integers(0, 20))
def test_property_lemma_identity(spec, extra_wait):
    """Hypothesis over pools: raw score * T == sum_t (j - v_t) exactly."""
    tags, offs, comp = [], [0], []
    for (base, nb, L) in spec:
        versions = base + np.sort(np.random.default_rng(L * 31 + nb).integers(0, nb + 1, size=L))
        c = int(versions.max()) + (nb % 2)
        tags.append(versions.astype(np.int32))
        offs.append(offs[-1] + L)
        comp.append(c)
    V = max(comp) + extra_wait
    t = np.concatenate(tags)
    sc, S, T = oracle.score(t, np.array(offs, np.int64), np.array(comp, np.int32), V)
    for i, seg in enumerate(tags):
        assert rel_close(sc[i], Fraction(int((V - seg.astype(np.int64)).sum()), seg.size))
