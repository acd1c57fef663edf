"""Pins of the oracle's streaming admission rule (Sec. 3.1, Algorithm 1):
the cutoff against numpy's inverted-CDF quantile, closed forms for the
draw, the reduction to exact top-b rejection when the window is the pool
itself, and the window ring against a plain list of everything observed."""
import numpy as np

import oracle


def _fill(w, values):
    for v in values:
        w.ring[w.head] = v
        w.head = (w.head + 1) % w.cap
        w.count = min(w.cap, w.count + 1)


def test_stream_cutoff_is_lower_empirical_quantile():
    rng = np.random.default_rng(31)
    for _ in range(200):
        cap = int(rng.integers(1, 600))
        w = oracle.StreamWindow(cap)
        _fill(w, rng.normal(0, 1, int(rng.integers(0, 2 * cap))).round(int(rng.integers(0, 4))))
        r = float(rng.choice([0.0, 0.1, 0.25, 0.5, 0.9, 0.95, rng.random()]))
        wmin = int(rng.integers(0, 40))
        entries = w.entries()
        st, kappa, drawn, kept = oracle.stream_admit(np.zeros(0), r, w, 0, window_min=wmin)
        rate = min(r, 0.9)
        if len(entries) < max(wmin, 1) or rate == 0.0:
            assert kappa == np.inf
        else:
            q = np.quantile(entries, 1.0 - rate, method="inverted_cdf")
            assert kappa == q, (len(entries), r)


def test_stream_zero_rate_rejects_nothing():
    rng = np.random.default_rng(32)
    w = oracle.StreamWindow(512)
    _fill(w, rng.random(512))
    s = rng.random(300) * 10
    st, kappa, drawn, kept = oracle.stream_admit(s, 0.0, w, 100)
    assert kappa == np.inf and drawn == kept == 100
    assert list(st) == [1] * 100 + [2] * 200


def test_stream_draw_invariants():
    rng = np.random.default_rng(33)
    for _ in range(300):
        n = int(rng.integers(0, 200))
        w = oracle.StreamWindow(int(rng.integers(1, 100)))
        _fill(w, rng.integers(0, 20, int(rng.integers(0, 150))).astype(float))
        s = rng.integers(0, 20, n).astype(float)
        B = int(rng.integers(0, n + 5))
        st, kappa, drawn, kept = oracle.stream_admit(s, float(rng.random()), w, B, window_min=int(rng.integers(0, 10)))
        assert kept == min(B, int((st == 1).sum())) and kept == int((st == 1).sum())
        assert drawn == int((st != 2).sum()) and all(st[:drawn] != 2) and all(st[drawn:] == 2)
        assert all(s[st == 0] > kappa) and all(s[st == 1] <= kappa)
        if kept < B:
            assert drawn == n
        else:
            assert drawn == 0 or st[drawn - 1] == 1          # the draw stops on the B-th retained one
        # a retained count reached exactly at the B-th score <= kappa in pool order
        if kept == B and B > 0:
            assert int((s[:drawn] <= kappa).sum()) == B


def test_stream_reduces_to_exact_top_b_when_window_is_the_pool():
    """Window = the pool's own scores, rate = b/N, draw the whole pool: with
    distinct scores the rejected set is exactly the b largest (C9)."""
    rng = np.random.default_rng(34)
    for _ in range(100):
        n = int(2 ** rng.integers(0, 10))          # b / n, 1 - b / n and (1 - b / n) n exact in binary64
        s = rng.permutation(n).astype(float) * 0.5 + rng.random() * 0.01
        b = int(rng.integers(0, n))
        w = oracle.StreamWindow(n)
        _fill(w, s)
        r = b / n
        st, kappa, drawn, kept = oracle.stream_admit(s, r, w, n, r_max=1.0, window_min=0)
        keep, rej = oracle.select(s, b)
        assert drawn == n
        assert np.array_equal(np.flatnonzero(st == 0), rej), (n, b)


def test_stream_window_holds_the_last_observed_scores():
    rng = np.random.default_rng(35)
    cap = 37
    w = oracle.StreamWindow(cap)
    seen = []
    for step in range(60):
        n = int(rng.integers(0, 30))
        s = rng.normal(0, 1, n)
        st, kappa, drawn, kept = oracle.stream_admit(s, float(rng.random()), w, int(rng.integers(0, 20)),
                                                     window_min=5)
        seen.extend(s[:drawn])
        assert np.array_equal(w.entries(), np.array(seen[-cap:]) if seen else np.zeros(0))
