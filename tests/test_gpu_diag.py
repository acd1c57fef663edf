"""GPU parity of Stale-k admission (Eq. (1) lag <= k) and the admission
diagnostics (Sec. 4), through the C ABI against the CPU oracle: keep flags,
lags, histograms and totals all bit-exact."""
import sys

import numpy as np
import pytest

import oracle
import poolgen

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(msg):
    sys.stdout.write("[gpu] %s\n" % msg)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def pace():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import os
    from paper_2609_36830_amd import _lib
    if not os.path.exists(_lib.library_path):
        from paper_2609_36830_amd import build
        build.build()
    import paper_2609_36830_amd as pace
    return pace


def D(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def H(t):
    return t.detach().cpu().numpy()


@pytest.mark.parametrize("name", ["tiny", "math", "multiturn", "stress"])
def test_stale_k_pools(pace, name):
    pool = poolgen.make_pool(name)
    sc, S, T = pace.pace_score(D(pool.tags), D(pool.offsets), D(pool.completion), pool.V)
    for k in (0, 2, 8, 100):
        say("stale-k %s k=%d" % (name, k))
        keep, lag = pace.pace_stale_k(S, T, D(pool.completion), pool.V, k)
        okeep, olag = oracle.stale_k(pool.tags, pool.offsets, pool.completion, pool.V, k)
        assert np.array_equal(H(keep), okeep)
        assert np.array_equal(H(lag).view(np.uint64), olag.view(np.uint64))


def test_stale_k_edge_shapes(pace):
    lens = np.array([0, 0, 1, 5, 0], np.int64)
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    tags = np.array([7, 10, -1, 10, 9, 8], np.int32)
    comp = np.array([10, 7, 10, 10, 10], np.int32)
    sc, S, T = pace.pace_score(D(tags), D(off), D(comp), 12)
    for k in (0, 1, 2, 3, 5):
        keep, lag = pace.pace_stale_k(S, T, D(comp), 12, k)
        okeep, olag = oracle.stale_k(tags, off, comp, 12, k)
        assert np.array_equal(H(keep), okeep) and np.array_equal(H(lag).view(np.uint64), olag.view(np.uint64))


@pytest.mark.parametrize("name", ["math", "multiturn", "stress"])
def test_diagnostics_pools(pace, name):
    pool = poolgen.make_pool(name)
    tags, off, comp = D(pool.tags), D(pool.offsets), D(pool.completion)
    sc, S, T = pace.pace_score(tags, off, comp, pool.V, D(pool.prefix_score), D(pool.window))
    b, _ = pace.pace_budget(pool.occupancy, pool.capacity)
    keep, _ = pace.pace_select(sc, b)
    osc, _, _ = oracle.score(pool.tags, pool.offsets, pool.completion, pool.V, pool.prefix_score, pool.window)
    okeep, _ = oracle.select(osc, b)
    assert np.array_equal(H(keep), okeep)
    rng = np.random.default_rng(81)
    for nb in (1, 9, 64, 1024):
        if nb == 9:
            edges = np.array([np.arange(10, dtype=np.float64)] * 3)
        else:
            edges = np.sort(rng.uniform(-1, 12, (3, nb + 1)), axis=1)
        say("diagnostics %s nbins=%d" % (name, nb))
        h, t = pace.pace_diagnostics(sc, S, T, comp, pool.V, keep, D(edges))
        oh, ot = oracle.diagnostics(pool.tags, pool.offsets, pool.completion, pool.V, osc, okeep, edges)
        assert np.array_equal(H(h), oh) and np.array_equal(H(t), ot)


def _direct_pool(rng, n, V=40):
    """Short trajectories (0..6 tokens) with tags in [c - 9, c] or -1."""
    lens = rng.integers(0, 7, n).astype(np.int64)
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    comp = rng.integers(0, V + 1, n).astype(np.int32)
    owner = np.repeat(np.arange(n), lens)
    c_tok = comp[owner].astype(np.int64)
    tags = np.maximum(c_tok - rng.integers(0, 10, owner.size), 0).astype(np.int32)
    tags[rng.random(owner.size) < 0.2] = -1
    return tags, off, comp


@pytest.mark.parametrize("n", [0, 1, 5, 1023, 1025, 4097, 10001])
def test_diagnostics_shapes(pace, n):
    """Empty, sub-round and several-round pools; NaN and infinite scores,
    scores and metrics exactly on edges, repeated edges, keep bytes above 1
    (retained), and bin counts from 1 to the maximum."""
    rng = np.random.default_rng(1000 + n)
    V = 40
    tags, off, comp = _direct_pool(rng, n, V)
    sc, S, T = pace.pace_score(D(tags), D(off), D(comp), V)
    osc, _, _ = oracle.score(tags, off, comp, V)
    assert np.array_equal(H(sc).view(np.uint64), osc.view(np.uint64))
    score = osc.copy()
    if n:
        pick = rng.integers(0, n, max(1, n // 7))
        score[pick] = rng.choice([np.nan, np.inf, -np.inf, 0.0, 3.0, 12.0], pick.size)
    keep = rng.choice(np.array([0, 1, 2, 255], np.uint8), n)
    for nb in (1, 2, 63, 64, 1023, 1024):
        if nb in (2, 63):
            # repeated edges, integer-valued so that K_wait lands on them
            base = np.sort(rng.integers(0, 13, nb + 1)).astype(np.float64)
            edges = np.array([base] * 3)
        else:
            edges = np.sort(rng.uniform(-1, 30, (3, nb + 1)), axis=1)
        say("diagnostics direct n=%d nbins=%d" % (n, nb))
        h, t = pace.pace_diagnostics(D(score), S, T, D(comp), V, D(keep), D(edges))
        oh, ot = oracle.diagnostics(tags, off, comp, V, score, keep, edges)
        assert np.array_equal(H(h), oh) and np.array_equal(H(t), ot)
