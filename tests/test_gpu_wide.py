"""GPU parity of the selection spread over the chip: pools beyond the rank
kernel's 8192 trajectories, where pace_filter_step and pace_select find the
rejection cut with per-workgroup histograms and one cut workgroup, then
classify every trajectory and compact with blocks of 64 trajectories.

Same bar as the other parity tests: S, T, score bits, budgets, keep flags,
reject ids, packed offsets, kept ids and packed columns are bit-exact against
the oracle. The cut search has several ways to end (a bin rejected whole,
pairwise ranking of the last candidates, equal keys ordered by id,
refinement from global memory when a bin holds more candidates than LDS),
and the score arrays below are built to reach each of them.
"""
import sys

import numpy as np
import pytest

import oracle
import poolgen

from tests.test_gpu_parity import D, H, assert_same, gpu_step, oracle_step

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def say(msg):
    sys.stdout.write("[gpu] %s\n" % msg)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def pace():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2609_36830_amd as pace
    return pace


FUSED = pytest.mark.parametrize("fused", [False, True], ids=["calls", "fused"])


@FUSED
@pytest.mark.parametrize("n", [16384, 65536])
def test_wide_pool_parity(pace, n, fused):
    """The scale pool (65536 trajectories, ~52M tokens) and its first 16384
    trajectories' recipe at n = 16384."""
    pool = poolgen.make_pool("wide", n=n)
    say("wide pool n=%d tokens=%d fused %s" % (pool.n, pool.n_tokens, fused))
    assert_same(gpu_step(pace, pool, fused=fused), oracle_step(pool), "wide n=%d" % n)


@FUSED
@pytest.mark.parametrize("mode", ["raw", "gen"])
def test_wide_pool_other_modes(pace, mode, fused):
    pool = poolgen.make_pool("wide", n=20000, seed=7)
    say("wide pool n=20000 mode %s fused %s" % (mode, fused))
    assert_same(gpu_step(pace, pool, mode=mode, fused=fused), oracle_step(pool, mode=mode), mode)


@FUSED
def test_wide_ties(pace, fused):
    """Raw scores of constant-version trajectories take few distinct values:
    long runs of equal keys around the cut, ordered by id."""
    rng = np.random.default_rng(5)
    lens = rng.integers(1, 300, size=30000)
    pool = poolgen.make_custom_pool(lens, V=12, seed=5, max_breaks=0, c_lag=3, W=0)
    say("wide ties n=%d" % pool.n)
    r = oracle_step(pool, mode="raw")
    assert len(np.unique(r["score"])) < 20
    assert_same(gpu_step(pace, pool, mode="raw", fused=fused), r, "ties")


@FUSED
@pytest.mark.parametrize("capacity,r_max", [(12000, 0.9), (11999, 0.9), (1, 0.9), (0, 1.0)])
def test_wide_budget_extremes(pace, capacity, r_max, fused):
    lens = np.random.default_rng(capacity + 3).integers(0, 500, size=12000)
    pool = poolgen.make_custom_pool(lens, V=50, seed=11, mask_frac=0.05, capacity=capacity, W=256)
    params = pace.default_params(r_max=r_max)
    say("wide budget capacity %d r_max %g fused %s" % (capacity, r_max, fused))
    g = gpu_step(pace, pool, params=params, fused=fused)
    r = oracle_step(pool, r_max=r_max)
    assert_same(g, r, "capacity %d" % capacity)


@pytest.mark.parametrize("n", [8193, 20000, 262144])
def test_wide_filter_step_edges(pace, n):
    """Ragged sizes, empty trajectories, masked tokens."""
    rng = np.random.default_rng(n)
    lens = rng.integers(0, 80, size=n)
    lens[rng.random(n) < 0.1] = 0
    pool = poolgen.make_custom_pool(lens, V=90, seed=n, mask_frac=0.2, W=512)
    say("wide edges n=%d tokens=%d" % (n, pool.n_tokens))
    assert_same(gpu_step(pace, pool, fused=True), oracle_step(pool), "edges n=%d" % n)


def _select_both(pace, sc, b, what):
    keep, rej = pace.pace_select(D(sc), b)
    torch.cuda.synchronize()
    rk, rr = oracle.select(sc, b)
    assert np.array_equal(H(keep), rk), ("keep", what, len(sc), b)
    assert np.array_equal(H(rej), rr), ("reject ids", what, len(sc), b)


def _score_cases(n, rng):
    one = 1.0
    ulp = np.nextafter(one, 2.0) - one
    cluster = rng.random(n)
    cluster[: n // 2] = 0.625                       # half the keys equal, the cut inside them
    return {
        "random": rng.random(n),
        "all_equal": np.full(n, 4.5),
        "two_values": np.where(rng.random(n) < 0.3, 2.0, 1.0),
        "cluster": cluster,
        "last_bits": one + rng.integers(0, 300, n) * ulp,    # keys differing in the low bits only
        "signed_zero_inf": np.choose(rng.integers(0, 4, n), [-0.0, 0.0, np.inf, -np.inf]),
        "wide_range": rng.standard_normal(n) * 10.0 ** rng.integers(-300, 300, n),
        "sorted_desc": np.sort(rng.random(n))[::-1].copy(),
        "integers": rng.integers(0, 5000, n).astype(float),
    }


@pytest.mark.parametrize("n", [8193, 16385, 50000, 262144])
def test_wide_select_cases(pace, n):
    rng = np.random.default_rng(n + 1)
    for name, sc in _score_cases(n, rng).items():
        say("wide select n=%d %s" % (n, name))
        for b in sorted({0, 1, n // 3, n // 2, n // 2 + 1, n - 1, n}):
            _select_both(pace, sc, b, name)


def test_wide_select_beyond_limit(pace):
    """262145 trajectories take the single-workgroup selection."""
    n = 262145
    sc = np.random.default_rng(3).random(n)
    say("select n=%d" % n)
    for b in (1, n // 2, n - 1):
        _select_both(pace, sc, b, "beyond")


@FUSED
def test_wide_multi_column_payload(pace, fused):
    """Blocks of 64 with every column width: int32 and fp32 columns copy by
    16-byte slots, the uint8 and int16 ones element by element, fp64 and
    int64 by slots of two elements."""
    pool = poolgen.make_pool("wide", n=20000, seed=9)
    rng = np.random.default_rng(9)
    N = pool.n_tokens
    cols = [pool.tags, rng.integers(0, 150000, N).astype(np.int32), rng.standard_normal(N).astype(np.float32),
            (pool.tags != -1).astype(np.uint8), (np.arange(N) % 30000).astype(np.int16), rng.standard_normal(N),
            rng.integers(-2 ** 62, 2 ** 62, N, dtype=np.int64)]
    say("wide multi-column n=%d tokens=%d fused %s" % (pool.n, N, fused))
    assert_same(gpu_step(pace, pool, cols=cols, fused=fused), oracle_step(pool, cols=cols), "wide multi-column")


def test_wide_unaligned_columns(pace):
    """Column pointers off 16-byte alignment take the element slots."""
    pool = poolgen.make_pool("wide", n=12000, seed=13)
    r = oracle_step(pool)
    N = pool.n_tokens
    rng = np.random.default_rng(13)
    host = [rng.integers(-2 ** 31, 2 ** 31 - 1, N).astype(np.int32), rng.standard_normal(N)]
    cols = []
    for h in host:
        big = torch.empty(N + 1, dtype=torch.from_numpy(h[:1]).dtype, device="cuda:0")
        big[1:] = D(h)
        cols.append(big[1:])
        assert cols[-1].data_ptr() % 16 != 0
    say("wide unaligned columns n=%d tokens=%d" % (pool.n, N))
    oo, ids, nkt, packed = pace.pace_compact(D(pool.offsets), D(r["keep"]), cols, n_tokens=N)
    torch.cuda.synchronize()
    nk = int(H(nkt)[0])
    assert nk == r["n_kept_tokens"]
    keep = r["keep"].astype(bool)
    spans = [np.arange(pool.offsets[i], pool.offsets[i + 1]) for i in range(pool.n) if keep[i]]
    idx = np.concatenate(spans) if spans else np.empty(0, np.int64)
    for h, p in zip(host, packed):
        assert np.array_equal(H(p)[:nk], h[idx])
