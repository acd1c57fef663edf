"""GPU parity: the HIP library, called through the C ABI, against the CPU
oracle on the same seeded pools, element by element.

Bar: version reductions (S, T), budgets, keep flags, reject ids, packed
offsets, kept ids and packed columns are bit-exact. Scores are within 1e-12
relative (the stated tolerance) and, because both sides evaluate the same
IEEE binary64 operations in the same order, are also required to be
bit-identical -- a reject set decided from scores that differ in the last
bit could otherwise differ at a near-tie.
"""
import sys

import numpy as np
import pytest

import oracle
import poolgen

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


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


DEV = "cuda:0"


def D(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def H(t):
    return t.detach().cpu().numpy()


def gpu_step(pace, pool, mode="effective", cols=None, params=None, r_hat_prev=0.0, fused=False):
    """One filter step through the C ABI: the four separate calls, or
    pace_filter_step when fused."""
    params = params or pace.default_params(w_wait=0.0 if mode == "gen" else 1.0)
    tags, off, comp = D(pool.tags), D(pool.offsets), D(pool.completion)
    prefix = None if mode == "raw" else D(pool.prefix_score)
    window = None if mode == "raw" else D(pool.window)
    cols_d = [tags] if cols is None else [D(c) for c in cols]
    if fused:
        r = pace.pace_filter_step(tags, off, comp, pool.V, pool.occupancy, pool.capacity, cols_d, prefix,
                                  window, params, r_hat_prev)
        torch.cuda.synchronize()
        b = r["budget"]
        n_kept = pool.n - b
        nk = int(H(r["n_kept_tokens"])[0])
        return dict(score=H(r["score"]), S=H(r["gen_sum"]), T=H(r["gen_count"]), budget=b, r_hat=r["r_hat"],
                    keep=H(r["keep"]), reject_ids=H(r["reject_ids"]), offsets_out=H(r["offsets_out"])[: n_kept + 1],
                    kept_ids=H(r["kept_ids"])[:n_kept], n_kept_tokens=nk,
                    packed=[H(p)[:nk] for p in r["cols_out"]])
    sc, S, T = pace.pace_score(tags, off, comp, pool.V, prefix, window, params)
    b, rh = pace.pace_budget(pool.occupancy, pool.capacity, params, r_hat_prev)
    keep, rej = pace.pace_select(sc, b)
    oo, ids, nkt, packed = pace.pace_compact(off, keep, cols_d, n_tokens=pool.n_tokens)
    torch.cuda.synchronize()
    n_kept = pool.n - b
    nk = int(H(nkt)[0])
    return dict(score=H(sc), S=H(S), T=H(T), budget=b, r_hat=rh, keep=H(keep), reject_ids=H(rej),
                offsets_out=H(oo)[: n_kept + 1], kept_ids=H(ids)[:n_kept], n_kept_tokens=nk,
                packed=[H(p)[:nk] for p in packed])


def assert_same(g, r, what=""):
    assert np.array_equal(g["S"], r["S"]), what + " S"
    assert np.array_equal(g["T"], r["T"]), what + " T"
    np.testing.assert_allclose(g["score"], r["score"], rtol=1e-12, atol=0, err_msg=what + " score")
    assert np.array_equal(g["score"].view(np.int64), r["score"].view(np.int64)), what + " score bits"
    assert g["budget"] == r["budget"] and g["r_hat"] == r["r_hat"], what + " budget"
    assert np.array_equal(g["keep"], r["keep"]), what + " keep"
    assert np.array_equal(g["reject_ids"], r["reject_ids"]), what + " reject ids"
    assert np.array_equal(g["offsets_out"], r["offsets_out"]), what + " offsets_out"
    assert np.array_equal(g["kept_ids"], r["kept_ids"]), what + " kept_ids"
    assert g["n_kept_tokens"] == r["n_kept_tokens"], what + " n_kept_tokens"
    for a, b in zip(g["packed"], r["packed"]):
        assert np.array_equal(a, b), what + " packed column"


def oracle_step(pool, mode="effective", cols=None, r_hat_prev=0.0, beta=0.0, gamma=4, window_min=32,
                r_max=0.9):
    return oracle.filter_step(pool, mode=mode, cols=cols, r_hat_prev=r_hat_prev, beta=beta,
                              gamma=gamma, window_min=window_min, r_max=r_max)


# ---------------------------------------------------------------------------
# The paper-shaped pools at their full sizes
# ---------------------------------------------------------------------------
FUSED = pytest.mark.parametrize("fused", [False, True], ids=["calls", "fused"])


@FUSED
@pytest.mark.parametrize("name", ["tiny", "math", "long", "multiturn"])
@pytest.mark.parametrize("mode", ["effective", "raw", "gen"])
def test_pool_parity(pace, name, mode, fused):
    pool = poolgen.make_pool(name)
    say("pool %s mode %s fused %s n=%d tokens=%d" % (name, mode, fused, pool.n, pool.n_tokens))
    assert_same(gpu_step(pace, pool, mode, fused=fused), oracle_step(pool, mode), "%s/%s" % (name, mode))


@FUSED
@pytest.mark.parametrize("mode", ["effective", "raw", "gen"])
def test_stress_pool_parity(pace, mode, fused):
    pool = poolgen.make_pool("stress")
    say("stress %s fused %s n=%d tokens=%d" % (mode, fused, pool.n, pool.n_tokens))
    g = gpu_step(pace, pool, mode, fused=fused)
    assert_same(g, oracle_step(pool, mode), "stress/" + mode)
    assert g["budget"] == 2731


@FUSED
@pytest.mark.parametrize("seed", [7, 8, 9])
@pytest.mark.parametrize("name", ["tiny", "math", "multiturn"])
def test_other_seeds(pace, name, seed, fused):
    pool = poolgen.make_pool(name, seed=seed, n=512 if name != "tiny" else None)
    say("seed %d pool %s fused %s" % (seed, name, fused))
    assert_same(gpu_step(pace, pool, fused=fused), oracle_step(pool), "%s seed %d" % (name, seed))


@FUSED
def test_stress_three_columns(pace, fused):
    """The stress pool with the three payload columns the benchmark's
    multi-column run carries: tags, int32 token ids, fp32 log-probs."""
    pool = poolgen.make_pool("stress")
    rng = np.random.default_rng(11)
    N = pool.n_tokens
    cols = [pool.tags, rng.integers(0, 150000, N).astype(np.int32), rng.standard_normal(N).astype(np.float32)]
    say("stress three columns fused %s tokens=%d" % (fused, N))
    assert_same(gpu_step(pace, pool, cols=cols, fused=fused), oracle_step(pool, cols=cols), "stress/3 cols")


@FUSED
def test_multi_column_payload(pace, fused):
    """Tags plus token ids (int32), behavior log-probs (fp32), a loss mask
    (uint8), positions (int16) and fp64 values, as separate columns."""
    pool = poolgen.make_pool("multiturn", n=700)
    rng = np.random.default_rng(3)
    N = pool.n_tokens
    cols = [pool.tags, rng.integers(0, 150000, N).astype(np.int32), rng.standard_normal(N).astype(np.float32),
            (pool.tags != -1).astype(np.uint8), (np.arange(N) % 30000).astype(np.int16),
            rng.standard_normal(N)]
    say("multi-column n=%d tokens=%d" % (pool.n, N))
    assert_same(gpu_step(pace, pool, cols=cols, fused=fused), oracle_step(pool, cols=cols), "multi-column")


# ---------------------------------------------------------------------------
# Edge cases
# ---------------------------------------------------------------------------
EDGE_LENGTHS = {
    "empty_pool": [],
    "one_empty": [0],
    "one_token": [1],
    "zeros_and_ones": [0, 1, 0, 0, 1, 1, 0, 2, 0, 3],
    "window_edges": [255, 256, 257, 2047, 2048, 2049, 8191, 8192, 8193, 0, 4096, 4097, 1023, 1025],
    "long_single": [100_000],
    "long_mixed": [3, 70_000, 0, 5, 40_000, 1, 1],
    "many_tiny": list(np.random.default_rng(5).integers(0, 6, size=5000)),
    "ragged_tail": list(np.random.default_rng(6).integers(100, 900, size=300)) + [3],
}


@FUSED
@pytest.mark.parametrize("case", sorted(EDGE_LENGTHS))
@pytest.mark.parametrize("mask_frac", [0.0, 0.35])
def test_edge_shapes(pace, case, mask_frac, fused):
    lens = EDGE_LENGTHS[case]
    pool = poolgen.make_custom_pool(lens, V=40, seed=len(lens) + 17, mask_frac=mask_frac, W=64)
    say("edge %s mask %.2f fused %s n=%d tokens=%d" % (case, mask_frac, fused, pool.n, pool.n_tokens))
    assert_same(gpu_step(pace, pool, fused=fused), oracle_step(pool), case)


@pytest.mark.parametrize("n", [8192, 8193])
@FUSED
def test_pool_at_rank_limit(pace, n, fused):
    """8192 trajectories take the rank-and-piece kernels in the fused call,
    8193 the separate ones."""
    lens = np.random.default_rng(n).integers(0, 700, size=n)
    pool = poolgen.make_custom_pool(lens, V=80, seed=n, mask_frac=0.1, W=512)
    say("n=%d fused %s" % (n, fused))
    assert_same(gpu_step(pace, pool, fused=fused), oracle_step(pool), "n=%d" % n)


@FUSED
def test_pool_above_register_capacity(pace, fused):
    """20000 trajectories: the fused call falls back to the separate kernels."""
    lens = np.random.default_rng(9).integers(0, 400, size=20000)
    pool = poolgen.make_custom_pool(lens, V=60, seed=99, mask_frac=0.1, W=512)
    say("n=20000 fused %s" % fused)
    assert_same(gpu_step(pace, pool, fused=fused), oracle_step(pool), "n=20000")


@FUSED
def test_all_masked_trajectories(pace, fused):
    pool = poolgen.make_custom_pool([500, 0, 300, 1000], V=30, seed=4, W=64)
    pool.tags[:500] = -1
    pool.tags[800:1800] = -1
    r = oracle_step(pool)
    assert r["T"][0] == 0 and r["T"][3] == 0
    assert_same(gpu_step(pace, pool, fused=fused), r, "all-masked")


def test_unaligned_tags_take_the_scalar_path(pace):
    pool = poolgen.make_pool("math", n=300)
    say("unaligned tags")
    big = torch.empty(pool.n_tokens + 1, dtype=torch.int32, device=DEV)
    big[1:] = D(pool.tags)
    tags = big[1:]
    assert tags.data_ptr() % 16 != 0
    params = pace.default_params()
    off, comp = D(pool.offsets), D(pool.completion)
    sc, S, T = pace.pace_score(tags, off, comp, pool.V, D(pool.prefix_score), D(pool.window), params)
    r = oracle_step(pool)
    assert np.array_equal(H(S), r["S"]) and np.array_equal(H(T), r["T"])
    assert np.array_equal(H(sc), r["score"])
    keep = D(r["keep"])
    oo, ids, nkt, packed = pace.pace_compact(off, keep, [tags], n_tokens=pool.n_tokens)
    torch.cuda.synchronize()
    assert np.array_equal(H(packed[0])[: r["n_kept_tokens"]], r["packed"][0])


@FUSED
def test_large_versions_take_the_wide_path(pace, fused):
    lens = [700, 20000, 5, 9000]
    pool = poolgen.make_custom_pool(lens, V=2 ** 30, seed=12, mask_frac=0.1, W=64)
    say("wide versions V=2^30 fused %s" % fused)
    assert_same(gpu_step(pace, pool, fused=fused), oracle_step(pool), "wide")


@FUSED
@pytest.mark.parametrize("V", [32766, 32767, 2 ** 24 - 2, 2 ** 24 - 1])
def test_reduce_mode_limits(pace, V, fused):
    """Every tag at V, next to the limits where the reduction changes its
    arithmetic (packed 2^15, 32-bit 2^24): full windows of the largest tags
    must neither carry into the packed count nor overflow a 32-bit window
    sum. Lengths put offsets at window edges and many windows inside one
    trajectory; a tenth of the tokens are masked."""
    lens = [70000, 1, 255, 256, 257, 3000, 0, 4096, 12345, 2047, 2049] + [300] * 40
    pool = poolgen.make_custom_pool(lens, V=V, seed=V % 1000, mask_frac=0.1, c_lag=0, W=64)
    pool.tags[:] = np.where(pool.tags == -1, -1, V).astype(np.int32)
    pool.completion[:] = V
    say("reduce limits V=%d fused %s" % (V, fused))
    assert_same(gpu_step(pace, pool, fused=fused), oracle_step(pool), "V=%d" % V)


@FUSED
def test_large_versions_many_boundaries(pace, fused):
    """64-bit window prefixes: short trajectories put boundaries in most
    blocks of the reduction while tag + 1 reaches 2^30."""
    lens = np.random.default_rng(31).integers(0, 300, size=3000)
    pool = poolgen.make_custom_pool(lens, V=2 ** 30, seed=31, mask_frac=0.2, W=64)
    say("wide versions, short trajectories fused %s" % fused)
    assert_same(gpu_step(pace, pool, fused=fused), oracle_step(pool), "wide short")


@FUSED
@pytest.mark.parametrize("gamma", [1, 2, 3, 4])
def test_gamma_and_window_min(pace, gamma, fused):
    pool = poolgen.make_pool("math", n=400)
    for wmin in (0, 32, 600):
        params = pace.default_params(gamma=gamma, window_min=wmin)
        say("gamma %d window_min %d fused %s" % (gamma, wmin, fused))
        g = gpu_step(pace, pool, params=params, fused=fused)
        r = oracle_step(pool, gamma=gamma, window_min=wmin)
        assert_same(g, r, "gamma %d wmin %d" % (gamma, wmin))


@FUSED
def test_large_window_in_global_memory(pace, fused):
    """A 6000-entry prefix window (beyond the LDS-staged size), gamma = 1."""
    pool = poolgen.make_custom_pool(np.full(300, 100), V=50, seed=21, W=6000)
    params = pace.default_params(gamma=1)
    say("window 6000 fused %s" % fused)
    assert_same(gpu_step(pace, pool, params=params, fused=fused), oracle_step(pool, gamma=1), "big window")


@FUSED
def test_budget_extremes(pace, fused):
    pool = poolgen.make_pool("tiny")
    for cap, rmax in ((64, 0.9), (200, 0.9), (0, 1.0), (0, 0.9), (63, 0.9)):
        pool.capacity = cap
        params = pace.default_params(r_max=rmax)
        say("budget capacity %d r_max %.1f fused %s" % (cap, rmax, fused))
        g = gpu_step(pace, pool, params=params, fused=fused)
        r = oracle_step(pool, r_max=rmax)
        assert_same(g, r, "capacity %d" % cap)


@FUSED
def test_ema_sequence(pace, fused):
    """beta = 0.9 across consecutive steps: r_hat threads through the host call."""
    pool = poolgen.make_pool("tiny")
    rg = ro = 0.0
    for occ in (64, 64, 60, 55, 49, 48, 40, 64):
        pool.occupancy = occ
        params = pace.default_params(beta=0.9)
        g = gpu_step(pace, pool, params=params, r_hat_prev=rg, fused=fused)
        r = oracle_step(pool, beta=0.9, r_hat_prev=ro)
        assert_same(g, r, "ema occ %d" % occ)
        rg, ro = g["r_hat"], r["r_hat"]


# ---------------------------------------------------------------------------
# Selection in isolation (same score array on both sides)
# ---------------------------------------------------------------------------
def _select_both(pace, sc, b):
    keep, rej = pace.pace_select(D(sc), b)
    torch.cuda.synchronize()
    rk, rr = oracle.select(sc, b)
    assert np.array_equal(H(keep), rk), ("keep", len(sc), b)
    assert np.array_equal(H(rej), rr), ("reject ids", len(sc), b)


def test_select_brute_force_small(pace):
    rng = np.random.default_rng(31)
    say("select n<=16 all budgets")
    for n in range(1, 17):
        for trial in range(6):
            sc = rng.integers(0, 3, n).astype(float) if trial % 2 else rng.random(n)
            if trial == 4:
                sc[:] = -0.0
            for b in range(0, n + 1):
                _select_both(pace, sc, b)


@pytest.mark.parametrize("n", [1023, 1024, 1025, 4096, 4097, 8192, 8193, 16384, 16385, 50000])
def test_select_sizes_and_ties(pace, n):
    rng = np.random.default_rng(n)
    say("select n=%d" % n)
    cases = [rng.random(n), rng.integers(0, 9, n).astype(float), np.full(n, 3.25),
             np.where(rng.random(n) < 0.5, -0.0, 0.0), rng.standard_normal(n) * 1e300,
             np.concatenate([np.full(n // 2, np.inf), -np.inf * np.ones(n - n // 2)])]
    for sc in cases:
        for b in sorted({0, 1, n // 3, n // 2, n - 1, n}):
            _select_both(pace, sc, b)


# ---------------------------------------------------------------------------
# Validation of preconditions on the device
# ---------------------------------------------------------------------------
def test_validate_flags(pace):
    pool = poolgen.make_pool("multiturn", n=300)
    say("validate")

    def run(tags, off, comp, V, window):
        e = pace.pace_validate(D(tags), D(off), D(comp), V, D(window))
        torch.cuda.synchronize()
        return int(H(e)[0])

    assert run(pool.tags, pool.offsets, pool.completion, pool.V, pool.window) == 0
    t = pool.tags.copy()
    i = int(np.flatnonzero(t >= 0)[1234])
    t[i] = pool.V + 5
    assert run(t, pool.offsets, pool.completion, pool.V, pool.window) == pace.BAD_TAG
    t = pool.tags.copy()
    t[7] = -3
    assert run(t, pool.offsets, pool.completion, pool.V, pool.window) == pace.BAD_TAG
    c = pool.completion.copy()
    c[5] = pool.V + 1
    assert run(pool.tags, pool.offsets, c, pool.V, pool.window) & pace.BAD_COMPLETION
    o = pool.offsets.copy()
    o[10], o[11] = o[11], o[10]
    assert run(pool.tags, o, pool.completion, pool.V, pool.window) & pace.BAD_OFFSETS
    w = pool.window.copy()
    w[3], w[4] = w[4], w[3] + 1.0
    assert run(pool.tags, pool.offsets, pool.completion, pool.V, w) == pace.BAD_WINDOW
    for name in ("tiny", "math"):
        p = poolgen.make_pool(name)
        assert run(p.tags, p.offsets, p.completion, p.V, p.window) == 0
        assert oracle.validate(p.tags, p.offsets, p.completion, p.V) == 0


# ---------------------------------------------------------------------------
# Determinism: identical bits run to run
# ---------------------------------------------------------------------------
@FUSED
def test_repeat_runs_identical(pace, fused):
    pool = poolgen.make_pool("long")
    say("determinism x5 on long pool fused %s" % fused)
    first = gpu_step(pace, pool, fused=fused)
    for _ in range(4):
        again = gpu_step(pace, pool, fused=fused)
        for k in ("score", "S", "T", "keep", "reject_ids", "offsets_out", "kept_ids"):
            assert np.array_equal(first[k], again[k]), k
        assert np.array_equal(first["packed"][0], again["packed"][0])
