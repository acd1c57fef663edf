"""GPU parity of group-level admission (Appendix B: mean aggregation within
prompt groups; groups budgeted, selected and compacted as units): the HIP
library through the C ABI against the CPU oracle, bit-exact (group scores
too: both sides add the members in order and divide once)."""
import dataclasses
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


def random_groups(rng, n, max_size=12, empty_frac=0.1, trailing_empty=True):
    sizes, left = [], n
    while left > 0:
        s = 0 if rng.random() < empty_frac else int(rng.integers(1, max_size + 1))
        s = min(s, left)
        sizes.append(s)
        left -= s
    if trailing_empty:
        sizes.append(0)
    return np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)


def group_step_parity(pace, pool, go, occ, cap, mode="effective", out=None):
    params = pace.default_params(w_wait=0.0 if mode == "gen" else 1.0)
    prefix = None if mode == "raw" else D(pool.prefix_score)
    window = None if mode == "raw" else D(pool.window)
    tags = D(pool.tags)
    r = pace.pace_group_filter_step(tags, D(pool.offsets), D(pool.completion), pool.V, D(go), occ, cap, [tags],
                                    prefix, window, params, out=out(tags) if out else None)
    torch.cuda.synchronize()
    o = oracle.group_filter_step(pool, go, occ, cap, mode=mode)
    assert r["budget"] == o["budget"]
    assert np.array_equal(H(r["score"]).view(np.uint64), o["score"].view(np.uint64))
    assert np.array_equal(H(r["gen_sum"]), o["S"]) and np.array_equal(H(r["gen_count"]), o["T"])
    assert np.array_equal(H(r["group_score"]).view(np.uint64), o["group_score"].view(np.uint64))
    assert np.array_equal(H(r["group_keep"]), o["group_keep"])
    assert np.array_equal(H(r["reject_group_ids"]), o["reject_group_ids"])
    assert np.array_equal(H(r["keep"]), o["keep"])
    n_kept = int(o["keep"].sum())
    nk = int(H(r["n_kept_tokens"])[0])
    assert nk == o["n_kept_tokens"]
    assert np.array_equal(H(r["offsets_out"])[: n_kept + 1], o["offsets_out"])
    assert np.array_equal(H(r["kept_ids"])[:n_kept], o["kept_ids"])
    assert np.array_equal(H(r["cols_out"][0])[:nk], o["packed"][0])
    return o


@pytest.mark.parametrize("mode", ["effective", "raw", "gen"])
def test_group_step_math_pool(pace, mode):
    pool = poolgen.make_pool("math")
    go = pool.group_offsets
    ng = len(go) - 1
    say("group step math pool mode=%s groups=%d" % (mode, ng))
    o = group_step_parity(pace, pool, go, ng, (pool.capacity + 7) // 8, mode)
    assert o["budget"] > 0


@pytest.mark.parametrize("grouping", ["eights", "random", "singletons", "one_group"])
def test_group_step_stress_pool(pace, grouping):
    pool = poolgen.make_pool("stress")
    rng = np.random.default_rng(21)
    if grouping == "eights":
        go = np.arange(0, pool.n + 1, 8, dtype=np.int64)
    elif grouping == "random":
        go = random_groups(rng, pool.n)
    elif grouping == "singletons":
        go = np.arange(pool.n + 1, dtype=np.int64)
    else:
        go = np.array([0, pool.n], np.int64)
    ng = len(go) - 1
    say("group step stress pool grouping=%s groups=%d" % (grouping, ng))
    group_step_parity(pace, pool, go, ng, ng // 3)


def test_group_step_reused_buffers(pace):
    """Preallocated outputs, reused across calls on two different pools of the
    same shape, give the oracle's results each time."""
    pool_a = poolgen.make_pool("math", n=300)
    pool_b = poolgen.make_pool("math", n=300, seed=9)
    go = np.arange(0, pool_a.n + 1, 4, dtype=np.int64)
    ng = len(go) - 1
    big = pool_a if pool_a.n_tokens >= pool_b.n_tokens else pool_b
    bufs = pace.group_step_buffers(pool_a.n, ng, [D(big.tags)], DEV)
    say("group step reused buffers, %d groups, %d and %d tokens" % (ng, pool_a.n_tokens, pool_b.n_tokens))
    for pool in (pool_a, pool_b, pool_a):
        group_step_parity(pace, pool, go, ng, ng // 3, out=lambda tags: bufs)
    with pytest.raises(ValueError):
        t = D(big.tags)
        pace.pace_group_filter_step(t, D(big.offsets), D(big.completion), big.V, D(go), ng, ng // 3,
                                    [t], out=pace.group_step_buffers(big.n, ng, [t[:-1]], DEV))


def test_group_step_more_groups_than_trajectories(pace):
    pool = poolgen.make_pool("tiny")
    rng = np.random.default_rng(22)
    go = random_groups(rng, pool.n, max_size=3, empty_frac=0.6)
    ng = len(go) - 1
    assert ng > pool.n
    say("group step tiny pool, %d groups over %d trajectories" % (ng, pool.n))
    group_step_parity(pace, pool, go, ng, ng // 2)


@pytest.mark.parametrize("empties,label", [(6, "7 groups per trajectory, under the 8192-group limit"),
                                           (8, "9 groups per trajectory, past the limit")])
def test_group_step_many_empty_groups(pace, empties, label):
    # Each of the math pool's 1024 trajectories follows `empties` empty
    # groups: 1024 trajectories then span more group offsets than one
    # workgroup stages (so threads search the global offsets too), and 9 per
    # trajectory take the group count past the fused step's limit.
    pool = poolgen.make_pool("math")
    sizes = np.tile(np.array([0] * empties + [1], np.int64), pool.n)
    go = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    ng = len(go) - 1
    say("group step math pool, %d groups (%s)" % (ng, label))
    o = group_step_parity(pace, pool, go, ng, ng - 512)
    assert 0 < int(o["keep"].sum()) < pool.n


@pytest.mark.parametrize("n,size", [(16384, 8), (65536, 8), (20000, 3)])
def test_group_step_wide_pools(pace, n, size):
    # Past 8192 trajectories the compaction takes blocks of 64 with group
    # sums (merge path); up to 8192 groups the fused group path writes them.
    pool = poolgen.make_pool("wide", n=n)
    rng = np.random.default_rng(n + size)
    if size == 3:
        go = random_groups(rng, pool.n, max_size=5, empty_frac=0.05)
    else:
        go = np.arange(0, pool.n + size, size, dtype=np.int64)
        go[-1] = pool.n
    ng = len(go) - 1
    say("group step wide pool n=%d, %d groups" % (pool.n, ng))
    o = group_step_parity(pace, pool, go, ng, ng // 3)
    assert 0 < int(o["keep"].sum()) < pool.n


def test_group_step_no_trajectories(pace):
    # Every group empty: the group scores are 0, the rejected ids are the
    # lowest ids, and nothing is packed.
    pool = poolgen.make_pool("tiny")
    empty = dataclasses.replace(pool, tags=pool.tags[:0], offsets=np.zeros(1, np.int64),
                                completion=pool.completion[:0], prefix_score=pool.prefix_score[:0])
    go = np.zeros(40, np.int64)
    say("group step, 39 empty groups and no trajectories")
    group_step_parity(pace, empty, go, 39, 20)


@pytest.mark.parametrize("occ,cap", [(10, 20), (64, 0), (64, 63)])
def test_group_step_budget_edges(pace, occ, cap):
    pool = poolgen.make_pool("tiny")
    go = np.arange(0, pool.n + 1, 1, dtype=np.int64)
    say("group budget edges occ=%d cap=%d" % (occ, cap))
    group_step_parity(pace, pool, go, occ, cap)


def test_group_score_and_expand_random(pace):
    rng = np.random.default_rng(23)
    for trial in range(30):
        n = int(rng.integers(0, 3000))
        go = random_groups(rng, n, max_size=int(rng.integers(1, 300)), trailing_empty=bool(trial % 2))
        s = rng.normal(10.0, 5.0, n) * rng.choice([1.0, 1e-6, 1e5])
        say("group score/expand trial %d n=%d groups=%d" % (trial, n, len(go) - 1))
        g = H(pace.pace_group_score(D(s), D(go)))
        assert np.array_equal(g.view(np.uint64), oracle.group_score(s, go).view(np.uint64))
        gk = (rng.random(len(go) - 1) < 0.5).astype(np.uint8)
        k = H(pace.pace_group_expand(D(go), D(gk), n))
        assert np.array_equal(k, oracle.group_expand(go, gk, n))


def test_validate_groups(pace):
    for go, n, bad in (([0, 3, 5], 5, False), ([0, 0, 5, 5], 5, False), ([1, 3, 5], 5, True),
                       ([0, 3, 4], 5, True), ([0, 4, 3, 5], 5, True), ([0], 0, False)):
        say("validate groups %s n=%d" % (go, n))
        e = int(H(pace.pace_validate_groups(D(np.array(go, np.int64)), n))[0])
        assert (e == pace.BAD_GROUPS) == bad and e in (0, pace.BAD_GROUPS)
