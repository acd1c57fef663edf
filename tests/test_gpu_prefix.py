"""GPU parity of the Prefix Forgetting Score (Eq. (5)): the HIP kernel
through the C ABI against the CPU oracle. The GPU adds the terms in a tree,
the oracle in token order, so values agree within a relative
(cap + 2) * 2^-53 (asserted as 1e-12 relative, the stated tolerance, and the
arithmetic bound); which prefixes have no score (NaN) must match exactly, and
repeated runs are bit-identical."""
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


def compare(pace, a, b, po, tags, cap, min_tokens):
    g = H(pace.pace_prefix_score(D(a), D(b), D(po), None if tags is None else D(tags), cap, min_tokens))
    o = oracle.prefix_score(a, b, po, tags, cap, min_tokens)
    assert np.array_equal(np.isnan(g), np.isnan(o))
    ok = ~np.isnan(o)
    bound = np.maximum((cap + 2) * 2.0 ** -53, 0.0) * np.abs(o[ok])
    assert np.all(np.abs(g[ok] - o[ok]) <= np.maximum(bound, 1e-12 * np.abs(o[ok])))
    assert np.all(np.abs(g[ok] - o[ok]) <= 1e-12 * np.abs(o[ok]))
    g2 = H(pace.pace_prefix_score(D(a), D(b), D(po), None if tags is None else D(tags), cap, min_tokens))
    assert np.array_equal(g.view(np.uint64), g2.view(np.uint64))
    return g, o


@pytest.mark.parametrize("name", ["stress", "multiturn", "long"])
def test_prefix_pools(pace, name):
    pool = poolgen.make_pool(name)
    ids, po, a, b, tags = poolgen.make_prefixes(pool, seed=1)
    for cap in (1024, 2048):
        say("prefix score %s pool: %d prefixes, %d tokens, cap %d" % (name, len(ids), po[-1], cap))
        compare(pace, a, b, po, tags, cap, 32)


def test_prefix_random_shapes(pace):
    rng = np.random.default_rng(61)
    for trial in range(30):
        n = int(rng.choice([0, 1, 5, 100, 5000]))
        lens = rng.choice([0, 1, 31, 32, 33, 255, 256, 257, 1023, 1024, 1025, 3000, 20000], n)
        po = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        m = int(po[-1])
        a = rng.normal(-2, 1, m).astype(np.float32)
        b = (a + rng.normal(0, rng.choice([0.0, 1e-4, 0.1, 3.0]), m)).astype(np.float32)
        tags = None
        if rng.random() < 0.6:
            tags = rng.integers(0, 100, m).astype(np.int32)
            tags[rng.random(m) < rng.choice([0.0, 0.3, 0.95])] = -1
        cap = int(rng.choice([0, 1, 32, 1024, 2048, 100000]))
        mt = int(rng.choice([0, 1, 32, 500]))
        say("prefix random trial %d n=%d tokens=%d cap=%d min=%d tags=%s" % (trial, n, m, cap, mt, tags is not None))
        compare(pace, a, b, po, tags, cap, mt)


def test_prefix_feeds_score(pace):
    """Prefix scores from the GPU drive pace_score's prefix weight; the
    oracle's score given the oracle's prefix scores must agree bit for bit
    wherever both sides agree on the prefix score bit for bit."""
    pool = poolgen.make_pool("stress")
    ids, po, a, b, tags = poolgen.make_prefixes(pool, seed=2)
    g = H(pace.pace_prefix_score(D(a), D(b), D(po), D(tags), 1024, 32))
    o = oracle.prefix_score(a, b, po, tags, 1024, 32)
    s_pre_g = np.full(pool.n, np.nan)
    s_pre_g[ids] = g
    s_pre_o = np.full(pool.n, np.nan)
    s_pre_o[ids] = o
    say("prefix -> score on the stress pool, %d prefixes" % len(ids))
    sc, _, _ = pace.pace_score(D(pool.tags), D(pool.offsets), D(pool.completion), pool.V, D(s_pre_g), D(pool.window))
    osc, _, _ = oracle.score(pool.tags, pool.offsets, pool.completion, pool.V, s_pre_g, pool.window)
    assert np.array_equal(H(sc).view(np.uint64), osc.view(np.uint64))
    same = np.array_equal(np.isnan(s_pre_g), np.isnan(s_pre_o))
    assert same
