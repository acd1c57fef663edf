"""GPU parity of the streaming admission rule (Sec. 3.1, Algorithm 1): the
HIP kernel through the C ABI against the CPU oracle, step by step, with
both sides carrying their own window state. Everything is bit-exact: the
statuses, reject ids, counts, the cutoff, and the window ring itself."""
import copy
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


def gpu_window(pace, ow):
    w = pace.StreamWindow(ow.cap, DEV)
    w.ring.copy_(D(ow.ring))
    w.state.copy_(D(np.array([ow.head, ow.count], np.int64)))
    return w


def check_step(pace, s, r_hat, ow, gw, B, r_max=0.9, window_min=32):
    params = pace.default_params(r_max=r_max, window_min=window_min)
    st, keep, rej, kappa, counts = pace.pace_stream_admit(D(s), r_hat, gw, B, params)
    torch.cuda.synchronize()
    ost, okappa, odrawn, okept = oracle.stream_admit(s, r_hat, ow, B, r_max=r_max, window_min=window_min)
    c = H(counts)
    assert (int(c[0]), int(c[1]), int(c[2])) == (odrawn, okept, odrawn - okept)
    assert np.array_equal(H(st), ost)
    assert np.array_equal(H(keep), (ost == 1).astype(np.uint8))
    assert np.array_equal(H(rej)[: odrawn - okept], np.flatnonzero(ost == 0))
    k = float(H(kappa)[0])
    assert k == okappa
    assert np.array_equal(H(gw.ring).view(np.uint64), ow.ring.view(np.uint64))
    assert list(H(gw.state)) == [ow.head, ow.count]
    return ost, okappa


def test_stream_single_steps_random(pace):
    rng = np.random.default_rng(41)
    for trial in range(60):
        cap = int(rng.choice([1, 2, 37, 512, 1024]))
        ow = oracle.StreamWindow(cap)
        fill = rng.normal(5.0, 2.0, int(rng.integers(0, 3 * cap))).round(int(rng.integers(0, 3)))
        for v in fill:
            ow.ring[ow.head] = v
            ow.head = (ow.head + 1) % cap
            ow.count = min(cap, ow.count + 1)
        gw = gpu_window(pace, ow)
        n = int(rng.choice([0, 1, 100, 4096, 8191, 8192, 8193, 20000]))
        s = rng.normal(5.0, 2.0, n).round(int(rng.integers(0, 3)))
        B = int(rng.integers(0, n + 10))
        r_hat = float(rng.choice([0.0, 0.25, 0.5, 0.9, 0.99, rng.random()]))
        wmin = int(rng.choice([0, 1, 32, 600]))
        say("stream single step trial %d cap=%d count=%d n=%d B=%d r_hat=%.3f wmin=%d"
            % (trial, cap, ow.count, n, B, r_hat, wmin))
        check_step(pace, s, r_hat, ow, gw, B, window_min=wmin)


def test_stream_sweep_math_pool(pace):
    """40 steps of a back-to-back sweep: pool slots refreshed each step, the
    budget's EMA (beta 0.9) carried by each side, the window evolving."""
    pool = copy.deepcopy(poolgen.make_pool("math"))
    V0 = pool.V
    B = 256
    ow = oracle.StreamWindow(512)
    gw = pace.StreamWindow(512, DEV)
    params = pace.default_params(beta=0.9)
    rh_o = rh_g = 0.0
    tags, off, comp, pre, win = D(pool.tags), D(pool.offsets), D(pool.completion), D(pool.prefix_score), D(pool.window)
    for step in range(40):
        slots = poolgen.sweep_step(pool, step, V0)
        for i in slots:
            lo, hi = int(pool.offsets[i]), int(pool.offsets[i + 1])
            tags[lo:hi] = D(pool.tags[lo:hi])
        comp.copy_(D(pool.completion))
        pre.copy_(D(pool.prefix_score))
        sc, _, _ = pace.pace_score(tags, off, comp, pool.V, pre, win, params)
        osc, _, _ = oracle.score(pool.tags, pool.offsets, pool.completion, pool.V, pool.prefix_score, pool.window)
        assert np.array_equal(H(sc).view(np.uint64), osc.view(np.uint64))
        _, rh_g = pace.pace_budget(pool.occupancy, pool.capacity, params, rh_g)
        _, rh_o = oracle.budget(pool.occupancy, pool.capacity, rh_o, 0.9, 0.9)
        assert rh_g == rh_o
        say("stream sweep step %d r_hat=%.4f window=%d" % (step, rh_o, ow.count))
        ost, okappa = check_step(pace, osc, rh_o, ow, gw, B)
        if step > 2:
            assert okappa < np.inf


def test_stream_step_fused_matches_oracle(pace):
    """pace_stream_step over 12 sweep steps of the math pool against the
    oracle's score, budget, stream_admit and compact in sequence."""
    pool = copy.deepcopy(poolgen.make_pool("math"))
    V0 = pool.V
    B = 200
    ow = oracle.StreamWindow(512)
    gw = pace.StreamWindow(512, DEV)
    params = pace.default_params(beta=0.9, window_min=16)
    rh_o = rh_g = 0.0
    tags, off, comp, pre, win = D(pool.tags), D(pool.offsets), D(pool.completion), D(pool.prefix_score), D(pool.window)
    bufs = None
    for step in range(12):
        slots = poolgen.sweep_step(pool, step, V0)
        for i in slots:
            lo, hi = int(pool.offsets[i]), int(pool.offsets[i + 1])
            tags[lo:hi] = D(pool.tags[lo:hi])
        comp.copy_(D(pool.completion))
        pre.copy_(D(pool.prefix_score))
        bufs, rh_g = pace.pace_stream_step(tags, off, comp, pool.V, pool.occupancy, pool.capacity, [tags], gw, B,
                                           pre, win, params, rh_g, bufs)
        torch.cuda.synchronize()
        osc, oS, oT = oracle.score(pool.tags, pool.offsets, pool.completion, pool.V, pool.prefix_score, pool.window)
        _, rh_o = oracle.budget(pool.occupancy, pool.capacity, rh_o, 0.9, 0.9)
        ost, okappa, odrawn, okept = oracle.stream_admit(osc, rh_o, ow, B, window_min=16)
        ooff, oids, opacked = oracle.compact(pool.offsets, (ost == 1).astype(np.uint8), [pool.tags])
        say("stream step fused, sweep step %d drawn=%d kept=%d" % (step, odrawn, okept))
        assert rh_g == rh_o
        assert np.array_equal(H(bufs["score"])[: pool.n].view(np.uint64), osc.view(np.uint64))
        assert np.array_equal(H(bufs["status"])[: pool.n], ost)
        assert float(H(bufs["kappa"])[0]) == okappa
        assert list(H(bufs["counts"])) == [odrawn, okept, odrawn - okept]
        assert np.array_equal(H(gw.ring).view(np.uint64), ow.ring.view(np.uint64))
        nk = int(H(bufs["n_kept_tokens"])[0])
        assert np.array_equal(H(bufs["offsets_out"])[: okept + 1], ooff)
        assert np.array_equal(H(bufs["kept_ids"])[:okept], oids)
        assert np.array_equal(H(bufs["cols_out"][0])[:nk], opacked[0])


@pytest.mark.parametrize("n", [0, 1, 17, 1000, 8192, 8193, 9000])
def test_stream_step_fused_shapes(pace, n):
    """pace_stream_step on ragged pools: partial 16-trajectory blocks and
    partial waves of the draw, empty and multi-piece (> 16384-token)
    trajectories, both sides of the piece-compaction limit (8192
    trajectories), two steps so that the second draws against a filled
    window; every output against the oracle's chain."""
    rng = np.random.default_rng(700 + n)
    V = 50
    lens = rng.integers(0, 40, n).astype(np.int64)
    lens[rng.random(n) < 0.1] = 0
    if n >= 17:
        lens[rng.integers(0, n, 2)] = [20000, 40000]
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    comp = rng.integers(V - 8, V + 1, n).astype(np.int32)
    owner = np.repeat(np.arange(n), lens)
    tags = np.maximum(comp[owner].astype(np.int64) - rng.integers(0, 12, owner.size), 0).astype(np.int32)
    tags[rng.random(owner.size) < 0.1] = -1
    occupancy, capacity = n, max(1, n // 3)
    B = int(rng.integers(1, n + 2))
    ow = oracle.StreamWindow(256)
    gw = pace.StreamWindow(256, DEV)
    params = pace.default_params(window_min=4)
    rh_o = rh_g = 0.0
    bufs = None
    for step in range(2):
        say("stream step fused shapes n=%d step=%d B=%d tokens=%d" % (n, step, B, int(off[-1])))
        bufs, rh_g = pace.pace_stream_step(D(tags), D(off), D(comp), V, occupancy, capacity, [D(tags)], gw, B,
                                           params=params, r_hat_prev=rh_g, buffers=bufs)
        torch.cuda.synchronize()
        osc, _, _ = oracle.score(tags, off, comp, V)
        _, rh_o = oracle.budget(occupancy, capacity, rh_o, 0.0, 0.9)
        ost, okappa, odrawn, okept = oracle.stream_admit(osc, rh_o, ow, B, window_min=4)
        ooff, oids, opacked = oracle.compact(off, (ost == 1).astype(np.uint8), [tags])
        assert rh_g == rh_o
        assert np.array_equal(H(bufs["score"])[:n].view(np.uint64), osc.view(np.uint64))
        assert np.array_equal(H(bufs["status"])[:n], ost)
        assert float(H(bufs["kappa"])[0]) == okappa
        assert list(H(bufs["counts"])) == [odrawn, okept, odrawn - okept]
        assert np.array_equal(H(gw.ring).view(np.uint64), ow.ring.view(np.uint64))
        nk = int(H(bufs["n_kept_tokens"])[0])
        assert nk == int(ooff[-1])
        assert np.array_equal(H(bufs["offsets_out"])[: okept + 1], ooff)
        assert np.array_equal(H(bufs["kept_ids"])[:okept], oids)
        assert np.array_equal(H(bufs["cols_out"][0])[:nk], opacked[0])


def test_stream_admit_unaligned_scores(pace):
    """A score array that is not 16-byte aligned takes the draw's element
    loads; same results as the oracle across ragged pool sizes."""
    rng = np.random.default_rng(77)
    for n in (1, 511, 513, 4096, 8193):
        s = rng.normal(5.0, 2.0, n).round(1)
        big = torch.empty(n + 1, dtype=torch.float64, device=DEV)
        big[1:] = D(s)
        sv = big[1:]
        assert sv.data_ptr() % 16 != 0
        ow = oracle.StreamWindow(128)
        gw = pace.StreamWindow(128, DEV)
        B = int(rng.integers(1, n + 2))
        for step in range(2):
            say("stream admit unaligned n=%d step=%d B=%d" % (n, step, B))
            params = pace.default_params(window_min=4)
            st, keep, rej, kappa, counts = pace.pace_stream_admit(sv, 0.5, gw, B, params)
            torch.cuda.synchronize()
            ost, okappa, odrawn, okept = oracle.stream_admit(s, 0.5, ow, B, window_min=4)
            assert np.array_equal(H(st), ost)
            assert float(H(kappa)[0]) == okappa
            assert list(H(counts)) == [odrawn, okept, odrawn - okept]
            assert np.array_equal(H(gw.ring).view(np.uint64), ow.ring.view(np.uint64))


def test_stream_sweep_stress_pool(pace):
    """The benchmark's streaming sweep configuration on the full stress pool:
    batch ceil(capacity / 3), a 512-entry window, beta 0.9, effective scores
    with prefix scores; six sweep steps (5% of slots refreshed per step), every
    output against the oracle's chain."""
    pool = copy.deepcopy(poolgen.make_pool("stress"))
    V0 = pool.V
    B = -(-pool.capacity // 3)
    ow = oracle.StreamWindow(512)
    gw = pace.StreamWindow(512, DEV)
    params = pace.default_params(beta=0.9)
    rh_o = rh_g = 0.0
    tags, off, comp, pre, win = D(pool.tags), D(pool.offsets), D(pool.completion), D(pool.prefix_score), D(pool.window)
    bufs = None
    for step in range(6):
        slots = poolgen.sweep_step(pool, step, V0)
        for i in slots:
            lo, hi = int(pool.offsets[i]), int(pool.offsets[i + 1])
            tags[lo:hi] = D(pool.tags[lo:hi])
        comp.copy_(D(pool.completion))
        pre.copy_(D(pool.prefix_score))
        bufs, rh_g = pace.pace_stream_step(tags, off, comp, pool.V, pool.occupancy, pool.capacity, [tags], gw, B,
                                           pre, win, params, rh_g, bufs)
        torch.cuda.synchronize()
        osc, _, _ = oracle.score(pool.tags, pool.offsets, pool.completion, pool.V, pool.prefix_score, pool.window)
        _, rh_o = oracle.budget(pool.occupancy, pool.capacity, rh_o, 0.9, 0.9)
        ost, okappa, odrawn, okept = oracle.stream_admit(osc, rh_o, ow, B, window_min=32)
        ooff, oids, opacked = oracle.compact(pool.offsets, (ost == 1).astype(np.uint8), [pool.tags])
        say("stream sweep stress step %d drawn=%d kept=%d kappa=%r" % (step, odrawn, okept, okappa))
        assert rh_g == rh_o
        assert np.array_equal(H(bufs["score"])[: pool.n].view(np.uint64), osc.view(np.uint64))
        assert np.array_equal(H(bufs["status"])[: pool.n], ost)
        assert float(H(bufs["kappa"])[0]) == okappa
        assert list(H(bufs["counts"])) == [odrawn, okept, odrawn - okept]
        assert np.array_equal(H(gw.ring).view(np.uint64), ow.ring.view(np.uint64))
        nk = int(H(bufs["n_kept_tokens"])[0])
        assert nk == int(ooff[-1])
        assert np.array_equal(H(bufs["offsets_out"])[: okept + 1], ooff)
        assert np.array_equal(H(bufs["kept_ids"])[:okept], oids)
        assert np.array_equal(H(bufs["cols_out"][0])[:nk], opacked[0])
