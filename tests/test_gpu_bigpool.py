"""A pool past the 32-bit token range: 2^31 + 2^28 int32 version tags
(9.7 GB), through pace_filter_step and through the four separate calls,
against the oracle. Every token position, span start and packed offset above
2^31 goes through the library's 64-bit paths; the span boundaries include one
exactly at 2^31.

The pool: 200 long trajectories of ~12M tokens, each three constant-version
segments 43-45 versions behind its completion and a 1000-token masked (tool,
tag -1) span, and 100 short ones (1000-4000 tokens, current tags) plus an
empty one, shuffled. Raw Staleness (no prefix weight), occupancy 301, target
101: the budget rejects exactly the 200 long trajectories, so the packed
batch is small enough to compare element by element."""
import sys

import numpy as np
import pytest

import oracle

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu, pytest.mark.slow]
DEV = "cuda:0"
N_TOKENS = (1 << 31) + (1 << 28)


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


def big_pool(seed=7):
    rng = np.random.default_rng(seed)
    V = 5000
    n_long, n_short = 200, 100
    short_len = rng.integers(1000, 4001, n_short)
    kinds = np.array(["L"] * n_long + ["S"] * n_short + ["E"])
    rng.shuffle(kinds)
    # The 178th long trajectory in pool order starts exactly at token 2^31:
    # the 177 long ones before it share 2^31 minus the short tokens before it,
    # the 23 from it on share the remaining 2^28 minus the short tokens after
    # it (equal shares with a +-20% jitter, fixed up to the exact totals).
    long_idx = np.flatnonzero(kinds == "L")
    cut = int(long_idx[n_long - 23])
    lens = np.zeros(len(kinds), np.int64)
    lens[kinds == "S"] = short_len
    for idx, total in ((long_idx[:n_long - 23], (1 << 31) - int(lens[:cut].sum())),
                       (long_idx[n_long - 23:], N_TOKENS - (1 << 31) - int(lens[cut:].sum()))):
        w = rng.uniform(0.8, 1.2, len(idx))
        ll = np.floor(w / w.sum() * total).astype(np.int64)
        ll[-1] += total - int(ll.sum())
        lens[idx] = ll
    assert lens[long_idx].min() > 4000
    offsets = np.zeros(len(kinds) + 1, np.int64)
    np.cumsum(lens, out=offsets[1:])
    assert offsets[cut] == (1 << 31)
    completion = (V - rng.integers(0, 9, len(kinds))).astype(np.int32)
    tags = np.empty(N_TOKENS, np.int32)
    for i, kind in enumerate(kinds):
        c, o, L = int(completion[i]), int(offsets[i]), int(lens[i])
        if kind == "L":
            a, b = sorted(int(x) for x in rng.integers(1, L - 1000, 2))
            tags[o:o + a] = c - 45
            tags[o + a:o + a + 1000] = -1
            tags[o + a + 1000:o + b + 1000] = c - 44
            tags[o + b + 1000:o + L] = c - 43
        elif kind == "S":
            tags[o:o + L] = c
    assert N_TOKENS == int(offsets[-1])
    return dict(tags=tags, offsets=offsets, completion=completion, V=V, occupancy=len(kinds),
                capacity=len(kinds) - n_long, n=len(kinds), kinds=kinds)


def test_filter_step_past_2_31_tokens(pace):
    say("building the %d-token pool" % N_TOKENS)
    p = big_pool()
    n = p["n"]
    offs = p["offsets"]
    assert (offs > (1 << 31)).sum() > 20
    say("oracle step (single thread)")
    sc, S, T = oracle.score(p["tags"], offs, p["completion"], p["V"])
    b, _ = oracle.budget(p["occupancy"], p["capacity"])
    keep, rej = oracle.select(sc, b)
    assert b == 200 and np.array_equal(np.sort(rej), np.flatnonzero(p["kinds"] == "L"))
    # closed form (Eq. (1), Lemma 1): S = sum over segments of length x (c - v)
    for i in np.flatnonzero(p["kinds"] != "L")[:5]:
        assert S[i] == 0 and T[i] == offs[i + 1] - offs[i]
    kept = np.flatnonzero(keep)
    off_out = np.concatenate([[0], np.cumsum(offs[kept + 1] - offs[kept])])
    packed = np.concatenate([p["tags"][offs[i]:offs[i + 1]] for i in kept])

    say("uploading %.1f GB of tags" % (p["tags"].nbytes / 1e9))
    D = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(DEV)
    tags, off, comp = D(p["tags"]), D(offs), D(p["completion"])

    def check(name, score, gS, gT, gkeep, grej, goff, gids, gnkt, gcol):
        say("checking %s" % name)
        assert np.array_equal(gS[:n].cpu().numpy(), S), name
        assert np.array_equal(gT[:n].cpu().numpy(), T), name
        assert np.array_equal(score[:n].cpu().numpy().view(np.int64), sc.view(np.int64)), name
        assert np.array_equal(gkeep[:n].cpu().numpy(), keep), name
        assert np.array_equal(grej[:b].cpu().numpy(), rej), name
        nk = n - b
        assert np.array_equal(goff[:nk + 1].cpu().numpy(), off_out), name
        assert np.array_equal(gids[:nk].cpu().numpy(), kept.astype(np.int32)), name
        assert int(gnkt.item()) == int(off_out[-1]), name
        assert np.array_equal(gcol[: int(off_out[-1])].cpu().numpy(), packed), name

    say("pace_filter_step")
    r = pace.pace_filter_step(tags, off, comp, p["V"], p["occupancy"], p["capacity"], [tags])
    torch.cuda.synchronize()
    assert r["budget"] == b
    check("pace_filter_step", r["score"], r["gen_sum"], r["gen_count"], r["keep"], r["reject_ids"],
          r["offsets_out"], r["kept_ids"], r["n_kept_tokens"], r["cols_out"][0])
    del r
    torch.cuda.empty_cache()

    say("separate calls")
    score, gS, gT = pace.pace_score(tags, off, comp, p["V"])
    gb, _ = pace.pace_budget(p["occupancy"], p["capacity"])
    assert gb == b
    gkeep, grej = pace.pace_select(score, gb)
    goff, gids, gnkt, gcols = pace.pace_compact(off, gkeep, [tags])
    torch.cuda.synchronize()
    check("separate calls", score, gS, gT, gkeep, grej, goff, gids, gnkt, gcols[0])
