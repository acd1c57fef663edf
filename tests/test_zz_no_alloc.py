"""pace_filter_step_noalloc, the filter step for callers that cannot allocate
device memory, against pace_filter_step with a caller workspace: two calls in
a row through the C ABI, the second on a smaller pool (the fixed scratch
keeps the first call's contents), every output bit for bit."""
import sys

import numpy as np
import pytest

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


def _inputs(name):
    pool = poolgen.make_pool(name)
    return pool, dict(tags=D(pool.tags), offsets=D(pool.offsets), completion=D(pool.completion),
                      prefix_score=D(pool.prefix_score), window_sorted=D(pool.window))


def _outputs(pool):
    n, nt = pool.n, pool.n_tokens
    def e(k, dt):   # poisoned, so a missing write shows
        fill = float("nan") if dt == torch.float64 else 0x5A
        return torch.full((k,), fill, dtype=dt, device=DEV)
    return dict(score_out=e(n, torch.float64), gen_sum_out=e(n, torch.int64), gen_count_out=e(n, torch.int64),
                keep_out=e(n, torch.uint8), reject_ids_out=e(n, torch.int32), cols_out=[e(nt, torch.int32)],
                offsets_out=e(n + 1, torch.int64), kept_ids_out=e(n, torch.int32), n_kept_tokens_out=e(1, torch.int64))


def _step(pace, fn, pool, x, out):
    return fn(x["tags"], x["offsets"], x["completion"], pool.V, pool.occupancy, pool.capacity, [x["tags"]],
              prefix_score=x["prefix_score"], window_sorted=x["window_sorted"], r_hat_prev=0.0, **out)


def _same(pool, r, o, r_ref, o_ref):
    n = pool.n
    b = r["budget"]
    assert b == r_ref["budget"] and r["r_hat"] == r_ref["r_hat"]
    nk = n - b
    nkt = int(o["n_kept_tokens_out"].item())
    assert nkt == int(o_ref["n_kept_tokens_out"].item())
    for key in ("score_out", "gen_sum_out", "gen_count_out", "keep_out"):
        assert torch.equal(o[key][:n], o_ref[key][:n]), key
    assert torch.equal(o["reject_ids_out"][:b], o_ref["reject_ids_out"][:b])
    assert torch.equal(o["offsets_out"][:nk + 1], o_ref["offsets_out"][:nk + 1])
    assert torch.equal(o["kept_ids_out"][:nk], o_ref["kept_ids_out"][:nk])
    assert torch.equal(o["cols_out"][0][:nkt], o_ref["cols_out"][0][:nkt])


def test_noalloc_matches_filter_step_on_two_calls(pace):
    pools = [_inputs("stress"), _inputs("tiny")]          # the second call is smaller
    refs = []
    for pool, x in pools:
        say("reference pace_filter_step: %d trajectories, %d tokens" % (pool.n, pool.n_tokens))
        o = _outputs(pool)
        refs.append((_step(pace, pace.pace_filter_step, pool, x, o), o))
    torch.cuda.synchronize()
    got = []
    for pool, x in pools:
        say("pace_filter_step_noalloc: %d trajectories, %d tokens" % (pool.n, pool.n_tokens))
        o = _outputs(pool)
        got.append((_step(pace, pace.pace_filter_step_noalloc, pool, x, o), o))
    torch.cuda.synchronize()
    for (pool, _), (r, o), (rr, oo) in zip(pools, got, refs):
        _same(pool, r, o, rr, oo)


def test_noalloc_refuses_a_pool_beyond_the_scratch(pace):
    pool, x = _inputs("tiny")
    say("pace_filter_step_noalloc beyond the scratch limit (host check)")
    need = pace.pace_workspace_bytes(pace.WS_FILTER_STEP, 1 << 22, pool.n_tokens)
    assert need > pace.NOALLOC_SCRATCH_BYTES
    off = torch.zeros((1 << 22) + 1, dtype=torch.int64, device=DEV)
    comp = torch.zeros(1 << 22, dtype=torch.int32, device=DEV)
    with pytest.raises(pace.PaceError) as e:
        pace.pace_filter_step_noalloc(x["tags"], off, comp, pool.V, 10, 5, [x["tags"]])
    assert e.value.code == pace.ERR_SCRATCH_LIMIT
