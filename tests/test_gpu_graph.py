"""The whole filter step (pace_filter_step with preallocated buffers) captured
in a HIP graph: the library allocates nothing, synchronises nothing and clears
nothing with memset, so the step records as plain kernel nodes. Each replay,
with the program's own eager work between replays, must give the eager
results bit for bit (and those match the oracle)."""
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


def outputs(step, n, n_tokens):
    return [step.score[:n], step.gen_sum[:n], step.gen_count[:n], step.keep[:n], step.reject_ids,
            step.offsets_out, step.kept_ids, step.n_kept_tokens, step.cols_out[0][:n_tokens]]


@pytest.mark.parametrize("name", ["math", "multiturn"])
def test_filter_step_graph_replays(pace, name):
    pool = poolgen.make_pool(name)
    tags, off, comp = D(pool.tags), D(pool.offsets), D(pool.completion)
    prefix, window = D(pool.prefix_score), D(pool.window)
    step = pace.FilterStep(pool.n, pool.n_tokens, [torch.int32], DEV)

    def run():
        step.r_hat = 0.0
        step.run(tags, off, comp, pool.V, pool.occupancy, pool.capacity, [tags], prefix, window)

    run()
    torch.cuda.synchronize()
    budget = step.budget
    ref = [t.clone() for t in outputs(step, pool.n, pool.n_tokens)]
    o = oracle.filter_step(pool, mode="effective", cols=[pool.tags])
    assert budget == o["budget"]
    assert np.array_equal(ref[0].cpu().numpy().view(np.uint64), o["score"].view(np.uint64))
    nk = int(ref[7].item())
    assert nk == o["n_kept_tokens"]
    assert np.array_equal(ref[8][:nk].cpu().numpy(), o["packed"][0])

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    say("%s: captured the step (budget %d); replaying" % (name, budget))
    for rep in range(3):
        for t in outputs(step, pool.n, pool.n_tokens):   # eager work between replays
            t.fill_(7 if t.dtype != torch.float64 else -1.5)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = outputs(step, pool.n, pool.n_tokens)
        for k, (a, b) in enumerate(zip(got, ref)):
            if k == 4:                                    # reject ids: the first `budget` entries
                a, b = a[:budget], b[:budget]
            if k in (5, 6):                               # packed offsets and ids: the kept entries
                kept = int((ref[3] != 0).sum().item())
                a, b = a[: kept + (1 if k == 5 else 0)], b[: kept + (1 if k == 5 else 0)]
            if k == 8:
                a, b = a[:nk], b[:nk]
            assert torch.equal(a, b), "replay %d output %d differs" % (rep, k)
        say("%s: replay %d matches the eager step" % (name, rep))
