"""bench.py's command line on the CPU: more than one GPU is refused with a
message before anything touches a device, and the algorithmic byte counts
follow their stated per-unit terms."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_kernel_bytes_terms():
    import bench
    import poolgen
    pool = poolgen.make_pool("tiny")
    kept_tok, W = 1000, 512
    kb = bench.kernel_bytes(pool, kept_tok, [4], W, True, 256)
    n, N = pool.n, pool.n_tokens
    chunks = bench.reduce_chunks(N, 256)
    assert kb["score_reduce"] == 4 * N + 8 * (n + 1) + 16 * n + 16 * chunks
    budget = max(0, pool.occupancy - pool.capacity)
    kept = n - min(budget, n)
    assert kb["compact_piece"] == 2 * 4 * kept_tok + 17 * n + 16 * (-(-n // 16)) + 12 * kept + 8 + 4 * budget
    # the step's total counts every tag once and the kept tokens twice
    assert bench.alg_bytes(pool, kept_tok, [4], W) >= 4 * N + 8 * kept_tok


def test_reduce_chunks_cover_the_pool():
    import bench
    for N in (0, 1, 2047, 2048, 2049, 50_134_755, 52_107_605):
        c = bench.reduce_chunks(N, 256)
        if N == 0:
            continue
        chunk = max(2048, -(-(-(-N // (256 * 16))) // 256) * 256)
        assert chunk % 256 == 0 and (c - 1) * chunk < N <= c * chunk
    assert np.isclose(bench.HBM_PEAK, 8.0e12)
