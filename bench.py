"""Benchmark of the PACE pool filter step (score -> budget -> select -> compact)
on one MI355X.

One step is one pass of the whole filter over one pool. The headline workload
is the stress pool: 4096 trajectories, log-normal lengths around 12k tokens up
to 32768 (50.1M int32 version tags), 0-16 version breaks each, V = 5000,
occupancy 3x the target (budget 2731), scored with Effective Staleness (prefix
window of 512, gamma 4), one int32 payload column (the tags) compacted into the
batch. Inputs are resident in HBM before timing. Steps run back to back
between one event pair over rotating copies of the pool, so that every step
starts with its copy out of the L2 and the 256 MB MALL.

The same measurement is repeated for the other pools (tiny, single-turn math,
long reasoning, multi-turn tool use, the stress pool with three payload
columns, and the wide pool: 65536 trajectories of log-normal lengths around
700 tokens, 52.1M tokens, target 21845) under "configs", each with the oracle
timed on the same pool; the
256-step sweep of the exact top-b step (V + 1 and 5% of the slots refreshed
per step, beta 0 and 0.9 with the smoothed rate carried) is under
"topb_sweep".

Prints ONE JSON line. Usage: python bench.py [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import copy
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12          # MI355X HBM3E, bytes/s
METRIC = "pool filter step: tokens/s and trajectories/s, % of HBM peak GB/s"
MALL_EVICT_BYTES = 640 << 20   # touched by the other copies before a copy's turn comes again


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="stress")
    ap.add_argument("--mode", default="effective", choices=["effective", "raw", "gen"])
    ap.add_argument("--cols", type=int, default=1, choices=[1, 3],
                    help="payload columns: 1 = tags; 3 = tags + token ids + fp32 log-probs")
    ap.add_argument("--configs", default="tiny,math,long,multiturn,stress3,wide",
                    help="pools measured besides the headline ('' = none); stress3 = stress with 3 columns")
    ap.add_argument("--topb-steps", type=int, default=256,
                    help="steps of the exact top-b sweep (0 = skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--sweep-steps", type=int, default=256,
                    help="steps of the back-to-back streaming-rule sweep (0 = skip)")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the graph, flushed, separate-call, group, streaming, prefix and aux legs")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run one plain 256 MiB device copy (counter calibration)")
    return ap.parse_args()


# (timer phase, kernel) of the fused step's launches: pools of up to 8192
# trajectories (rank path), and larger ones (level-0 histogram of the cut
# search, cut-and-classify, merge-path compaction over blocks of 64
# trajectories)
PHASES = ((0, "score_reduce"), (1, "score_finalize"), (2, "rank"), (3, "compact_piece"))
PHASES_WIDE = ((0, "score_reduce"), (1, "score_finalize"), (2, "cut_hist"), (6, "classify"),
               (3, "compact_wide"))


def cpu_model():
    """The host CPU's model name, from /proc/cpuinfo where there is one."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


def reduce_chunks(n_tokens, cus):
    """Token chunks of score_reduce: one per resident wave (CUs x 16),
    256-token aligned, at least 2048 tokens."""
    waves = cus * 16
    chunk = max(2048, -(-(-(-n_tokens // waves)) // 256) * 256)
    return -(-n_tokens // chunk)


def kernel_bytes(pool, n_keep_tok, col_bytes, W, use_prefix, cus):
    """Algorithmic bytes of each kernel of the fused step:
    score_reduce   4 B per tag read, 8 B per offset, 16 B per trajectory
                   (piece sum and count written), 16 B per chunk (carry);
    score_finalize offsets (2 x 8 B), completion 4 B, prefix score 8 B and
                   the window when used, the pieces (16 B per trajectory and
                   per chunk) read; score 8 B, S and T 16 B written (pools
                   above 8192 trajectories: plus the group key extremes,
                   16 B per 128 trajectories);
    rank           score 8 B and span offsets 16 B read, keep flag 1 B and the
                   block partials (16 B per 16 trajectories) written;
    cut_hist       score 8 B read and level-0 digit 2 B written per
                   trajectory, the group extremes read, the 2048-bin
                   histogram (8 KiB) added;
    classify       score 8 B, offsets 16 B and digit 2 B read, keep flag 1 B
                   written per trajectory, the histogram read, the block
                   partials (16 B per 64 trajectories) and their group sums
                   (16 B per 1024 trajectories) written;
    compact_piece  every kept element of each column read and written, keep
    compact_wide   flags and offsets (17 B per trajectory), the block
                   partials (and, for compact_wide, their group sums) read,
                   packed offsets (8 B) and kept ids (4 B) per kept
                   trajectory and rejected ids (4 B per rejection) written."""
    n, N = pool.n, pool.n_tokens
    chunks = reduce_chunks(N, cus)
    wide = n > 8192
    blk = 64 if wide else 16
    blocks = -(-n // blk)
    groups = -(-n // 128)
    bgroups = -(-n // 1024)
    budget = max(0, pool.occupancy - pool.capacity)
    kept = n - min(budget, n)
    pre = (8 * n + 8 * W) if use_prefix else 0
    return {
        "score_reduce": 4 * N + 8 * (n + 1) + 16 * n + 16 * chunks,
        "score_finalize": 16 * n + 4 * n + pre + 16 * n + 16 * chunks + 8 * n + 16 * n + (16 * groups if wide else 0),
        "rank": 8 * n + 16 * n + n + 16 * blocks,
        "cut_hist": 8 * n + 2 * n + 16 * groups + 8192,
        "classify": 8 * n + 16 * n + 2 * n + n + 8192 + 16 * blocks + 16 * bgroups,
        "compact_wide" if wide else "compact_piece":
            sum(2 * e * n_keep_tok for e in col_bytes) + 17 * n + 16 * blocks
            + (16 * bgroups if wide else 0) + 12 * kept + 8 + 4 * budget,
    }


def alg_bytes(pool, n_keep_tok, col_bytes, W, use_prefix=True):
    """Algorithmic bytes of one step: every tag read once, every kept token of
    each payload column read and written once, plus the per-trajectory arrays
    each call reads or writes (offsets, completion, prefix, score, S, T, keep,
    reject ids, packed offsets, kept ids) and the prefix window."""
    n, N = pool.n, pool.n_tokens
    b = 4 * N + sum(2 * e * n_keep_tok for e in col_bytes)
    pre = (8 * n + 8 * W) if use_prefix else 0
    score_call = n * (8 + 8 + 4 + 8 + 8 + 8) + pre          # offsets x2, completion, score, S, T
    select_call = n * (8 + 1) + 4 * max(0, pool.occupancy - pool.capacity)
    compact_call = n * (8 + 8 + 1 + 8 + 4)                    # offsets x2, keep, offsets_out, kept ids
    return b + score_call + select_call + compact_call


def reduce_traffic(config, cols):
    """HBM bytes per score_reduce launch measured with rocprofv3 counters
    (FETCH_SIZE x 2.0 + WRITE_SIZE x 1.0, the factors a plain device copy of
    known size gives), or None when the kernel's sources have changed since
    the counters were taken or no counters exist for this pool."""
    import hashlib
    h = hashlib.sha256()
    for f in ("score.hip", "score_math.hpp", "device_util.hpp"):
        with open(os.path.join(ROOT, "paper_2609_36830_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    rec = REDUCE_COUNTERS.get(config) if cols == 1 else None
    if rec is None or rec["sha256"] != h.hexdigest():
        return None
    return rec["bytes"]


# config -> {"sha256": digest of the score_reduce sources, "bytes": HBM bytes per launch}
REDUCE_COUNTERS = {
    # profiles/filter_step_hbm_counters.md: FETCH_SIZE 98218.9 KiB, WRITE_SIZE 170.2 KiB
    "stress": {"sha256": "97cdaed24ff7101054241bfed79d2b19a6fa70afd19992b81495cc102254f5b9", "bytes": 201326592},
    # profiles/filter_step_hbm_counters.md: FETCH_SIZE 103516.6 KiB, WRITE_SIZE 1139.1 KiB
    "wide": {"sha256": "97cdaed24ff7101054241bfed79d2b19a6fa70afd19992b81495cc102254f5b9", "bytes": 213168435},
}


def extra_columns(pool, ncols):
    """Host payload columns: the tags, then (3 columns) int32 token ids and fp32
    behaviour log-probs."""
    cols = [pool.tags]
    if ncols == 3:
        rng = np.random.default_rng(1)
        cols += [rng.integers(0, 150000, pool.n_tokens).astype(np.int32),
                 rng.standard_normal(pool.n_tokens).astype(np.float32)]
    return cols


def spin_cycles(k):
    """A device-side spin queued ahead of k steps, long enough for the host to
    enqueue all of them before the device reaches the first."""
    return max(20_000_000, 2_000_000 * k)


class Rotation:
    """R copies of a pool's payload columns (the first is the tags), each with
    its own full-capacity output columns, sharing the small per-trajectory
    inputs and outputs. R is chosen so that the other copies' traffic evicts a
    copy from L2 and the MALL before its turn comes again (at least 3)."""

    def __init__(self, pace, pool, host_cols, mode, dev, params):
        import torch
        self.pace, self.pool, self.dev, self.params = pace, pool, dev, params
        D = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        self.off, self.comp = D(pool.offsets), D(pool.completion)
        self.prefix = None if mode == "raw" else D(pool.prefix_score)
        self.window = None if mode == "raw" else D(pool.window)
        self.W = 0 if self.window is None else self.window.numel()
        base = [D(c) for c in host_cols]
        self.col_bytes = [c.element_size() for c in base]
        n, nt = pool.n, pool.n_tokens
        touched = 4 * nt + 2 * sum(self.col_bytes) * nt // 3 + 1
        self.R = int(min(1024, max(3, -(-MALL_EVICT_BYTES // touched) + 1)))
        self.ins = [base] + [[c.clone() for c in base] for _ in range(self.R - 1)]
        self.outs = [[torch.empty_like(c) for c in base] for _ in range(self.R)]
        e = lambda k, dt: torch.empty(max(k, 1), dtype=dt, device=dev)
        self.score, self.S, self.T = e(n, torch.float64), e(n, torch.int64), e(n, torch.int64)
        self.keep, self.rej = e(n, torch.uint8), e(n, torch.int32)
        self.off_out, self.ids, self.nkt = e(n + 1, torch.int64), e(n, torch.int32), e(1, torch.int64)
        self.ws = e(pace.pace_workspace_bytes(pace.WS_FILTER_STEP, n, nt), torch.uint8)

    def step(self, k, r_hat=0.0, tags=None, comp=None, prefix=None, V=None, cols=None, out_k=None):
        pool = self.pool
        ins = self.ins[k % self.R] if cols is None else cols
        outs = self.outs[(k if out_k is None else out_k) % self.R]
        return self.pace.pace_filter_step(
            ins[0] if tags is None else tags, self.off, self.comp if comp is None else comp,
            pool.V if V is None else V, pool.occupancy, pool.capacity, ins,
            self.prefix if prefix is None else prefix, self.window, self.params, r_hat,
            score_out=self.score, gen_sum_out=self.S, gen_count_out=self.T, keep_out=self.keep,
            reject_ids_out=self.rej, cols_out=outs, offsets_out=self.off_out, kept_ids_out=self.ids,
            n_kept_tokens_out=self.nkt, workspace=self.ws)


def measure_pool(pace, pool, host_cols, mode, K, dev, stream, cus, config_name):
    """Cold rotated steps of pace_filter_step on one pool: K steps back to
    back between one event pair (ms_per_step), then K more with each kernel
    timed by its own events (kernel_us_mean) for the roofline of the
    dominant kernel."""
    import torch
    params = pace.default_params(w_wait=0.0 if mode == "gen" else 1.0)
    rot = Rotation(pace, pool, host_cols, mode, dev, params)
    for k in range(rot.R):                          # untimed pass over every copy
        rot.step(k)
    torch.cuda.synchronize()
    n_keep_tok = int(rot.nkt.item())
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda._sleep(spin_cycles(K))
    ev[0].record(stream)
    t0 = time.perf_counter()
    budget = None
    for k in range(K):
        budget = rot.step(k)["budget"]
    t_enq = time.perf_counter() - t0
    ev[1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev[0].elapsed_time(ev[1]) / K
    assert int(rot.nkt.item()) == n_keep_tok
    # each kernel timed by its own events, same rotation
    phases = PHASES if pool.n <= 8192 else PHASES_WIDE
    kev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in phases]
           for _ in range(K)]
    for pairs in kev:
        for a, b in pairs:
            a.record(stream)
            b.record(stream)
    torch.cuda.synchronize()
    for k in range(K):
        for m, (ph, _) in enumerate(phases):
            pace.pace_time_next_kernel(ph, *kev[k][m])
        rot.step(k)
    torch.cuda.synchronize()
    kus = {name: float(np.mean([kev[k][m][0].elapsed_time(kev[k][m][1]) * 1e3 for k in range(K)]))
           for m, (_, name) in enumerate(phases)}
    B = alg_bytes(pool, n_keep_tok, rot.col_bytes, rot.W, rot.prefix is not None)
    kb = kernel_bytes(pool, n_keep_tok, rot.col_bytes, rot.W, rot.prefix is not None, cus)
    dom = max(kus, key=kus.get)
    t_dom = kus[dom] * 1e-6
    res = {
        "n_traj": pool.n, "n_tokens": pool.n_tokens, "budget": budget, "kept_tokens": n_keep_tok,
        "payload_cols": len(host_cols), "mode": mode,
        "ms_per_step": ms, "tokens_per_s": pool.n_tokens / (ms * 1e-3),
        "trajectories_per_s": pool.n / (ms * 1e-3),
        "alg_bytes_per_step": B, "hbm_frac_of_peak": B / (ms * 1e-3) / HBM_PEAK,
        "kernel_us_mean": kus,
        "roofline": {"kernel": dom, "bound": "hbm", "achieved": kb[dom] / t_dom / 1e9,
                     "peak": HBM_PEAK / 1e9, "unit": "GB/s", "frac": kb[dom] / t_dom / HBM_PEAK,
                     "traffic": reduce_traffic(config_name, len(host_cols)) if dom == "score_reduce" else None,
                     "alg_bytes": kb[dom]},
        "timing": "%d steps back to back between one event pair over %d rotating pool copies, each copy "
                  "evicted from L2 and MALL before its turn; host enqueue %.2f ms of %.2f ms wall"
                  % (K, rot.R, t_enq * 1e3, wall * 1e3),
    }
    return res, rot


def oracle_ms(pool, mode, host_cols, min_steps=5, min_s=1.0):
    """The oracle's whole filter step on the same pool, single-threaded: mean
    ms per step over at least min_steps steps and min_s seconds."""
    import oracle
    reps = 0
    t0 = time.perf_counter()
    while reps < min_steps or time.perf_counter() - t0 < min_s:
        oracle.filter_step(pool, mode=mode, cols=host_cols)
        reps += 1
    return (time.perf_counter() - t0) / reps * 1e3, reps


def topb_sweep(pace, pool0, steps, mode, dev, stream):
    """The exact top-b step swept back to back: step s runs on the pool as it
    stands after s refreshes (current version V0 + s, 5% of the slots
    replaced by freshly completed rollouts, length-preserving), with the
    smoothed rate of Eq. (4) carried from step to step, at beta 0 and 0.9.
    Every step's pool state is staged on the device beforehand as its own
    copy (refresh uploads are not timed), so each step reads tags no other
    step touched since the untimed pass: the sweep is cold. Timed twice: all
    steps between one event pair (ms_per_step), then each step between its
    own events (the p10/p50/p90, which include two event records per step)."""
    import torch
    import poolgen
    pool = copy.deepcopy(pool0)
    V0 = pool.V
    D = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    staged, comps, pres, Vs = [], [], [], []
    prev = D(pool.tags)
    for s in range(steps):
        slots = poolgen.sweep_step(pool, s, V0)
        t = prev.clone()
        runs = np.split(slots, np.flatnonzero(np.diff(slots) != 1) + 1)
        for r in runs:
            lo, hi = int(pool.offsets[r[0]]), int(pool.offsets[r[-1] + 1])
            t[lo:hi].copy_(torch.from_numpy(pool.tags[lo:hi]))
        staged.append(t)
        comps.append(D(pool.completion))
        pres.append(None if mode == "raw" else D(pool.prefix_score))
        Vs.append(pool.V)
        prev = t
    torch.cuda.synchronize()
    out = {"steps": steps, "refresh": "5%% of slots (%d) per step, length-preserving, c = V"
           % max(1, int(round(0.05 * pool.n))), "cold": True,
           "staging": "each step's pool state is its own device copy (%.1f GB staged, untimed)"
           % (steps * pool.n_tokens * 4 / 1e9)}
    for beta in (0.0, 0.9):
        params = pace.default_params(beta=beta, w_wait=0.0 if mode == "gen" else 1.0)
        rot = Rotation(pace, pool0, [pool0.tags], mode, dev, params)
        rot.ins = rot.ins[:1]

        def run(s, r_hat):
            return rot.step(0, r_hat, tags=staged[s], comp=comps[s], prefix=pres[s], V=Vs[s],
                            cols=[staged[s]], out_k=s % 3)

        r_hat = 0.0
        for s in range(steps):                          # untimed pass
            r_hat = run(s, r_hat)["r_hat"]
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        budgets, kept = [], []
        r_hat = 0.0
        torch.cuda._sleep(spin_cycles(steps))
        ev[0].record(stream)
        t0 = time.perf_counter()
        for s in range(steps):
            r = run(s, r_hat)
            r_hat = r["r_hat"]
            budgets.append(r["budget"])
        t_enq = time.perf_counter() - t0
        ev[1].record(stream)
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / steps
        pev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        r_hat = 0.0
        torch.cuda._sleep(spin_cycles(steps))
        for s in range(steps):
            pev[s][0].record(stream)
            r_hat = run(s, r_hat)["r_hat"]
            pev[s][1].record(stream)
        torch.cuda.synchronize()
        per = np.array([a.elapsed_time(b) for a, b in pev])
        key = "beta_%g" % beta
        out[key] = {
            "ms_per_step": ms, "tokens_per_s": pool0.n_tokens / (ms * 1e-3),
            "trajectories_per_s": pool0.n / (ms * 1e-3),
            "per_step_ms_p10_p50_p90": [float(np.percentile(per, q)) for q in (10, 50, 90)],
            "host_enqueue_ms": t_enq * 1e3,
            "budget_first_last": [budgets[0], budgets[-1]],
            "budget_at_steps_0_1_2_4_8_16_32_64_128_last": [budgets[min(i, steps - 1)]
                                                          for i in (0, 1, 2, 4, 8, 16, 32, 64, 128, steps - 1)],
            "final_r_hat": r_hat,
        }
        del rot
    del staged, comps, pres
    torch.cuda.empty_cache()
    return out


def aux_bench(pace, pool, rot, comp, K, flush, dev, stream):
    """Cold-cache kernel times (own events) of the single-kernel calls that
    follow a step: Stale-k admission (k = 8) and the admission diagnostics
    (64 bins per metric), on the last step's scores and keep flags."""
    import torch
    n = pool.n
    S, T, sc, keep = rot.S[:n], rot.T[:n], rot.score[:n], rot.keep[:n]
    edges = torch.stack([torch.linspace(0, 16, 65, dtype=torch.float64, device=dev)] * 3)
    skeep = torch.empty(n, dtype=torch.uint8, device=dev)
    lag = torch.empty(n, dtype=torch.float64, device=dev)
    hist = torch.empty((3, 2, 66), dtype=torch.int64, device=dev)
    tot = torch.empty((2, 4), dtype=torch.int64, device=dev)
    calls = {
        "stale_k": lambda: pace.pace_stale_k(S, T, comp, pool.V, 8, skeep, lag),
        "diagnostics": lambda: pace.pace_diagnostics(sc, S, T, comp, pool.V, keep, edges, hist, tot),
    }
    res = {}
    for name, fn in calls.items():
        evs = []
        for k in range(K + 2):
            ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
            ev[0].record(stream)
            ev[1].record(stream)
            evs.append(ev)
        torch.cuda.synchronize()
        for k in range(K + 2):
            flush.max()
            pace.pace_time_next_kernel(pace.PHASE_AUX, *evs[k])
            fn()
        torch.cuda.synchronize()
        res[name + "_us_mean"] = float(np.mean([e[0].elapsed_time(e[1]) * 1e3 for e in evs[2:]]))
    res["stale_k_admitted"] = int(skeep.sum().item())
    return res


def prefix_bench(pace, pool, K, flush, dev, stream, cap=1024, min_tokens=32):
    """Prefix Forgetting Score (Eq. (5)) over the pool's synthetic rescored
    prefixes (every trajectory with a version break, its tokens before the
    first break), cold caches, kernel timed by its own events. Algorithmic
    bytes: 12 B (two f32 log-probs and the tag) per token up to each prefix's
    cap-th eligible token, plus 16 B of offsets and 8 B of output per prefix."""
    import torch
    import poolgen
    ids, po, a, b, tg = poolgen.make_prefixes(pool, seed=0)
    n = len(ids)
    read = 0
    for k in range(n):
        elig = np.flatnonzero(tg[po[k]:po[k + 1]] != -1)
        read += int(elig[cap - 1]) + 1 if len(elig) >= cap else int(po[k + 1] - po[k])
    alg = 12 * read + 24 * n
    Dt = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    da, db, dp, dtg = Dt(a), Dt(b), Dt(po), Dt(tg)
    out = torch.empty(max(n, 1), dtype=torch.float64, device=dev)
    evs = []
    for k in range(K + 2):
        ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
        ev[0].record(stream)
        ev[1].record(stream)
        evs.append(ev)
    torch.cuda.synchronize()
    for k in range(K + 2):
        flush.max()
        pace.pace_time_next_kernel(pace.PHASE_PREFIX, *evs[k])
        pace.pace_prefix_score(da, db, dp, dtg, cap, min_tokens, out)
    torch.cuda.synchronize()
    us = np.array([e[0].elapsed_time(e[1]) * 1e3 for e in evs[2:]])
    t = float(us.mean()) * 1e-6
    return {"entry": "pace_prefix_score", "prefixes": n, "prefix_tokens": int(po[-1]), "cap": cap,
            "kernel_us_mean": float(us.mean()), "alg_bytes": alg, "achieved_GBps": alg / t / 1e9,
            "hbm_frac_of_peak": alg / t / HBM_PEAK, "scored": int(np.isfinite(out[:n].cpu().numpy()).sum())}


def stream_sweep(args, pace, pool, rot, dev, stream):
    """Back-to-back sweep with the streaming admission rule (no cache flush):
    per step s the current version is V0 + s and 5% of the slots are refreshed
    as fresh rollouts (host generation and upload outside the events); the
    timed step is one pace_stream_step call: pace_budget (beta 0.9, r_hat
    carried), pace_score, one pace_stream_admit draw of a batch of
    ceil(target / 3) and pace_compact of the retained batch. Runs on copies of
    the pool; warm (the refreshed spans were just uploaded and nothing evicts
    the rest)."""
    import torch
    import poolgen
    spool = copy.deepcopy(pool)
    V0 = spool.V
    stags, scomp = rot.ins[0][0].clone(), rot.comp.clone()
    spre = rot.prefix.clone() if rot.prefix is not None else None
    scols = [stags]
    n, nt = pool.n, pool.n_tokens
    params = pace.default_params(beta=0.9, w_wait=0.0 if args.mode == "gen" else 1.0)
    batch = -(-pool.capacity // 3)
    win = pace.StreamWindow(512, dev)
    bufs = pace.stream_step_buffers(n, nt, [c.dtype for c in scols], dev)
    counts = torch.empty(args.sweep_steps * 3, dtype=torch.int64, device=dev)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.sweep_steps)]
    r_hat = 0.0
    for step in range(args.sweep_steps):
        slots = poolgen.sweep_step(spool, step, V0)
        runs = np.split(slots, np.flatnonzero(np.diff(slots) != 1) + 1)
        for r in runs:
            lo, hi = int(spool.offsets[r[0]]), int(spool.offsets[r[-1] + 1])
            stags[lo:hi].copy_(torch.from_numpy(spool.tags[lo:hi]), non_blocking=False)
        scomp.copy_(torch.from_numpy(spool.completion))
        if spre is not None:
            spre.copy_(torch.from_numpy(spool.prefix_score))
        # keep the device busy (a short spin, no memory traffic) while the host
        # issues the step, so the events time the step's kernels, not the
        # host's call overhead
        torch.cuda._sleep(400000)
        evs[step][0].record(stream)
        _, r_hat = pace.pace_stream_step(stags, rot.off, scomp, spool.V, spool.occupancy, spool.capacity, scols,
                                         win, batch, spre, rot.window, params, r_hat, bufs)
        evs[step][1].record(stream)
        counts[3 * step: 3 * step + 3].copy_(bufs["counts"])
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in evs])
    c = counts.view(-1, 3).cpu().numpy()
    return {
        "entry": "pace_stream_step (budget, score, stream admit, compact), back to back, warm",
        "steps": args.sweep_steps, "batch": batch, "beta": 0.9, "window": 512,
        "ms_per_step": float(ms.mean()), "ms_p10_p50_p90": [float(np.percentile(ms, q)) for q in (10, 50, 90)],
        "tokens_per_s": nt / (float(ms.mean()) * 1e-3),
        "final_r_hat": r_hat,
        "mean_drawn": float(c[:, 0].mean()), "mean_retained": float(c[:, 1].mean()),
        "mean_rejected": float(c[:, 2].mean()), "last_rejected": int(c[-1, 2]),
    }


def headline_extras(args, pace, pool, rot, K, dev, stream):
    """Further views of the headline step: HIP graph replays of the same
    rotation, steps after an explicit 512 MiB cache flush (per-step events),
    the four separate calls, warm steps, the group step, the streaming sweep,
    prefix scores and the auxiliary kernels."""
    import torch
    res = {}
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev).view(torch.int32)
    flush.fill_(1)
    n, nt = pool.n, pool.n_tokens
    n_keep_tok = int(rot.nkt.item())
    # graph replays of the rotation (the budget is fixed at capture; this
    # pool's occupancy does not change)
    graphs = []
    for k in range(rot.R):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            rot.step(k)
        graphs.append(g)
    for k in range(2 * rot.R):
        graphs[k % rot.R].replay()
    gv = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    torch.cuda._sleep(spin_cycles(K))
    gv[0].record(stream)
    for k in range(K):
        graphs[k % rot.R].replay()
    gv[1].record(stream)
    torch.cuda.synchronize()
    res["graph_rotation_ms_per_step"] = gv[0].elapsed_time(gv[1]) / K
    res["graph_timing"] = "the same rotation with each copy's step captured once in a HIP graph and replayed"
    assert int(rot.nkt.item()) == n_keep_tok
    del graphs
    # flushed steps, each bracketed by its own events
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K)]
    for k in range(K):
        flush.max()
        ev[k][0].record(stream)
        rot.step(0)
        ev[k][1].record(stream)
    torch.cuda.synchronize()
    per_step = np.array([e[0].elapsed_time(e[1]) for e in ev])
    res["flushed_ms_per_step"] = float(per_step.mean())
    res["flushed_ms_p10_p50_p90"] = [float(np.percentile(per_step, q)) for q in (10, 50, 90)]
    res["flushed_timing"] = "each step after a 512 MiB cache flush, bracketed by its own event pair"
    # the four separate calls, events around each
    step = pace.FilterStep(n, nt, [c.dtype for c in rot.ins[0]], dev, rot.params)
    cols = rot.ins[0]
    cev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    for k in range(K):
        flush.max()
        cev[k][0].record(stream)
        step.score_only(cols[0], rot.off, rot.comp, pool.V, rot.prefix, rot.window)
        cev[k][1].record(stream)
        step.budget, _ = pace.pace_budget(pool.occupancy, pool.capacity, step.params, 0.0)
        pace.pace_select(step.score[:n], step.budget, step.keep[:n], step.reject_ids, step.ws[1])
        cev[k][2].record(stream)
        pace.pace_compact(rot.off, step.keep[:n], cols, [c[:nt] for c in step.cols_out], step.offsets_out,
                          step.kept_ids, step.n_kept_tokens, step.ws[2], n_tokens=nt)
        cev[k][3].record(stream)
    torch.cuda.synchronize()
    assert int(step.n_kept_tokens.item()) == n_keep_tok
    res["separate_calls_ms_per_step"] = float(np.mean([e[0].elapsed_time(e[3]) for e in cev]))
    res["per_call_ms"] = {"pace_score": float(np.mean([e[0].elapsed_time(e[1]) for e in cev])),
                          "pace_budget+pace_select": float(np.mean([e[1].elapsed_time(e[2]) for e in cev])),
                          "pace_compact": float(np.mean([e[2].elapsed_time(e[3]) for e in cev]))}
    # warm back-to-back steps (no flush, one copy)
    wv = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    torch.cuda._sleep(spin_cycles(K))
    wv[0].record(stream)
    for k in range(K):
        rot.step(0)
    wv[1].record(stream)
    torch.cuda.synchronize()
    res["warm_ms_per_step"] = wv[0].elapsed_time(wv[1]) / K
    # group-level admission: prompt groups of 8, occupancy and target in groups
    go = torch.arange(0, n + 1, 8, dtype=torch.int64, device=dev)
    if int(go[-1]) != n:
        go = torch.cat([go, torch.tensor([n], dtype=torch.int64, device=dev)])
    n_groups = go.numel() - 1
    g_occ, g_cap = n_groups, -(-pool.capacity // 8)
    gws = torch.empty(pace.pace_workspace_bytes(pace.WS_FILTER_STEP, max(n, n_groups), nt),
                      dtype=torch.uint8, device=dev)
    gev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K + 2)]
    gout = pace.group_step_buffers(n, n_groups, cols, dev)
    g_res = None
    for k in range(K + 2):
        flush.max()
        gev[k][0].record(stream)
        g_res = pace.pace_group_filter_step(cols[0], rot.off, rot.comp, pool.V, go, g_occ, g_cap, cols, rot.prefix,
                                            rot.window, rot.params, 0.0, workspace=gws, out=gout)
        gev[k][1].record(stream)
    torch.cuda.synchronize()
    g_ms = np.array([e[0].elapsed_time(e[1]) for e in gev[2:]])
    g_kept_tok = int(g_res["n_kept_tokens"].item())
    res["group_step"] = {
        "entry": "pace_group_filter_step (groups of 8, group mean score), flushed per step",
        "n_groups": n_groups, "occupancy_groups": g_occ, "target_groups": g_cap,
        "budget_groups": g_res["budget"], "kept_tokens": g_kept_tok,
        "ms_per_step": float(g_ms.mean()), "tokens_per_s": nt / (float(g_ms.mean()) * 1e-3),
        "hbm_frac_of_peak": (alg_bytes(pool, g_kept_tok, rot.col_bytes, rot.W, rot.prefix is not None)
                             + n_groups * (8 + 8 + 8 + 1 + 4) + n) / (float(g_ms.mean()) * 1e-3) / HBM_PEAK,
    }
    if args.sweep_steps > 0:
        res["stream_sweep"] = stream_sweep(args, pace, pool, rot, dev, stream)
    res["prefix_score"] = prefix_bench(pace, pool, K, flush, dev, stream)
    res["aux_kernels"] = aux_bench(pace, pool, rot, rot.comp, K, flush, dev, stream)
    del flush
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the filter step has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    import poolgen
    import paper_2609_36830_amd as pace
    from paper_2609_36830_amd import _lib
    if not os.path.exists(_lib.library_path):
        raise SystemExit("libpace.so is not built: run __graft_entry__.build() first")

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    K = args.steps
    t_start = time.perf_counter()

    def log(msg):
        sys.stderr.write("[bench %.1fs] %s\n" % (time.perf_counter() - t_start, msg))
        sys.stderr.flush()

    # ---- headline -------------------------------------------------------------
    pool = poolgen.make_pool(args.config)
    host_cols = extra_columns(pool, args.cols)
    log("headline: %s pool, %d column(s), %s staleness" % (args.config, args.cols, args.mode))
    # warm-up: untimed steps on the pool (library code objects, allocator)
    head, rot = measure_pool(pace, pool, host_cols, args.mode, max(args.warmup, 1), dev, stream, cus, args.config)
    head, rot = measure_pool(pace, pool, host_cols, args.mode, K, dev, stream, cus, args.config)
    ms = head["ms_per_step"]
    out = {
        "metric": METRIC,
        "value": head["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64+f64",
        "data": "synthetic",
        "config": {
            "workload": "%s pool: %d trajectories, %d tokens, V=%d, occupancy %d, target %d, "
                        "%s staleness, %d payload column(s), cold L2/MALL per step"
                        % (args.config, pool.n, pool.n_tokens, pool.V, pool.occupancy,
                           pool.capacity, args.mode, len(host_cols)),
            "n_traj": pool.n, "n_tokens": pool.n_tokens, "budget": head["budget"],
            "kept_tokens": head["kept_tokens"], "mode": args.mode, "payload_cols": len(host_cols),
            "parallelism": "single GPU",
        },
        "trajectories_per_s": head["trajectories_per_s"],
        "hbm_frac_of_peak": head["hbm_frac_of_peak"],
        "alg_bytes_per_step": head["alg_bytes_per_step"],
        "timing": head["timing"],
        "entry": "pace_filter_step (score -> budget -> select -> compact)",
        "kernel_us_mean": head["kernel_us_mean"],
        "roofline": head["roofline"],
    }

    # ---- the other pools ----------------------------------------------------
    configs = {}
    for name in [c for c in args.configs.split(",") if c]:
        base, ncols = (name[:-1], 3) if name.endswith("3") else (name, 1)
        log("config %s" % name)
        p = pool if base == args.config else poolgen.make_pool(base)
        hc = extra_columns(p, ncols)
        r, _ = measure_pool(pace, p, hc, args.mode, K, dev, stream, cus, base)
        if not args.no_cpu_baseline:
            oms, reps = oracle_ms(p, args.mode, hc)
            r["oracle"] = {"ms_per_step": oms, "tokens_per_s": p.n_tokens / (oms * 1e-3),
                           "trajectories_per_s": p.n / (oms * 1e-3), "steps": reps, "cores": 1}
            r["gpu_over_oracle"] = oms / r["ms_per_step"]
        configs[name] = r
        torch.cuda.empty_cache()
    if configs:
        out["configs"] = configs
        out["configs_note"] = ("each pool timed like the headline (cold rotated steps); oracle = the "
                               "single-threaded C oracle's whole step on the same pool, 1 core, on %s"
                               % cpu_model())

    # ---- exact top-b sweep ----------------------------------------------------
    if args.topb_steps > 0:
        log("top-b sweep, %d steps" % args.topb_steps)
        out["topb_sweep"] = topb_sweep(pace, pool, args.topb_steps, args.mode, dev, stream)

    if not args.no_extras:
        log("headline extras")
        out.update(headline_extras(args, pace, pool, rot, K, dev, stream))

    if args.calib_copy:
        a = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        a.fill_(3)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()

    if not args.no_cpu_baseline:
        log("cpu baseline")
        import oracle
        reps = 0
        ts = time.perf_counter()
        while reps < 3 or time.perf_counter() - ts < args.cpu_seconds:
            oracle.filter_step(pool, mode=args.mode, cols=host_cols)
            reps += 1
        t_cpu = time.perf_counter() - ts
        B = head["alg_bytes_per_step"]
        out["cpu_baseline"] = {
            "value": reps * pool.n_tokens / t_cpu, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "trajectories_per_s": reps * pool.n / t_cpu, "GBps": reps * B / t_cpu / 1e9,
            "ms_per_step": t_cpu / reps * 1e3,
            "sample": "%d full oracle filter steps (score, budget, select, compact) on the same "
                      "%s pool, single-threaded C, %.1f s, on %s (%d host threads visible)"
                      % (reps, args.config, t_cpu, cpu_model(), os.cpu_count() or 0),
        }
    out["bench_wall_s"] = time.perf_counter() - t_start
    print(json.dumps(out))


if __name__ == "__main__":
    main()
