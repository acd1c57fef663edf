"""Benchmark of the PACE pool filter step (score -> budget -> select -> compact)
on one MI355X.

One step is one pass of the whole filter over one pool. The workload is the
stress pool: 4096 trajectories, log-normal lengths around 12k tokens up to
32768 (50.1M int32 version tags), 0-16 version breaks each, V = 5000,
occupancy 3x the target (budget 2731), scored with Effective Staleness
(prefix window of 512, gamma 4), one int32 payload column (the tags)
compacted into the batch. Inputs are resident in HBM before timing. The
headline times K steps back to back between one event pair, over three copies
of the pool used in rotation: one step moves more bytes than the 256 MB MALL
holds, so each step starts with its pool copy out of the caches. The same
steps are also timed one by one after an explicit 512 MiB cache flush.

Prints ONE JSON line. Usage: python bench.py [--steps K] [--warmup W]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12          # MI355X HBM3E, bytes/s
METRIC = "pool filter step: tokens/s and trajectories/s, % of HBM peak GB/s"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="stress")
    ap.add_argument("--mode", default="effective", choices=["effective", "raw", "gen"])
    ap.add_argument("--cols", type=int, default=1, choices=[1, 3],
                    help="payload columns: 1 = tags; 3 = tags + token ids + fp32 log-probs")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--sweep-steps", type=int, default=256,
                    help="steps of the back-to-back streaming-rule sweep (0 = skip)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run one plain 256 MiB device copy (counter calibration)")
    return ap.parse_args()


# (timer phase, kernel) of the fused step's launches
PHASES = ((0, "score_reduce"), (1, "score_finalize"), (2, "rank"), (3, "compact_piece"))


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


def reduce_bytes(pool, cus):
    """Algorithmic bytes of one score_reduce launch: 4 B per tag read, 8 B per
    offset read, 16 B per trajectory (piece sum and count written) and 16 B
    per token chunk (carry written); one chunk per resident wave (CUs x 16),
    2048-token aligned."""
    waves = cus * 16
    chunk = max(2048, -(-(-(-pool.n_tokens // waves)) // 2048) * 2048)
    chunks = -(-pool.n_tokens // chunk)
    return 4 * pool.n_tokens + 8 * (pool.n + 1) + 16 * pool.n + 16 * chunks


def reduce_traffic(config):
    """HBM bytes per score_reduce launch measured with rocprofv3 counters
    (FETCH_SIZE x 2.0 + WRITE_SIZE x 1.0, the factors a plain device copy of
    known size gives), or None when the kernel's sources have changed since
    the counters were taken."""
    import hashlib
    h = hashlib.sha256()
    for f in ("score.hip", "score_math.hpp", "device_util.hpp"):
        with open(os.path.join(ROOT, "paper_2609_36830_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    rec = REDUCE_COUNTERS.get(config)
    if rec is None or rec["sha256"] != h.hexdigest():
        return None
    return rec["bytes"]


# config -> {"sha256": digest of the score_reduce sources, "bytes": HBM bytes per launch}
REDUCE_COUNTERS = {
    # profiles/score_reduce_stress_hbm_counters.md: FETCH_SIZE 98152.6 KiB, WRITE_SIZE 175.7 KiB
    "stress": {"sha256": "f08e39fb9827a71d47a05d77e52064ab4794caa43ed46ea0bc13f540b3d8af53", "bytes": 201196442},
}


def aux_bench(pace, pool, step, off, comp, K, flush, dev, stream):
    """Cold-cache kernel times (own events) of the single-kernel calls that
    follow a step: Stale-k admission (k = 8) and the admission diagnostics
    (64 bins per metric), on the last step's scores and keep flags."""
    import torch
    n = pool.n
    S, T, sc, keep = step.gen_sum[:n], step.gen_count[:n], step.score[:n], step.keep[:n]
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


def stream_sweep(args, pace, pool, tags, off, comp, prefix, window, cols, dev, stream):
    """Back-to-back sweep with the streaming admission rule (no cache flush):
    per step s the current version is V0 + s and 5% of the slots are refreshed
    as fresh rollouts (host generation and upload outside the events); the
    timed step is one pace_stream_step call: pace_budget (beta 0.9, r_hat
    carried), pace_score, one pace_stream_admit draw of a batch of
    ceil(target / 3) and pace_compact of the retained batch. Runs on copies of
    the pool."""
    import copy
    import torch
    import poolgen
    spool = copy.deepcopy(pool)
    V0 = spool.V
    stags, scomp = tags.clone(), comp.clone()
    spre = prefix.clone() if prefix is not None else None
    scols = [stags] + list(cols[1:])
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
        lo, hi = int(spool.offsets[slots.min()]), int(spool.offsets[slots.max() + 1])
        if slots.max() - slots.min() + 1 == len(slots):
            stags[lo:hi].copy_(torch.from_numpy(spool.tags[lo:hi]), non_blocking=False)
        else:
            stags.copy_(torch.from_numpy(spool.tags))
        scomp.copy_(torch.from_numpy(spool.completion))
        if spre is not None:
            spre.copy_(torch.from_numpy(spool.prefix_score))
        # keep the device busy (a short spin, no memory traffic) while the host
        # issues the step, so the events time the step's kernels, not the
        # host's call overhead
        torch.cuda._sleep(400000)
        evs[step][0].record(stream)
        _, r_hat = pace.pace_stream_step(stags, off, scomp, spool.V, spool.occupancy, spool.capacity, scols,
                                         win, batch, spre, window, params, r_hat, bufs)
        evs[step][1].record(stream)
        counts[3 * step: 3 * step + 3].copy_(bufs["counts"])
    torch.cuda.synchronize()
    ms = np.array([a.elapsed_time(b) for a, b in evs])
    c = counts.view(-1, 3).cpu().numpy()
    return {
        "entry": "pace_stream_step (budget, score, stream admit, compact), back to back, no flush",
        "steps": args.sweep_steps, "batch": batch, "beta": 0.9, "window": 512,
        "ms_per_step": float(ms.mean()), "ms_p10_p50_p90": [float(np.percentile(ms, q)) for q in (10, 50, 90)],
        "tokens_per_s": nt / (float(ms.mean()) * 1e-3),
        "final_r_hat": r_hat,
        "mean_drawn": float(c[:, 0].mean()), "mean_retained": float(c[:, 1].mean()),
        "mean_rejected": float(c[:, 2].mean()), "last_rejected": int(c[-1, 2]),
    }


def alg_bytes(pool, n_keep_tok, col_bytes, W):
    """Algorithmic bytes of one step: every tag read once, every kept token of
    each payload column read and written once, plus the per-trajectory arrays
    each call reads or writes (offsets, completion, prefix, score, S, T, keep,
    reject ids, packed offsets, kept ids) and the prefix window."""
    n, N = pool.n, pool.n_tokens
    b = 4 * N + sum(2 * e * n_keep_tok for e in col_bytes)
    score_call = n * (8 + 8 + 4 + 8 + 8 + 8 + 8) + 8 * W       # offsets x2, completion, prefix, score, S, T
    select_call = n * (8 + 1) + 4 * (pool.occupancy - pool.capacity)
    compact_call = n * (8 + 8 + 1 + 8 + 4)                      # offsets x2, keep, offsets_out, kept ids
    return b + score_call + select_call + compact_call, 4 * N + score_call


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
        from paper_2609_36830_amd import build
        build.build()

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    pool = poolgen.make_pool(args.config)
    D = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    tags, off, comp = D(pool.tags), D(pool.offsets), D(pool.completion)
    prefix = None if args.mode == "raw" else D(pool.prefix_score)
    window = None if args.mode == "raw" else D(pool.window)
    W = 0 if window is None else window.numel()
    host_cols = [pool.tags]
    if args.cols == 3:
        rng = np.random.default_rng(1)
        host_cols += [rng.integers(0, 150000, pool.n_tokens).astype(np.int32),
                      rng.standard_normal(pool.n_tokens).astype(np.float32)]
    cols = [tags] + [D(c) for c in host_cols[1:]]
    params = pace.default_params(w_wait=0.0 if args.mode == "gen" else 1.0)
    step = pace.FilterStep(pool.n, pool.n_tokens, [c.dtype for c in cols], dev, params)
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev).view(torch.int32)
    flush.fill_(1)
    stream = torch.cuda.current_stream(dev)

    def calls_step(evs=None):
        """The four separate calls (per-call events)."""
        if evs:
            evs[0].record(stream)
        step.score_only(tags, off, comp, pool.V, prefix, window)
        if evs:
            evs[1].record(stream)
        step.budget, _ = pace.pace_budget(pool.occupancy, pool.capacity, step.params, 0.0)
        pace.pace_select(step.score[: pool.n], step.budget, step.keep[: pool.n], step.reject_ids, step.ws[1])
        if evs:
            evs[2].record(stream)
        pace.pace_compact(off, step.keep[: pool.n], cols, [c[: pool.n_tokens] for c in step.cols_out],
                          step.offsets_out, step.kept_ids, step.n_kept_tokens, step.ws[2],
                          n_tokens=pool.n_tokens)
        if evs:
            evs[3].record(stream)

    def fused_step(evs=None):
        """One pace_filter_step call: the whole step in three launches."""
        if evs:
            evs[0].record(stream)
        step.r_hat = 0.0
        step.run(tags, off, comp, pool.V, pool.occupancy, pool.capacity, cols, prefix, window, fused=True)
        if evs:
            evs[1].record(stream)

    for _ in range(args.warmup):
        flush.max()
        fused_step()
        flush.max()
        calls_step()
    torch.cuda.synchronize()

    # Timed region: K cold-cache steps (pace_filter_step), each bracketed by HIP events.
    K = args.steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(K):
        flush.max()
        fused_step(ev[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per_step = np.array([e[0].elapsed_time(e[1]) for e in ev])           # ms
    n_keep_tok = int(step.n_kept_tokens.item())
    budget = step.budget

    # Headline timing: K steps back to back between one pair of events, over
    # R copies of the pool (same content, different addresses) used in
    # rotation. Each step moves ~335 MB, more than the 256 MB MALL, so a copy
    # is evicted by the time its turn comes again: every step starts cold,
    # with no flush kernel and no per-step event inside the timed region. A
    # device spin queued before the first event lets the host enqueue all K
    # steps before the device reaches them.
    R = 3
    rot = [(tags, cols, step)]
    for _r in range(R - 1):
        t2 = tags.clone()
        c2 = [t2] + [c.clone() for c in cols[1:]]
        rot.append((t2, c2, pace.FilterStep(pool.n, pool.n_tokens, [c.dtype for c in c2], dev, params)))
    for k in range(2 * R):                                  # untimed pass
        t_, c_, s_ = rot[k % R]
        s_.r_hat = 0.0
        s_.run(t_, off, comp, pool.V, pool.occupancy, pool.capacity, c_, prefix, window, fused=True)
    rev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    torch.cuda._sleep(20_000_000)
    rev[0].record(stream)
    t_rot = time.perf_counter()
    for k in range(K):
        t_, c_, s_ = rot[k % R]
        s_.r_hat = 0.0
        s_.run(t_, off, comp, pool.V, pool.occupancy, pool.capacity, c_, prefix, window, fused=True)
    t_enq = time.perf_counter() - t_rot
    rev[1].record(stream)
    torch.cuda.synchronize()
    wall_rot = time.perf_counter() - t_rot
    rot_ms = rev[0].elapsed_time(rev[1]) / K
    assert all(int(s_.n_kept_tokens.item()) == n_keep_tok for _, _, s_ in rot)
    # The same rotation as HIP graph replays: each copy's step captured once
    # (the budget is fixed at capture; this pool's occupancy does not change),
    # the K replays back to back between one event pair.
    graphs = []
    for t_, c_, s_ in rot:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            s_.r_hat = 0.0
            s_.run(t_, off, comp, pool.V, pool.occupancy, pool.capacity, c_, prefix, window, fused=True)
        graphs.append(g)
    for k in range(2 * R):
        graphs[k % R].replay()
    gv = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    torch.cuda._sleep(20_000_000)
    gv[0].record(stream)
    for k in range(K):
        graphs[k % R].replay()
    gv[1].record(stream)
    torch.cuda.synchronize()
    graph_ms = gv[0].elapsed_time(gv[1]) / K
    assert all(int(s_.n_kept_tokens.item()) == n_keep_tok for _, _, s_ in rot)
    del graphs
    # the same rotation with each kernel timed by its own events: its reduce
    # time against the flushed one shows whether the steps really start cold
    rk = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in PHASES]
          for _ in range(K)]
    for pairs in rk:
        for a, b in pairs:
            a.record(stream)
            b.record(stream)
    torch.cuda.synchronize()
    for k in range(K):
        t_, c_, s_ = rot[k % R]
        s_.r_hat = 0.0
        for m, (ph, _) in enumerate(PHASES):
            pace.pace_time_next_kernel(ph, *rk[k][m])
        s_.run(t_, off, comp, pool.V, pool.occupancy, pool.capacity, c_, prefix, window, fused=True)
    torch.cuda.synchronize()
    rot_kernel_us = {name: float(np.mean([rk[k][m][0].elapsed_time(rk[k][m][1]) * 1e3 for k in range(K)]))
                     for m, (_, name) in enumerate(PHASES)}
    del rot

    # The same step as four separate calls, for per-call times.
    cev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    for k in range(K):
        flush.max()
        calls_step(cev[k])
    torch.cuda.synchronize()
    calls_step_ms = np.array([e[0].elapsed_time(e[3]) for e in cev])
    per_score = np.array([e[0].elapsed_time(e[1]) for e in cev])
    per_select = np.array([e[1].elapsed_time(e[2]) for e in cev])
    per_compact = np.array([e[2].elapsed_time(e[3]) for e in cev])
    assert int(step.n_kept_tokens.item()) == n_keep_tok

    # Per-kernel durations: K more cold steps, each phase's kernel launched
    # with its own HIP event pair (hipExtLaunchKernel), so each pair times
    # that kernel's execution on the stream it runs on.
    def ev_pair():
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        b.record(stream)
        return a, b
    kev = [[ev_pair() for _ in PHASES] for _ in range(K)]
    torch.cuda.synchronize()
    for k in range(K):
        flush.max()
        for m, (ph, _) in enumerate(PHASES):
            pace.pace_time_next_kernel(ph, *kev[k][m])
        fused_step()
    torch.cuda.synchronize()
    kernel_us = {name: np.array([kev[k][m][0].elapsed_time(kev[k][m][1]) * 1e3 for k in range(K)])
                 for m, (_, name) in enumerate(PHASES)}

    # Group-level admission on the same pool: prompt groups of 8 trajectories,
    # occupancy and target counted in groups (NEXT-1 row), cold steps.
    go = torch.arange(0, pool.n + 1, 8, dtype=torch.int64, device=dev)
    if int(go[-1]) != pool.n:
        go = torch.cat([go, torch.tensor([pool.n], dtype=torch.int64, device=dev)])
    n_groups = go.numel() - 1
    g_occ, g_cap = n_groups, -(-pool.capacity // 8)
    gws = torch.empty(pace.pace_workspace_bytes(pace.WS_FILTER_STEP, max(pool.n, n_groups), pool.n_tokens),
                      dtype=torch.uint8, device=dev)
    gev = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(K + 2)]
    gout = pace.group_step_buffers(pool.n, n_groups, cols, dev)
    g_res = None
    for k in range(K + 2):
        flush.max()
        gev[k][0].record(stream)
        g_res = pace.pace_group_filter_step(tags, off, comp, pool.V, go, g_occ, g_cap, cols, prefix, window,
                                            params, 0.0, workspace=gws, out=gout)
        gev[k][1].record(stream)
    torch.cuda.synchronize()
    g_ms = np.array([e[0].elapsed_time(e[1]) for e in gev[2:]])
    g_kept_tok = int(g_res["n_kept_tokens"].item())

    # Warm back-to-back steps (no flush) for context.
    warm_ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    warm_ev[0].record(stream)
    for k in range(K):
        fused_step()
    warm_ev[1].record(stream)
    torch.cuda.synchronize()
    warm_ms = warm_ev[0].elapsed_time(warm_ev[1]) / K

    sweep = stream_sweep(args, pace, pool, tags, off, comp, prefix, window, cols, dev, stream) \
        if args.sweep_steps > 0 else None
    prefix_res = prefix_bench(pace, pool, K, flush, dev, stream)
    aux_res = aux_bench(pace, pool, step, off, comp, K, flush, dev, stream)

    if args.calib_copy:
        a = torch.empty(256 << 20, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        a.fill_(3)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()

    ms = rot_ms
    B, B_score = alg_bytes(pool, n_keep_tok, [c.element_size() for c in cols], W)
    score_ms = float(per_score.mean())
    B_red = reduce_bytes(pool, torch.cuda.get_device_properties(dev).multi_processor_count)
    red_s = float(kernel_us["score_reduce"].mean()) * 1e-6
    out = {
        "metric": METRIC,
        "value": pool.n_tokens / (ms * 1e-3),
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
                           pool.capacity, args.mode, len(cols)),
            "n_traj": pool.n, "n_tokens": pool.n_tokens, "budget": budget,
            "kept_tokens": n_keep_tok, "mode": args.mode, "payload_cols": len(cols),
            "parallelism": "single GPU",
        },
        "trajectories_per_s": pool.n / (ms * 1e-3),
        "hbm_frac_of_peak": B / (ms * 1e-3) / HBM_PEAK,
        "alg_bytes_per_step": B,
        "timing": "%d steps back to back between one event pair, over %d rotating pool copies "
                  "(each step's traffic exceeds the MALL, so every step starts cold); host enqueue %.2f ms "
                  "of %.2f ms wall" % (K, R, t_enq * 1e3, wall_rot * 1e3),
        "graph_rotation_ms_per_step": graph_ms,
        "graph_timing": "the same rotation with each copy's step captured once in a HIP graph and replayed",
        "flushed_ms_per_step": float(per_step.mean()),
        "rotation_kernel_us_mean": rot_kernel_us,
        "flushed_ms_p10_p50_p90": [float(np.percentile(per_step, q)) for q in (10, 50, 90)],
        "flushed_timing": "each step after a 512 MiB cache flush, bracketed by its own event pair",
        "entry": "pace_filter_step (score -> budget -> select -> compact, 4 launches)",
        "separate_calls_ms_per_step": float(calls_step_ms.mean()),
        "per_call_ms": {"pace_score": score_ms, "pace_budget+pace_select": float(per_select.mean()),
                        "pace_compact": float(per_compact.mean())},
        "kernel_us_mean": {k: float(v.mean()) for k, v in kernel_us.items()},
        "kernel_us_p50": {k: float(np.median(v)) for k, v in kernel_us.items()},
        "warm_ms_per_step": warm_ms,
        "stream_sweep": sweep,
        "prefix_score": prefix_res,
        "aux_kernels": aux_res,
        "group_step": {
            "entry": "pace_group_filter_step (groups of 8, group mean score)",
            "n_groups": n_groups, "occupancy_groups": g_occ, "target_groups": g_cap,
            "budget_groups": g_res["budget"], "kept_tokens": g_kept_tok,
            "ms_per_step": float(g_ms.mean()),
            "tokens_per_s": pool.n_tokens / (float(g_ms.mean()) * 1e-3),
            "hbm_frac_of_peak": (alg_bytes(pool, g_kept_tok, [c.element_size() for c in cols], W)[0]
                                 + n_groups * (8 + 8 + 8 + 1 + 4) + pool.n) / (float(g_ms.mean()) * 1e-3) / HBM_PEAK,
        },
        "wall_s_timed_region": wall_rot,
        "roofline": {
            "kernel": "score_reduce",
            "bound": "hbm",
            "achieved": B_red / red_s / 1e9,
            "peak": HBM_PEAK / 1e9,
            "unit": "GB/s",
            "frac": B_red / red_s / HBM_PEAK,
            "traffic": reduce_traffic(args.config),
            "alg_bytes": B_red,
        },
    }
    if not args.no_cpu_baseline:
        import oracle
        reps, t_cpu = 0, 0.0
        ts = time.perf_counter()
        while reps < 3 or time.perf_counter() - ts < args.cpu_seconds:
            oracle.filter_step(pool, mode=args.mode, cols=host_cols)
            reps += 1
        t_cpu = time.perf_counter() - ts
        out["cpu_baseline"] = {
            "value": reps * pool.n_tokens / t_cpu, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "trajectories_per_s": reps * pool.n / t_cpu, "GBps": reps * B / t_cpu / 1e9,
            "ms_per_step": t_cpu / reps * 1e3,
            "sample": "%d full oracle filter steps (score, budget, select, compact) on the same "
                      "%s pool, single-threaded C, %.1f s, on %s (%d host threads visible)"
                      % (reps, args.config, t_cpu, cpu_model(), os.cpu_count() or 0),
        }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
