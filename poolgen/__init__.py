"""Seeded synthetic trajectory pools for the PACE filter step.

This module only draws inputs. It computes none of the method's arithmetic
(no staleness, no score, no budget, no selection): it emits the arrays a
rollout system would hand to the trainer, and both the CPU oracle and the
GPU library consume them unchanged.

A pool is a CSR layout over tokens:

* ``tags``        int32 [N_tok]  behavior policy version of each token
                  (Sec. 2, "Trajectory Lifecycle"); -1 marks a non-generated
                  token (tool output in multi-turn rollouts, which stays in
                  context but is masked from the loss, App. B "ReTool").
* ``offsets``     int64 [n+1]    trajectory i owns tokens [offsets[i], offsets[i+1]).
* ``completion``  int32 [n]      trainer version c(tau) when tau completed.
* ``V``           int            current trainer version j.
* ``occupancy``, ``capacity``    N_j and N^tar of Eq. (3).
* ``prefix_score`` float64 [n]   s_pre of Eq. (5); NaN where the rollout was
                  never interrupted (prefix scores exist only at interruptions,
                  App. B "Admission and prefix-scoring parameters").
* ``window``      float64 [W]    sorted recent prefix scores (Eq. (8)).

Shapes follow the paper's workloads (single-turn math, long reasoning,
multi-turn tool use; Sec. 4 and App. B). All randomness comes from numpy's
PCG64 seeded per pool, so a (config, seed) pair always yields the same bytes.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

__all__ = ["Pool", "CONFIGS", "make_pool", "make_custom_pool", "refresh_slots"]


@dataclasses.dataclass
class Pool:
    name: str
    tags: np.ndarray          # int32 [N_tok]
    offsets: np.ndarray       # int64 [n+1]
    completion: np.ndarray    # int32 [n]
    V: int
    occupancy: int
    capacity: int
    prefix_score: np.ndarray  # float64 [n]
    window: np.ndarray        # float64 [W], ascending
    group_offsets: Optional[np.ndarray] = None  # int64 [g+1] over trajectories
    seed: int = 0

    @property
    def n(self) -> int:
        return int(self.offsets.shape[0] - 1)

    @property
    def n_tokens(self) -> int:
        return int(self.tags.shape[0])


# Pool recipes. Lengths are log-normal around a median with the spread that
# reproduces the stated token totals, clipped to the stated range.
CONFIGS: Dict[str, dict] = {
    # 64 trajectories, U{128..2048} tokens, 0-2 version breaks, c = last tag,
    # V = 20, target 48.
    "tiny": dict(n=64, V=20, capacity=48, seed=101, kind="uniform",
                 len_lo=128, len_hi=2048, breaks=("uniform", 0, 2),
                 c_lag=4, last_lag=0),
    # 1024 trajectories in groups of 8, LN(median 3000) clipped 256..16384,
    # 0-3 breaks, V = 200, occupancy 1.5x target.
    "math": dict(n=1024, V=200, capacity=683, seed=102, kind="lognormal",
                 median=3000.0, sigma=0.749, len_lo=256, len_hi=16384,
                 breaks=("uniform", 0, 3), c_lag=8, last_lag=1, group=8),
    # 2048 trajectories, heavy-tailed LN(median 8000) clipped 512..32768,
    # up to 6 breaks skewed toward long rollouts, V = 1000, occupancy 2x.
    "long": dict(n=2048, V=1000, capacity=1024, seed=103, kind="lognormal",
                 median=8000.0, sigma=0.656, len_lo=512, len_hi=32768,
                 breaks=("binomial_len", 6), c_lag=8, last_lag=1),
    # 2048 multi-turn trajectories: 2-12 generated turns of 64..2048 tokens,
    # separated by masked tool spans of 32..1024 tokens; V = 500,
    # occupancy 1.3x target.
    "multiturn": dict(n=2048, V=500, capacity=1575, seed=104, kind="multiturn",
                      turns=(2, 12), gen=(64, 2048), tool=(32, 1024),
                      breaks=("uniform", 0, 4), c_lag=8, last_lag=1),
    # 4096 trajectories, LN(median 12000) up to 32768 (~50M tokens),
    # 0-16 breaks, V = 5000, occupancy 3x target.
    "stress": dict(n=4096, V=5000, capacity=1365, seed=105, kind="lognormal",
                   median=12000.0, sigma=0.185, len_lo=512, len_hi=32768,
                   breaks=("uniform", 0, 16), c_lag=8, last_lag=1),
    # Scale case beyond the paper's pool sizes: 65536 short trajectories,
    # LN(median 700) clipped 64..8192 (~52M tokens), 0-4 breaks, V = 5000,
    # occupancy 3x target (the selection spread over the chip).
    "wide": dict(n=65536, V=5000, capacity=21845, seed=106, kind="lognormal",
                 median=700.0, sigma=0.5, len_lo=64, len_hi=8192,
                 breaks=("uniform", 0, 4), c_lag=8, last_lag=1),
}


def _lengths(rng: np.random.Generator, cfg: dict, n: int) -> np.ndarray:
    if cfg["kind"] == "uniform":
        return rng.integers(cfg["len_lo"], cfg["len_hi"] + 1, size=n, dtype=np.int64)
    z = rng.standard_normal(n)
    L = np.rint(np.exp(np.log(cfg["median"]) + cfg["sigma"] * z))
    return np.clip(L, cfg["len_lo"], cfg["len_hi"]).astype(np.int64)


def _n_breaks(rng: np.random.Generator, spec, L: int, cfg: dict) -> int:
    if spec[0] == "uniform":
        return int(rng.integers(spec[1], spec[2] + 1))
    if spec[0] == "binomial_len":
        p = (L - cfg["len_lo"]) / float(cfg["len_hi"] - cfg["len_lo"])
        return int(rng.binomial(spec[1], min(max(p, 0.0), 1.0)))
    raise ValueError(spec)


def _version_path(rng: np.random.Generator, k: int, c: int, last_lag: int):
    """Versions of the k+1 generation segments: each break raises the version
    by 1 or 2; the final segment runs at c - U{0..last_lag}."""
    last = c - (int(rng.integers(0, last_lag + 1)) if last_lag > 0 else 0)
    inc = rng.integers(1, 3, size=k)
    start = last - int(inc.sum())
    vers = np.empty(k + 1, dtype=np.int64)
    vers[0] = start
    if k:
        vers[1:] = start + np.cumsum(inc)
    return np.maximum(vers, 0)


def _single_turn(rng, cfg, n, V):
    L = _lengths(rng, cfg, n)
    seg_v, seg_len, comp, nbreaks = [], [], np.empty(n, np.int64), np.empty(n, np.int64)
    for i in range(n):
        Li = int(L[i])
        k = min(_n_breaks(rng, cfg["breaks"], Li, cfg), Li - 1)
        c = V - int(rng.integers(0, cfg["c_lag"] + 1))
        vers = _version_path(rng, k, c, cfg["last_lag"])
        if cfg["last_lag"] == 0:   # tiny pool: completion version = last tag
            c = int(vers[-1])
        cuts = np.sort(rng.choice(Li - 1, size=k, replace=False) + 1) if k else np.empty(0, np.int64)
        bounds = np.concatenate(([0], cuts, [Li]))
        seg_v.append(vers)
        seg_len.append(np.diff(bounds))
        comp[i] = c
        nbreaks[i] = k
    v = np.concatenate(seg_v)
    ln = np.concatenate(seg_len)
    tags = np.repeat(v.astype(np.int32), ln)
    offsets = np.zeros(n + 1, np.int64)
    offsets[1:] = np.cumsum(L)
    return tags, offsets, comp.astype(np.int32), nbreaks


def _multi_turn(rng, cfg, n, V):
    seg_v, seg_len, comp, nbreaks, lens = [], [], np.empty(n, np.int64), np.empty(n, np.int64), np.empty(n, np.int64)
    for i in range(n):
        turns = int(rng.integers(cfg["turns"][0], cfg["turns"][1] + 1))
        gen = rng.integers(cfg["gen"][0], cfg["gen"][1] + 1, size=turns)
        tool = rng.integers(cfg["tool"][0], cfg["tool"][1] + 1, size=turns - 1)
        G = int(gen.sum())
        turn_start = np.concatenate(([0], np.cumsum(gen)[:-1]))  # generated-token index of each turn start
        k = _n_breaks(rng, cfg["breaks"], G, cfg)
        pos = set()
        for _ in range(k):
            if turns > 1 and rng.random() < 0.5:
                pos.add(int(turn_start[int(rng.integers(1, turns))]))
            else:
                pos.add(int(rng.integers(1, G)))
        cuts = np.array(sorted(pos), dtype=np.int64)
        c = V - int(rng.integers(0, cfg["c_lag"] + 1))
        vers = _version_path(rng, len(cuts), c, cfg["last_lag"])
        # version of every generated token, then interleave masked tool spans
        gbounds = np.concatenate(([0], cuts, [G]))
        gver = np.repeat(vers, np.diff(gbounds))
        gsplit = np.split(gver, np.cumsum(gen)[:-1])
        parts_v, parts_l = [], []
        for t in range(turns):
            g = gsplit[t]
            # run-length encode this turn's versions
            chg = np.flatnonzero(np.diff(g)) + 1
            b = np.concatenate(([0], chg, [len(g)]))
            parts_v.append(g[b[:-1]])
            parts_l.append(np.diff(b))
            if t < turns - 1:
                parts_v.append(np.array([-1], np.int64))
                parts_l.append(np.array([tool[t]], np.int64))
        seg_v.append(np.concatenate(parts_v))
        seg_len.append(np.concatenate(parts_l))
        comp[i] = c
        nbreaks[i] = len(cuts)
        lens[i] = G + int(tool.sum())
    tags = np.repeat(np.concatenate(seg_v).astype(np.int32), np.concatenate(seg_len))
    offsets = np.zeros(n + 1, np.int64)
    offsets[1:] = np.cumsum(lens)
    return tags, offsets, comp.astype(np.int32), nbreaks


def _prefix_scores(rng, nbreaks: np.ndarray, W: int = 512):
    """s_pre ~ log-normal(median 0.02, sigma 1) for interrupted rollouts,
    NaN otherwise; the window holds W earlier draws of the same law, sorted."""
    n = nbreaks.shape[0]
    s = np.exp(np.log(0.02) + rng.standard_normal(n))
    s[nbreaks == 0] = np.nan
    window = np.sort(np.exp(np.log(0.02) + rng.standard_normal(W)))
    return s, window


def make_pool(name: str, seed: Optional[int] = None, n: Optional[int] = None) -> Pool:
    """Build one of the named pools. ``n`` overrides the trajectory count
    (and scales the capacity target proportionally) for reduced-size cases."""
    cfg = CONFIGS[name]
    seed = cfg["seed"] if seed is None else int(seed)
    n_traj = cfg["n"] if n is None else int(n)
    rng = np.random.default_rng(seed)
    V = cfg["V"]
    if cfg["kind"] == "multiturn":
        tags, offsets, comp, nb = _multi_turn(rng, cfg, n_traj, V)
    else:
        tags, offsets, comp, nb = _single_turn(rng, cfg, n_traj, V)
    ps, window = _prefix_scores(rng, nb)
    cap = cfg["capacity"] if n is None else int(round(cfg["capacity"] * n_traj / cfg["n"]))
    groups = None
    if cfg.get("group"):
        g = cfg["group"]
        groups = np.arange(0, n_traj + 1, g, dtype=np.int64)
        if groups[-1] != n_traj:
            groups = np.append(groups, n_traj)
    return Pool(name=name, tags=tags, offsets=offsets, completion=comp, V=V,
                occupancy=n_traj, capacity=cap, prefix_score=ps, window=window,
                group_offsets=groups, seed=seed)


def make_custom_pool(lengths, V: int, seed: int, max_breaks: int = 3,
                     mask_frac: float = 0.0, c_lag: int = 8,
                     capacity: Optional[int] = None, W: int = 512,
                     prefix_nan_frac: float = 0.3) -> Pool:
    """Small pools with explicit lengths (zero allowed) for edge cases.
    Tags are non-decreasing per trajectory, <= c <= V; a fraction
    ``mask_frac`` of tokens is overwritten with the mask tag -1."""
    rng = np.random.default_rng(seed)
    lengths = np.asarray(lengths, dtype=np.int64)
    n = lengths.shape[0]
    seg_v, seg_len = [], []
    comp = np.empty(n, np.int64)
    for i in range(n):
        Li = int(lengths[i])
        c = max(V - int(rng.integers(0, c_lag + 1)), 0)
        k = min(int(rng.integers(0, max_breaks + 1)), max(Li - 1, 0))
        vers = _version_path(rng, k, c, 1)
        cuts = np.sort(rng.choice(Li - 1, size=k, replace=False) + 1) if k else np.empty(0, np.int64)
        bounds = np.concatenate(([0], cuts, [Li]))
        seg_v.append(vers)
        seg_len.append(np.diff(bounds))
        comp[i] = c
    tags = np.repeat(np.concatenate(seg_v).astype(np.int32), np.concatenate(seg_len)) if n else np.empty(0, np.int32)
    if mask_frac > 0 and tags.size:
        m = rng.random(tags.size) < mask_frac
        tags[m] = -1
    offsets = np.zeros(n + 1, np.int64)
    offsets[1:] = np.cumsum(lengths)
    s = np.exp(np.log(0.02) + rng.standard_normal(n))
    s[rng.random(n) < prefix_nan_frac] = np.nan
    window = np.sort(np.exp(np.log(0.02) + rng.standard_normal(W))) if W else np.empty(0)
    cap = (2 * n) // 3 if capacity is None else capacity
    return Pool(name="custom", tags=tags, offsets=offsets, completion=comp.astype(np.int32),
                V=V, occupancy=n, capacity=cap, prefix_score=s, window=window, seed=seed)


def refresh_slots(pool: Pool, step: int, frac: float = 0.05, seed_base: int = 0):
    """Length-preserving refresh of ``frac`` of the pool for step ``step`` of a
    back-to-back sweep: slots [(m*step) mod n, +m) are regenerated as freshly
    completed rollouts (c = V), their tags redrawn. Returns (slot ids, new
    tags for those slots concatenated in slot order, new completion values)."""
    n = pool.n
    m = max(1, int(round(frac * n)))
    rng = np.random.default_rng(seed_base + 7919 * (step + 1))
    slots = (np.arange(m) + m * step) % n
    new_tags, new_c = [], np.empty(m, np.int32)
    for k, i in enumerate(slots):
        Li = int(pool.offsets[i + 1] - pool.offsets[i])
        c = pool.V
        kk = min(int(rng.integers(0, 17)), max(Li - 1, 0))
        vers = _version_path(rng, kk, c, 1)
        cuts = np.sort(rng.choice(Li - 1, size=kk, replace=False) + 1) if kk else np.empty(0, np.int64)
        bounds = np.concatenate(([0], cuts, [Li]))
        new_tags.append(np.repeat(vers.astype(np.int32), np.diff(bounds)))
        new_c[k] = c
    return slots, (np.concatenate(new_tags) if new_tags else np.empty(0, np.int32)), new_c


def sweep_step(pool: Pool, step: int, V0: int, frac: float = 0.05, seed_base: int = 0):
    """Advances a pool in place to step ``step`` of a back-to-back sweep: the
    current version becomes V0 + step and ``frac`` of the slots are refreshed
    as freshly completed, never-interrupted rollouts (refresh_slots; their
    prefix score becomes NaN). Returns the refreshed slot ids, so that a
    device copy can be updated span by span."""
    pool.V = V0 + step
    slots, new_tags, new_c = refresh_slots(pool, step, frac, seed_base)
    pos = 0
    for k, i in enumerate(slots):
        lo, hi = int(pool.offsets[i]), int(pool.offsets[i + 1])
        pool.tags[lo:hi] = new_tags[pos:pos + hi - lo]
        pos += hi - lo
        pool.completion[i] = new_c[k]
        if pool.prefix_score is not None:
            pool.prefix_score[i] = np.nan
    return slots


def make_prefixes(pool: Pool, seed: int = 0):
    """Synthetic rescored prefixes for a pool: every trajectory with a version
    break was interrupted there, and its prefix is its tokens before the first
    break. Behaviour log-probabilities are drawn per token (f32, <= 0); the
    rescoring policy's ones add a per-prefix drift. Returns (traj_ids,
    prefix_offsets int64[m+1], lp_new f32, lp_behavior f32, tags int32)."""
    rng = np.random.default_rng(seed + 4242)
    ids, lens = [], []
    for i in range(pool.n):
        lo, hi = int(pool.offsets[i]), int(pool.offsets[i + 1])
        t = pool.tags[lo:hi]
        gen = np.flatnonzero(t != -1)
        if len(gen) == 0:
            continue
        first = t[gen[0]]
        later = gen[t[gen] != first]
        if len(later) == 0:
            continue
        ids.append(i)
        lens.append(int(later[0]))
    ids = np.array(ids, np.int64)
    po = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    m = int(po[-1])
    tags = np.empty(m, np.int32)
    for k, i in enumerate(ids):
        lo = int(pool.offsets[i])
        tags[po[k]:po[k + 1]] = pool.tags[lo:lo + lens[k]]
    lp_b = np.minimum(rng.normal(-1.2, 0.8, m), 0.0).astype(np.float32)
    drift = np.repeat(rng.lognormal(np.log(0.02), 1.0, len(ids)), lens)
    lp_n = np.minimum(lp_b + rng.normal(0.0, 1.0, m) * drift, 0.0).astype(np.float32)
    return ids, po, lp_n, lp_b, tags
