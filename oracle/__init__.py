"""CPU oracle of the PACE filter step -- TEST INFRASTRUCTURE ONLY.

A plain single-threaded C implementation (``pace_oracle.c``) of the paper's
definitions, wrapped here with ctypes over numpy arrays. Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it. The GPU library does not import, link or call anything here, and
nothing here imports the GPU library.

Functions mirror the filter step: ``validate``, ``score`` (Eq. (1)-(2),
(6)-(9)), ``budget`` (Eq. (3)-(4)), ``select`` (Sec. 3.1 rejection rule,
exact count, ties to the lower id) and ``compact`` (Algorithm 1: survivors
packed into the training batch).
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "pace_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

OK = 0
ERR_ARG = -1
ERR_PRECONDITION = -3


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (IEEE double, no contraction, no fast-math)."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-fPIC", "-shared",
                               "-ffp-contract=off", "-fno-fast-math",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def load_library(path: str):
    """Open an oracle shared object and declare its C signatures."""
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    i64, i32, d = ctypes.c_int64, ctypes.c_int32, ctypes.c_double
    lib.oracle_validate.argtypes = [P, P, i64, i64, P, i32]
    lib.oracle_score.argtypes = [P, P, i64, i64, P, i32, P, P, i64, d, i32, i64, P, P, P]
    lib.oracle_budget.argtypes = [i64, i64, d, d, P, P]
    lib.oracle_select.argtypes = [P, i64, i64, P, P]
    lib.oracle_compact.argtypes = [P, i64, i64, P, ctypes.c_int, P, P, P, P, P, P]
    lib.oracle_group_score.argtypes = [P, i64, P, i64, P]
    lib.oracle_group_expand.argtypes = [P, i64, i64, P, P]
    lib.oracle_stream_admit.argtypes = [P, i64, d, d, i64, i64, P, i64, P, P, P, P, P, P]
    lib.oracle_prefix_score.argtypes = [P, P, P, P, i64, i64, i64, i64, P]
    lib.oracle_stale_k.argtypes = [P, P, i64, i64, P, i32, i64, P, P]
    lib.oracle_diagnostics.argtypes = [P, P, i64, i64, P, i32, P, P, P, i64, P, P]
    for f in ("oracle_validate", "oracle_score", "oracle_budget", "oracle_select", "oracle_compact",
              "oracle_group_score", "oracle_group_expand", "oracle_stream_admit", "oracle_prefix_score",
              "oracle_stale_k", "oracle_diagnostics"):
        getattr(lib, f).restype = ctypes.c_int
    return lib


def build_sanitized(out_path: str) -> str:
    """Compile a copy of the oracle with AddressSanitizer and
    UndefinedBehaviorSanitizer (any finding aborts), for the sanitizer run of
    the pin suite; returns its path."""
    subprocess.check_call(["gcc", "-O1", "-g", "-std=c99", "-fPIC", "-shared",
                           "-ffp-contract=off", "-fno-fast-math", "-fno-omit-frame-pointer",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-o", out_path, _SRC, "-lm"])
    return out_path


def _load():
    """The oracle library: the in-tree build, or the build named by
    PACE_ORACLE_LIB (the sanitizer run of the pin suite sets it)."""
    global _lib
    if _lib is None:
        path = os.environ.get("PACE_ORACLE_LIB")
        if not path:
            path = _LIB_PATH
            if not os.path.exists(path):
                build(force=False)
        _lib = load_library(path)
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class OracleError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__("%s failed with code %d" % (what, code))
        self.code = code


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def validate(tags, offsets, completion, V) -> int:
    tags, offsets, completion = _c(tags, np.int32), _c(offsets, np.int64), _c(completion, np.int32)
    n = offsets.shape[0] - 1
    return _load().oracle_validate(_p(tags), _p(offsets), n, tags.shape[0], _p(completion), int(V))


def score(tags, offsets, completion, V, prefix=None, window=None, w_wait=1.0,
          gamma=4, window_min=32, check=True):
    """Returns (score float64[n], S int64[n], T int64[n]) or raises."""
    tags, offsets, completion = _c(tags, np.int32), _c(offsets, np.int64), _c(completion, np.int32)
    n = offsets.shape[0] - 1
    prefix = None if prefix is None else _c(prefix, np.float64)
    window = np.empty(0) if window is None else _c(window, np.float64)
    out = np.empty(n, np.float64)
    S = np.empty(n, np.int64)
    T = np.empty(n, np.int64)
    rc = _load().oracle_score(_p(tags), _p(offsets), n, tags.shape[0], _p(completion), int(V),
                              _p(prefix), _p(window), window.shape[0], float(w_wait), int(gamma),
                              int(window_min), _p(out), _p(S), _p(T))
    if rc != OK:
        if check:
            raise OracleError(rc, "oracle_score")
        return rc
    return out, S, T


def budget(N, N_tar, r_hat_prev=0.0, beta=0.0, r_max=0.9, check=True):
    """Returns (budget, r_hat)."""
    rh = ctypes.c_double(float(r_hat_prev))
    b = ctypes.c_int64(0)
    rc = _load().oracle_budget(int(N), int(N_tar), float(beta), float(r_max),
                               ctypes.addressof(rh), ctypes.addressof(b))
    if rc != OK:
        if check:
            raise OracleError(rc, "oracle_budget")
        return rc
    return int(b.value), float(rh.value)


def select(score_arr, budget_n, check=True):
    """Returns (keep uint8[n], reject_ids int32[budget])."""
    s = _c(score_arr, np.float64)
    n = s.shape[0]
    keep = np.empty(n, np.uint8)
    rej = np.empty(max(int(budget_n), 0), np.int32)
    rc = _load().oracle_select(_p(s), n, int(budget_n), _p(keep), _p(rej))
    if rc != OK:
        if check:
            raise OracleError(rc, "oracle_select")
        return rc
    return keep, rej


def compact(offsets, keep, cols: Sequence[np.ndarray], check=True):
    """Returns (offsets_out int64[n_kept+1], kept_ids int32[n_kept], packed cols)."""
    offsets = _c(offsets, np.int64)
    keep = _c(keep, np.uint8)
    n = offsets.shape[0] - 1
    cols = [np.ascontiguousarray(c) for c in cols]
    n_tokens = int(cols[0].shape[0]) if cols else int(offsets[-1])
    outs = [np.empty_like(c) for c in cols]
    nc = len(cols)
    cin = (ctypes.c_void_p * max(nc, 1))(*[c.ctypes.data for c in cols])
    cout = (ctypes.c_void_p * max(nc, 1))(*[o.ctypes.data for o in outs])
    eb = (ctypes.c_int32 * max(nc, 1))(*[c.dtype.itemsize for c in cols])
    off_out = np.empty(n + 1, np.int64)
    ids = np.empty(max(n, 1), np.int32)
    nk = ctypes.c_int64(0)
    rc = _load().oracle_compact(_p(offsets), n, n_tokens, _p(keep), nc, cin, eb, cout,
                                _p(off_out), _p(ids), ctypes.addressof(nk))
    if rc != OK:
        if check:
            raise OracleError(rc, "oracle_compact")
        return rc
    n_kept = int(keep.astype(bool).sum())
    tot = int(nk.value)
    return off_out[: n_kept + 1].copy(), ids[:n_kept].copy(), [o[:tot].copy() for o in outs]


def filter_step(pool, mode="effective", w_wait=None, gamma=4, window_min=32,
                beta=0.0, r_max=0.9, r_hat_prev=0.0, cols=None):
    """One whole filter step on a poolgen.Pool: score -> budget -> select -> compact.
    mode: 'effective' (Eq. (7)), 'raw' (F = 1) or 'gen' (w_wait = 0, Eq. (7) weight)."""
    prefix = None if mode == "raw" else pool.prefix_score
    window = None if mode == "raw" else pool.window
    if w_wait is None:
        w_wait = 0.0 if mode == "gen" else 1.0
    sc, S, T = score(pool.tags, pool.offsets, pool.completion, pool.V, prefix, window,
                     w_wait, gamma, window_min)
    b, r_hat = budget(pool.occupancy, pool.capacity, r_hat_prev, beta, r_max)
    keep, rej = select(sc, b)
    cols = [pool.tags] if cols is None else cols
    off_out, ids, packed = compact(pool.offsets, keep, cols)
    return dict(score=sc, S=S, T=T, budget=b, r_hat=r_hat, keep=keep, reject_ids=rej,
                offsets_out=off_out, kept_ids=ids, packed=packed,
                n_kept_tokens=int(off_out[-1]))


def group_score(score_arr, group_offsets, check=True):
    """Mean member score per prompt group (empty group: 0)."""
    s = _c(score_arr, np.float64)
    go = _c(group_offsets, np.int64)
    ng = go.shape[0] - 1
    out = np.empty(max(ng, 1), np.float64)
    rc = _load().oracle_group_score(_p(s), s.shape[0], _p(go), ng, _p(out))
    if rc != OK:
        if check:
            raise OracleError(rc, "oracle_group_score")
        return rc
    return out[:ng].copy()


def group_expand(group_offsets, group_keep, n, check=True):
    """Trajectory keep flags uint8[n] from group keep flags."""
    go = _c(group_offsets, np.int64)
    gk = _c(group_keep, np.uint8)
    ng = go.shape[0] - 1
    keep = np.empty(max(int(n), 1), np.uint8)
    rc = _load().oracle_group_expand(_p(go), ng, int(n), _p(gk), _p(keep))
    if rc != OK:
        if check:
            raise OracleError(rc, "oracle_group_expand")
        return rc
    return keep[: int(n)].copy()


def group_filter_step(pool, group_offsets, occupancy, capacity, mode="effective", w_wait=None,
                      gamma=4, window_min=32, beta=0.0, r_max=0.9, r_hat_prev=0.0, cols=None):
    """One filter step with prompt groups as the admission unit: trajectory
    scores, group means, a budget in groups (occupancy and capacity count
    groups), group selection, and compaction of the kept groups' members."""
    prefix = None if mode == "raw" else pool.prefix_score
    window = None if mode == "raw" else pool.window
    if w_wait is None:
        w_wait = 0.0 if mode == "gen" else 1.0
    sc, S, T = score(pool.tags, pool.offsets, pool.completion, pool.V, prefix, window,
                     w_wait, gamma, window_min)
    gs = group_score(sc, group_offsets)
    b, r_hat = budget(occupancy, capacity, r_hat_prev, beta, r_max)
    gkeep, grej = select(gs, b)
    keep = group_expand(group_offsets, gkeep, pool.n)
    cols = [pool.tags] if cols is None else cols
    off_out, ids, packed = compact(pool.offsets, keep, cols)
    return dict(score=sc, S=S, T=T, group_score=gs, budget=b, r_hat=r_hat, group_keep=gkeep,
                reject_group_ids=grej, keep=keep, offsets_out=off_out, kept_ids=ids, packed=packed,
                n_kept_tokens=int(off_out[-1]))


class StreamWindow:
    """The sliding window of observed scores (a ring of `cap` entries)."""

    def __init__(self, cap=512):
        self.ring = np.zeros(cap, np.float64)
        self.cap, self.head, self.count = cap, 0, 0

    def copy(self):
        w = StreamWindow(self.cap)
        w.ring[:] = self.ring
        w.head, w.count = self.head, self.count
        return w

    def entries(self):
        """The window's scores, oldest first."""
        return np.array([self.ring[(self.head - self.count + t) % self.cap] for t in range(self.count)])


def stream_admit(score_arr, r_hat, window: StreamWindow, batch_size, r_max=0.9, window_min=32, check=True):
    """One step of the streaming rule; updates `window` in place. Returns
    (status uint8[n]: 0 rejected, 1 retained, 2 not drawn; kappa; n_drawn; n_retained)."""
    s = _c(score_arr, np.float64)
    n = s.shape[0]
    status = np.empty(max(n, 1), np.uint8)
    head, cnt = ctypes.c_int64(window.head), ctypes.c_int64(window.count)
    kappa = ctypes.c_double(0.0)
    drawn, kept = ctypes.c_int64(0), ctypes.c_int64(0)
    rc = _load().oracle_stream_admit(_p(s), n, float(r_hat), float(r_max), int(window_min), int(batch_size),
                                     _p(window.ring), window.cap, ctypes.addressof(head), ctypes.addressof(cnt),
                                     _p(status), ctypes.addressof(kappa), ctypes.addressof(drawn),
                                     ctypes.addressof(kept))
    if rc != OK:
        if check:
            raise OracleError(rc, "oracle_stream_admit")
        return rc
    window.head, window.count = int(head.value), int(cnt.value)
    return status[:n].copy(), float(kappa.value), int(drawn.value), int(kept.value)


def prefix_score(lp_new, lp_behavior, prefix_offsets, tags=None, cap=1024, min_tokens=32, check=True):
    """Eq. (5): mean |lp_new - lp_behavior| over each prefix's first `cap`
    eligible tokens (tag != -1); NaN below `min_tokens` eligible tokens."""
    a = _c(lp_new, np.float32)
    b = _c(lp_behavior, np.float32)
    po = _c(prefix_offsets, np.int64)
    tg = None if tags is None else _c(tags, np.int32)
    n = po.shape[0] - 1
    out = np.empty(max(n, 1), np.float64)
    rc = _load().oracle_prefix_score(_p(a), _p(b), _p(tg), _p(po), n, a.shape[0], int(cap), int(min_tokens), _p(out))
    if rc != OK:
        if check:
            raise OracleError(rc, "oracle_prefix_score")
        return rc
    return out[:n].copy()


def stale_k(tags, offsets, completion, V, k, check=True):
    """Stale-k admission (Eq. (1) lag <= k). Returns (keep uint8[n], lag f64[n])."""
    tags = _c(tags, np.int32)
    offsets = _c(offsets, np.int64)
    completion = _c(completion, np.int32)
    n = offsets.shape[0] - 1
    keep = np.empty(max(n, 1), np.uint8)
    lag = np.empty(max(n, 1), np.float64)
    rc = _load().oracle_stale_k(_p(tags), _p(offsets), n, tags.shape[0], _p(completion), int(V), int(k),
                                _p(keep), _p(lag))
    if rc != OK:
        if check:
            raise OracleError(rc, "oracle_stale_k")
        return rc
    return keep[:n].copy(), lag[:n].copy()


def diagnostics(tags, offsets, completion, V, score_arr, keep, edges, check=True):
    """Kept/rejected histograms of K_wait, K_gen, K_eff and exact totals.
    edges: f64 [3][nbins+1]. Returns (hist int64[3][2][nbins+2], totals int64[2][4])."""
    tags = _c(tags, np.int32)
    offsets = _c(offsets, np.int64)
    completion = _c(completion, np.int32)
    s = _c(score_arr, np.float64)
    kp = _c(keep, np.uint8)
    e = _c(edges, np.float64)
    nbins = e.shape[1] - 1
    n = offsets.shape[0] - 1
    hist = np.empty((3, 2, nbins + 2), np.int64)
    tot = np.empty((2, 4), np.int64)
    rc = _load().oracle_diagnostics(_p(tags), _p(offsets), n, tags.shape[0], _p(completion), int(V), _p(s),
                                    _p(kp), _p(e), nbins, _p(hist), _p(tot))
    if rc != OK:
        if check:
            raise OracleError(rc, "oracle_diagnostics")
        return rc
    return hist, tot

