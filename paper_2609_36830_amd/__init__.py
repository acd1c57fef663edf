"""PACE pool filter step on AMD Instinct MI355X (gfx950).

Thin ctypes binding of ``libpace.so`` (declared in ``include/pace.h``). Each
function has the C entry point's name and only marshals arguments: it checks
tensor dtypes/devices, allocates output tensors that were not supplied, and
passes raw device pointers plus the current HIP stream. Every step of the
filter runs in the library's HIP kernels; there is no CPU or PyTorch
fallback, and importing this package on a machine without the built library
fails loudly.

    score, S, T      = pace_score(tags, offsets, completion, V, prefix, window)
    budget, r_hat    = pace_budget(occupancy, capacity, r_hat_prev=0.0)
    keep, reject_ids = pace_select(score, budget)
    off_out, ids, n_kept_tokens, packed = pace_compact(offsets, keep, [tags])
"""
from __future__ import annotations

import ctypes
from typing import Optional, Sequence

import torch

from ._lib import PaceParams, lib, library_path

__all__ = [
    "PaceError", "PaceParams", "default_params", "pace_workspace_bytes", "pace_score",
    "pace_budget", "pace_select", "pace_compact", "pace_validate", "pace_filter_step",
    "pace_filter_step_noalloc", "FilterStep",
    "library_path", "WS_SCORE", "WS_SELECT", "WS_COMPACT", "WS_FILTER_STEP",
    "BAD_OFFSETS", "BAD_COMPLETION", "BAD_TAG", "BAD_WINDOW",
]

WS_SCORE, WS_SELECT, WS_COMPACT, WS_FILTER_STEP = 0, 1, 2, 3
BAD_OFFSETS, BAD_COMPLETION, BAD_TAG, BAD_WINDOW, BAD_GROUPS = 0x1, 0x2, 0x4, 0x8, 0x10
PHASE_REDUCE, PHASE_FINALIZE, PHASE_SELECT, PHASE_COMPACT, PHASE_PREFIX, PHASE_AUX, PHASE_CLASSIFY = \
    0, 1, 2, 3, 4, 5, 6


class PaceError(RuntimeError):
    def __init__(self, code: int, fn: str):
        msg = lib().pace_strerror(code).decode()
        super().__init__("%s: %s (code %d)" % (fn, msg, code))
        self.code = code


def _check(code: int, fn: str):
    if code != 0:
        raise PaceError(code, fn)


def default_params(**kw) -> PaceParams:
    p = PaceParams()
    lib().pace_default_params(ctypes.byref(p))
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dev(t: torch.Tensor, dtype, name: str) -> torch.Tensor:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if t.dtype != dtype:
        raise ValueError("%s must have dtype %s, got %s" % (name, dtype, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t


def _stream(device: torch.device, stream=None) -> int:
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def pace_workspace_bytes(which: int, n_traj: int, n_tokens: int) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().pace_workspace_bytes(int(which), int(n_traj), int(n_tokens), ctypes.byref(out)),
           "pace_workspace_bytes")
    return int(out.value)


def _workspace(which, n, nt, device, ws):
    need = pace_workspace_bytes(which, n, nt)
    if ws is None:
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=device)
    return ws


def pace_score(tags, offsets, completion, current_version, prefix_score=None, window_sorted=None,
               params: Optional[PaceParams] = None, score_out=None, gen_sum_out=None,
               gen_count_out=None, workspace=None, stream=None, with_counts=True):
    """Eq. (1)-(2), (6)-(9). Returns (score f64[n], S i64[n] or None, T i64[n] or None)."""
    _dev(tags, torch.int32, "tags")
    _dev(offsets, torch.int64, "offsets")
    _dev(completion, torch.int32, "completion")
    n = offsets.numel() - 1
    nt = tags.numel()
    dev = tags.device
    if prefix_score is not None:
        _dev(prefix_score, torch.float64, "prefix_score")
    W = 0
    if window_sorted is not None:
        _dev(window_sorted, torch.float64, "window_sorted")
        W = window_sorted.numel()
    if score_out is None:
        score_out = torch.empty(n, dtype=torch.float64, device=dev)
    if with_counts:
        if gen_sum_out is None:
            gen_sum_out = torch.empty(n, dtype=torch.int64, device=dev)
        if gen_count_out is None:
            gen_count_out = torch.empty(n, dtype=torch.int64, device=dev)
    ws = _workspace(WS_SCORE, n, nt, dev, workspace)
    _check(lib().pace_score(_ptr(tags), _ptr(offsets), n, nt, _ptr(completion), int(current_version),
                            _ptr(prefix_score), _ptr(window_sorted), W,
                            ctypes.byref(params) if params is not None else None,
                            _ptr(score_out), _ptr(gen_sum_out), _ptr(gen_count_out),
                            _ptr(ws), ws.numel(), _stream(dev, stream)), "pace_score")
    return score_out, gen_sum_out, gen_count_out


def pace_budget(occupancy: int, capacity: int, params: Optional[PaceParams] = None,
                r_hat_prev: float = 0.0):
    """Eq. (3)-(4) on the host. Returns (budget, r_hat)."""
    rh = ctypes.c_double(float(r_hat_prev))
    b = ctypes.c_int64(0)
    _check(lib().pace_budget(int(occupancy), int(capacity),
                             ctypes.byref(params) if params is not None else None,
                             ctypes.byref(rh), ctypes.byref(b)), "pace_budget")
    return int(b.value), float(rh.value)


def pace_select(score, budget: int, keep_out=None, reject_ids_out=None, workspace=None, stream=None):
    """Reject exactly `budget` highest scores, ties to the lower id.
    Returns (keep u8[n], reject_ids i32[budget])."""
    _dev(score, torch.float64, "score")
    n = score.numel()
    dev = score.device
    if keep_out is None:
        keep_out = torch.empty(n, dtype=torch.uint8, device=dev)
    if reject_ids_out is None:
        reject_ids_out = torch.empty(max(int(budget), 1), dtype=torch.int32, device=dev)
    ws = _workspace(WS_SELECT, n, 0, dev, workspace)
    _check(lib().pace_select(_ptr(score), n, int(budget), _ptr(keep_out), _ptr(reject_ids_out),
                             _ptr(ws), ws.numel(), _stream(dev, stream)), "pace_select")
    return keep_out, reject_ids_out[: int(budget)]


def pace_compact(offsets, keep, cols: Sequence[torch.Tensor], cols_out=None, offsets_out=None,
                 kept_ids_out=None, n_kept_tokens_out=None, workspace=None, stream=None,
                 n_tokens: Optional[int] = None):
    """Pack kept spans of every column. Returns (offsets_out i64[n+1], kept_ids i32[n],
    n_kept_tokens i64[1] device scalar, packed columns at full capacity). Only the
    first n_kept+1 / n_kept / n_kept_tokens entries are meaningful."""
    _dev(offsets, torch.int64, "offsets")
    _dev(keep, torch.uint8, "keep")
    n = offsets.numel() - 1
    dev = offsets.device
    cols = list(cols)
    if n_tokens is None:
        n_tokens = cols[0].numel() if cols else int(offsets[-1].item())
    for k, c in enumerate(cols):
        if not c.is_cuda or not c.is_contiguous() or c.numel() != n_tokens:
            raise ValueError("column %d must be a contiguous device tensor of n_tokens elements" % k)
    if cols_out is None:
        cols_out = [torch.empty_like(c) for c in cols]
    if offsets_out is None:
        offsets_out = torch.empty(n + 1, dtype=torch.int64, device=dev)
    if kept_ids_out is None:
        kept_ids_out = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
    if n_kept_tokens_out is None:
        n_kept_tokens_out = torch.empty(1, dtype=torch.int64, device=dev)
    ws = _workspace(WS_COMPACT, n, n_tokens, dev, workspace)
    nc = len(cols)
    cin = (ctypes.c_void_p * max(nc, 1))(*[c.data_ptr() for c in cols])
    cout = (ctypes.c_void_p * max(nc, 1))(*[c.data_ptr() for c in cols_out])
    eb = (ctypes.c_int32 * max(nc, 1))(*[c.element_size() for c in cols])
    _check(lib().pace_compact(_ptr(offsets), n, int(n_tokens), _ptr(keep), nc, cin, eb, cout,
                              _ptr(offsets_out), _ptr(kept_ids_out), _ptr(n_kept_tokens_out),
                              _ptr(ws), ws.numel(), _stream(dev, stream)), "pace_compact")
    return offsets_out, kept_ids_out, n_kept_tokens_out, cols_out


def pace_validate(tags, offsets, completion, current_version, window_sorted=None, err_out=None,
                  stream=None):
    """Device check of Lemma 1's preconditions. Returns the int32[1] error word tensor."""
    _dev(tags, torch.int32, "tags")
    _dev(offsets, torch.int64, "offsets")
    _dev(completion, torch.int32, "completion")
    dev = tags.device
    W = 0
    if window_sorted is not None:
        _dev(window_sorted, torch.float64, "window_sorted")
        W = window_sorted.numel()
    if err_out is None:
        err_out = torch.empty(1, dtype=torch.int32, device=dev)
    _check(lib().pace_validate(_ptr(tags), _ptr(offsets), offsets.numel() - 1, tags.numel(),
                               _ptr(completion), int(current_version), _ptr(window_sorted), W,
                               _ptr(err_out), _stream(dev, stream)), "pace_validate")
    return err_out


def pace_filter_step(tags, offsets, completion, current_version, occupancy, capacity, cols,
                     prefix_score=None, window_sorted=None, params: Optional[PaceParams] = None,
                     r_hat_prev: float = 0.0, score_out=None, gen_sum_out=None, gen_count_out=None,
                     keep_out=None, reject_ids_out=None, cols_out=None, offsets_out=None,
                     kept_ids_out=None, n_kept_tokens_out=None, workspace=None, stream=None,
                     with_counts=True, _noalloc=False):
    """One whole filter step (Algorithm 1). Returns a dict with budget, r_hat and
    the outputs of pace_score / pace_select / pace_compact (full-capacity tensors;
    reject_ids is cut to the budget)."""
    _dev(tags, torch.int32, "tags")
    _dev(offsets, torch.int64, "offsets")
    _dev(completion, torch.int32, "completion")
    n = offsets.numel() - 1
    nt = tags.numel()
    dev = tags.device
    W = 0
    if prefix_score is not None:
        _dev(prefix_score, torch.float64, "prefix_score")
    if window_sorted is not None:
        _dev(window_sorted, torch.float64, "window_sorted")
        W = window_sorted.numel()
    cols = list(cols)
    for k, c in enumerate(cols):
        if not c.is_cuda or not c.is_contiguous() or c.numel() != nt:
            raise ValueError("column %d must be a contiguous device tensor of n_tokens elements" % k)
    e = lambda k, dt: torch.empty(k, dtype=dt, device=dev)
    score_out = e(n, torch.float64) if score_out is None else score_out
    if with_counts:
        gen_sum_out = e(n, torch.int64) if gen_sum_out is None else gen_sum_out
        gen_count_out = e(n, torch.int64) if gen_count_out is None else gen_count_out
    keep_out = e(n, torch.uint8) if keep_out is None else keep_out
    reject_ids_out = e(max(n, 1), torch.int32) if reject_ids_out is None else reject_ids_out
    cols_out = [torch.empty_like(c) for c in cols] if cols_out is None else cols_out
    offsets_out = e(n + 1, torch.int64) if offsets_out is None else offsets_out
    kept_ids_out = e(max(n, 1), torch.int32) if kept_ids_out is None else kept_ids_out
    n_kept_tokens_out = e(1, torch.int64) if n_kept_tokens_out is None else n_kept_tokens_out
    nc = len(cols)
    cin = (ctypes.c_void_p * max(nc, 1))(*[c.data_ptr() for c in cols])
    cout = (ctypes.c_void_p * max(nc, 1))(*[c.data_ptr() for c in cols_out])
    eb = (ctypes.c_int32 * max(nc, 1))(*[c.element_size() for c in cols])
    rh = ctypes.c_double(float(r_hat_prev))
    b = ctypes.c_int64(0)
    args = (_ptr(tags), _ptr(offsets), n, nt, _ptr(completion), int(current_version),
            _ptr(prefix_score), _ptr(window_sorted), W, int(occupancy), int(capacity),
            ctypes.byref(params) if params is not None else None,
            ctypes.byref(rh), ctypes.byref(b), _ptr(score_out), _ptr(gen_sum_out),
            _ptr(gen_count_out), _ptr(keep_out), _ptr(reject_ids_out), nc, cin, eb,
            cout, _ptr(offsets_out), _ptr(kept_ids_out), _ptr(n_kept_tokens_out))
    if _noalloc:
        _check(lib().pace_filter_step_noalloc(*args, _stream(dev, stream)), "pace_filter_step_noalloc")
    else:
        ws = _workspace(WS_FILTER_STEP, n, nt, dev, workspace)
        _check(lib().pace_filter_step(*args, _ptr(ws), ws.numel(), _stream(dev, stream)), "pace_filter_step")
    return dict(budget=int(b.value), r_hat=float(rh.value), score=score_out, gen_sum=gen_sum_out,
                gen_count=gen_count_out, keep=keep_out, reject_ids=reject_ids_out[: int(b.value)],
                offsets_out=offsets_out, kept_ids=kept_ids_out, n_kept_tokens=n_kept_tokens_out,
                cols_out=cols_out)


def pace_filter_step_noalloc(tags, offsets, completion, current_version, occupancy, capacity, cols, **kw):
    """pace_filter_step with the workspace in the library's fixed device
    scratch (PACE_NOALLOC_SCRATCH_BYTES per device): same arguments (no
    `workspace`) and results. Allocates nothing when every output is passed."""
    if "workspace" in kw:
        raise ValueError("pace_filter_step_noalloc takes no workspace")
    return pace_filter_step(tags, offsets, completion, current_version, occupancy, capacity, cols,
                            _noalloc=True, **kw)


NOALLOC_SCRATCH_BYTES = 16 << 20
ERR_SCRATCH_LIMIT = -5


def pace_group_score(score, group_offsets, group_score_out=None, stream=None):
    """Mean member score of each prompt group (empty group: 0)."""
    _dev(score, torch.float64, "score")
    _dev(group_offsets, torch.int64, "group_offsets")
    ng = group_offsets.numel() - 1
    if group_score_out is None:
        group_score_out = torch.empty(ng, dtype=torch.float64, device=score.device)
    _check(lib().pace_group_score(_ptr(score), score.numel(), _ptr(group_offsets), ng, _ptr(group_score_out),
                                  _stream(score.device, stream)), "pace_group_score")
    return group_score_out


def pace_group_expand(group_offsets, group_keep, n_traj: int, keep_out=None, stream=None):
    """Trajectory keep flags from group keep flags."""
    _dev(group_offsets, torch.int64, "group_offsets")
    _dev(group_keep, torch.uint8, "group_keep")
    ng = group_offsets.numel() - 1
    if keep_out is None:
        keep_out = torch.empty(int(n_traj), dtype=torch.uint8, device=group_keep.device)
    _check(lib().pace_group_expand(_ptr(group_offsets), ng, int(n_traj), _ptr(group_keep), _ptr(keep_out),
                                   _stream(group_keep.device, stream)), "pace_group_expand")
    return keep_out


def pace_validate_groups(group_offsets, n_traj: int, err_out=None, stream=None):
    """Device check of the group offsets; returns the int32 error word tensor."""
    _dev(group_offsets, torch.int64, "group_offsets")
    dev = group_offsets.device
    if err_out is None:
        err_out = torch.empty(1, dtype=torch.int32, device=dev)
    _check(lib().pace_validate_groups(_ptr(group_offsets), group_offsets.numel() - 1, int(n_traj),
                                      _ptr(err_out), _stream(dev, stream)), "pace_validate_groups")
    return err_out


def group_step_buffers(n: int, n_groups: int, cols, device):
    """Output buffers for repeated pace_group_filter_step calls on pools of at
    most n trajectories, n_groups groups and the columns' sizes (pass as
    ``out``): no allocation inside the calls."""
    e = lambda k, dt: torch.empty(k, dtype=dt, device=device)
    return dict(score=e(max(n, 1), torch.float64), gen_sum=e(max(n, 1), torch.int64),
                gen_count=e(max(n, 1), torch.int64), group_score=e(max(n_groups, 1), torch.float64),
                group_keep=e(max(n_groups, 1), torch.uint8), reject_group_ids=e(max(n_groups, 1), torch.int32),
                keep=e(max(n, 1), torch.uint8), cols_out=[torch.empty_like(c) for c in cols],
                offsets_out=e(n + 1, torch.int64), kept_ids=e(max(n, 1), torch.int32),
                n_kept_tokens=e(1, torch.int64))


def pace_group_filter_step(tags, offsets, completion, current_version, group_offsets, occupancy, capacity,
                           cols, prefix_score=None, window_sorted=None, params: Optional[PaceParams] = None,
                           r_hat_prev: float = 0.0, workspace=None, stream=None, out=None):
    """One filter step with prompt groups as the admission unit (occupancy and
    capacity count groups). Returns a dict like pace_filter_step plus
    group_score, group_keep and reject_group_ids (cut to the budget). ``out``:
    buffers from group_step_buffers, written in place of fresh ones."""
    _dev(tags, torch.int32, "tags")
    _dev(offsets, torch.int64, "offsets")
    _dev(completion, torch.int32, "completion")
    _dev(group_offsets, torch.int64, "group_offsets")
    n = offsets.numel() - 1
    ng = group_offsets.numel() - 1
    nt = tags.numel()
    dev = tags.device
    W = 0
    if prefix_score is not None:
        _dev(prefix_score, torch.float64, "prefix_score")
    if window_sorted is not None:
        _dev(window_sorted, torch.float64, "window_sorted")
        W = window_sorted.numel()
    cols = list(cols)
    for k, c in enumerate(cols):
        if not c.is_cuda or not c.is_contiguous() or c.numel() != nt:
            raise ValueError("column %d must be a contiguous device tensor of n_tokens elements" % k)
    o = out if out is not None else group_step_buffers(n, ng, cols, dev)
    if (o["score"].numel() < max(n, 1) or o["group_score"].numel() < max(ng, 1)
            or o["offsets_out"].numel() < n + 1 or len(o["cols_out"]) != len(cols)
            or any(a.numel() < c.numel() or a.dtype != c.dtype or not a.is_contiguous()
                   for a, c in zip(o["cols_out"], cols))):
        raise ValueError("out buffers are too small for this pool, or do not match its columns")
    score_out, gen_sum_out, gen_count_out = o["score"][:n], o["gen_sum"][:n], o["gen_count"][:n]
    group_score_out, group_keep_out = o["group_score"], o["group_keep"]
    reject_group_ids_out = o["reject_group_ids"]
    keep_out = o["keep"]
    cols_out = [a[:nt] for a in o["cols_out"]]
    offsets_out, kept_ids_out = o["offsets_out"][: n + 1], o["kept_ids"]
    n_kept_tokens_out = o["n_kept_tokens"]
    ws = _workspace(WS_FILTER_STEP, max(n, ng), nt, dev, workspace)
    nc = len(cols)
    cin = (ctypes.c_void_p * max(nc, 1))(*[c.data_ptr() for c in cols])
    cout = (ctypes.c_void_p * max(nc, 1))(*[c.data_ptr() for c in cols_out])
    eb = (ctypes.c_int32 * max(nc, 1))(*[c.element_size() for c in cols])
    rh = ctypes.c_double(float(r_hat_prev))
    b = ctypes.c_int64(0)
    _check(lib().pace_group_filter_step(
        _ptr(tags), _ptr(offsets), n, nt, _ptr(completion), int(current_version), _ptr(prefix_score),
        _ptr(window_sorted), W, _ptr(group_offsets), ng, int(occupancy), int(capacity),
        ctypes.byref(params) if params is not None else None, ctypes.byref(rh), ctypes.byref(b),
        _ptr(score_out), _ptr(gen_sum_out), _ptr(gen_count_out), _ptr(group_score_out), _ptr(group_keep_out),
        _ptr(reject_group_ids_out), _ptr(keep_out), nc, cin, eb, cout, _ptr(offsets_out), _ptr(kept_ids_out),
        _ptr(n_kept_tokens_out), _ptr(ws), ws.numel(), _stream(dev, stream)), "pace_group_filter_step")
    return dict(budget=int(b.value), r_hat=float(rh.value), score=score_out, gen_sum=gen_sum_out,
                gen_count=gen_count_out, group_score=group_score_out[:ng], group_keep=group_keep_out[:ng],
                reject_group_ids=reject_group_ids_out[: int(b.value)], keep=keep_out[:n],
                offsets_out=offsets_out, kept_ids=kept_ids_out, n_kept_tokens=n_kept_tokens_out,
                cols_out=cols_out)


class StreamWindow:
    """Device state of the streaming rule's score window: a ring of `cap`
    scores and its {head, count} pair (a fresh window is empty)."""

    def __init__(self, cap=512, device="cuda"):
        self.ring = torch.zeros(cap, dtype=torch.float64, device=device)
        self.state = torch.zeros(2, dtype=torch.int64, device=device)
        self.cap = cap


def pace_stream_admit(score, r_hat: float, window: StreamWindow, batch_size: int,
                      params: Optional[PaceParams] = None, status_out=None, keep_out=None,
                      reject_ids_out=None, kappa_out=None, counts_out=None, stream=None):
    """One step of the streaming rule. Returns (status, keep, reject_ids, kappa,
    counts) as device tensors; counts = [drawn, retained, rejected]."""
    _dev(score, torch.float64, "score")
    n = score.numel()
    dev = score.device
    e = lambda k, dt: torch.empty(k, dtype=dt, device=dev)
    status_out = e(max(n, 1), torch.uint8) if status_out is None else status_out
    keep_out = e(max(n, 1), torch.uint8) if keep_out is None else keep_out
    reject_ids_out = e(max(n, 1), torch.int32) if reject_ids_out is None else reject_ids_out
    kappa_out = e(1, torch.float64) if kappa_out is None else kappa_out
    counts_out = e(3, torch.int64) if counts_out is None else counts_out
    _check(lib().pace_stream_admit(_ptr(score), n, float(r_hat), ctypes.byref(params) if params is not None else None,
                                   int(batch_size), _ptr(window.ring), window.cap, _ptr(window.state),
                                   _ptr(status_out), _ptr(keep_out), _ptr(reject_ids_out), _ptr(kappa_out),
                                   _ptr(counts_out), _stream(dev, stream)), "pace_stream_admit")
    return status_out[:n], keep_out[:n], reject_ids_out, kappa_out, counts_out


def stream_step_buffers(n: int, n_tokens: int, col_dtypes: Sequence[torch.dtype], device):
    """Preallocated outputs for repeated pace_stream_step calls."""
    e = lambda k, dt: torch.empty(k, dtype=dt, device=device)
    return dict(score=e(max(n, 1), torch.float64), gen_sum=e(max(n, 1), torch.int64),
                gen_count=e(max(n, 1), torch.int64), status=e(max(n, 1), torch.uint8),
                keep=e(max(n, 1), torch.uint8), reject_ids=e(max(n, 1), torch.int32),
                kappa=e(1, torch.float64), counts=e(3, torch.int64),
                cols_out=[e(max(n_tokens, 1), dt) for dt in col_dtypes], offsets_out=e(n + 1, torch.int64),
                kept_ids=e(max(n, 1), torch.int32), n_kept_tokens=e(1, torch.int64),
                workspace=e(max(pace_workspace_bytes(WS_FILTER_STEP, n, n_tokens), 256), torch.uint8))


def pace_stream_step(tags, offsets, completion, current_version, occupancy, capacity, cols,
                     window: StreamWindow, batch_size: int, prefix_score=None, window_sorted=None,
                     params: Optional[PaceParams] = None, r_hat_prev: float = 0.0, buffers=None, stream=None):
    """One trainer step under the streaming rule (budget, score, draw, compact
    of the retained batch). Returns (buffers dict, r_hat)."""
    _dev(tags, torch.int32, "tags")
    _dev(offsets, torch.int64, "offsets")
    _dev(completion, torch.int32, "completion")
    n = offsets.numel() - 1
    nt = tags.numel()
    dev = tags.device
    W = 0
    if prefix_score is not None:
        _dev(prefix_score, torch.float64, "prefix_score")
    if window_sorted is not None:
        _dev(window_sorted, torch.float64, "window_sorted")
        W = window_sorted.numel()
    cols = list(cols)
    b = buffers if buffers is not None else stream_step_buffers(n, nt, [c.dtype for c in cols], dev)
    nc = len(cols)
    cin = (ctypes.c_void_p * max(nc, 1))(*[c.data_ptr() for c in cols])
    cout = (ctypes.c_void_p * max(nc, 1))(*[c.data_ptr() for c in b["cols_out"]])
    eb = (ctypes.c_int32 * max(nc, 1))(*[c.element_size() for c in cols])
    rh = ctypes.c_double(float(r_hat_prev))
    ws = b["workspace"]
    _check(lib().pace_stream_step(
        _ptr(tags), _ptr(offsets), n, nt, _ptr(completion), int(current_version), _ptr(prefix_score),
        _ptr(window_sorted), W, int(occupancy), int(capacity), ctypes.byref(params) if params is not None else None,
        ctypes.byref(rh), int(batch_size), _ptr(window.ring), window.cap, _ptr(window.state), _ptr(b["score"]),
        _ptr(b["gen_sum"]), _ptr(b["gen_count"]), _ptr(b["status"]), _ptr(b["keep"]), _ptr(b["reject_ids"]),
        _ptr(b["kappa"]), _ptr(b["counts"]), nc, cin, eb, cout, _ptr(b["offsets_out"]), _ptr(b["kept_ids"]),
        _ptr(b["n_kept_tokens"]), _ptr(ws), ws.numel(), _stream(dev, stream)), "pace_stream_step")
    return b, float(rh.value)


def pace_prefix_score(lp_new, lp_behavior, prefix_offsets, tags=None, cap: int = 1024, min_tokens: int = 32,
                      s_pre_out=None, stream=None):
    """Eq. (5) per rescored prefix; NaN when fewer than min_tokens tokens count."""
    _dev(lp_new, torch.float32, "lp_new")
    _dev(lp_behavior, torch.float32, "lp_behavior")
    _dev(prefix_offsets, torch.int64, "prefix_offsets")
    if tags is not None:
        _dev(tags, torch.int32, "tags")
    n = prefix_offsets.numel() - 1
    if s_pre_out is None:
        s_pre_out = torch.empty(max(n, 1), dtype=torch.float64, device=lp_new.device)
    _check(lib().pace_prefix_score(_ptr(lp_new), _ptr(lp_behavior), _ptr(tags), _ptr(prefix_offsets), n,
                                   lp_new.numel(), int(cap), int(min_tokens), _ptr(s_pre_out),
                                   _stream(lp_new.device, stream)), "pace_prefix_score")
    return s_pre_out[:n]


def pace_stale_k(gen_sum, gen_count, completion, current_version, k: int, keep_out=None, lag_out=None,
                 with_lag=True, stream=None):
    """Stale-k admission (Eq. (1) lag <= k). Returns (keep u8[n], lag f64[n] or None)."""
    _dev(gen_sum, torch.int64, "gen_sum")
    _dev(gen_count, torch.int64, "gen_count")
    _dev(completion, torch.int32, "completion")
    n = completion.numel()
    dev = completion.device
    keep_out = torch.empty(max(n, 1), dtype=torch.uint8, device=dev) if keep_out is None else keep_out
    if with_lag and lag_out is None:
        lag_out = torch.empty(max(n, 1), dtype=torch.float64, device=dev)
    _check(lib().pace_stale_k(_ptr(gen_sum), _ptr(gen_count), _ptr(completion), int(current_version), n, int(k),
                              _ptr(keep_out), _ptr(lag_out), _stream(dev, stream)), "pace_stale_k")
    return keep_out[:n], (lag_out[:n] if lag_out is not None else None)


def pace_diagnostics(score, gen_sum, gen_count, completion, current_version, keep, edges, hist_out=None,
                     totals_out=None, stream=None):
    """Kept/rejected staleness histograms. edges: f64 [3, nbins+1] device tensor.
    Returns (hist int64 [3, 2, nbins+2], totals int64 [2, 4])."""
    _dev(score, torch.float64, "score")
    _dev(edges, torch.float64, "edges")
    n = score.numel()
    nbins = edges.shape[1] - 1
    dev = score.device
    hist_out = torch.empty((3, 2, nbins + 2), dtype=torch.int64, device=dev) if hist_out is None else hist_out
    totals_out = torch.empty((2, 4), dtype=torch.int64, device=dev) if totals_out is None else totals_out
    _check(lib().pace_diagnostics(_ptr(score), _ptr(gen_sum), _ptr(gen_count), _ptr(completion),
                                  int(current_version), _ptr(keep), n, _ptr(edges), int(nbins), _ptr(hist_out),
                                  _ptr(totals_out), _stream(dev, stream)), "pace_diagnostics")
    return hist_out, totals_out


def pace_time_next_kernel(phase: int, start=None, stop=None):
    """Arm a one-shot timer on the next kernel of `phase` launched from this
    thread. start/stop are torch.cuda.Event(enable_timing=True) objects that
    have been recorded once (so that their HIP events exist); None for both
    disarms. Afterwards start.elapsed_time(stop) is that kernel's own time."""
    def handle(ev):
        if ev is None:
            return None
        if not ev.cuda_event:
            raise PaceError(-1, "pace_time_next_kernel (record the event once before arming it)")
        return ev.cuda_event
    _check(_lib.lib().pace_time_next_kernel(int(phase), handle(start), handle(stop)), "pace_time_next_kernel")


class FilterStep:
    """Preallocated buffers for repeated filter steps over pools of one shape
    (n trajectories, n_tokens tokens, the given payload columns). ``run``
    enqueues score -> budget -> select -> compact on the current stream with no
    allocation and no host synchronisation."""

    def __init__(self, n: int, n_tokens: int, col_dtypes: Sequence[torch.dtype], device,
                 params: Optional[PaceParams] = None):
        dev = torch.device(device)
        self.n, self.n_tokens, self.device = n, n_tokens, dev
        self.params = params if params is not None else default_params()
        e = lambda k, dt: torch.empty(k, dtype=dt, device=dev)
        self.score = e(max(n, 1), torch.float64)
        self.gen_sum = e(max(n, 1), torch.int64)
        self.gen_count = e(max(n, 1), torch.int64)
        self.keep = e(max(n, 1), torch.uint8)
        self.reject_ids = e(max(n, 1), torch.int32)
        self.offsets_out = e(n + 1, torch.int64)
        self.kept_ids = e(max(n, 1), torch.int32)
        self.n_kept_tokens = e(1, torch.int64)
        self.cols_out = [e(max(n_tokens, 1), dt) for dt in col_dtypes]
        self.ws = [e(max(pace_workspace_bytes(w, n, n_tokens), 256), torch.uint8)
                   for w in (WS_SCORE, WS_SELECT, WS_COMPACT, WS_FILTER_STEP)]
        self.r_hat = 0.0
        self.budget = 0

    def score_only(self, tags, offsets, completion, V, prefix=None, window=None, stream=None):
        return pace_score(tags, offsets, completion, V, prefix, window, self.params,
                          self.score[: self.n], self.gen_sum[: self.n], self.gen_count[: self.n],
                          self.ws[0], stream)

    def run(self, tags, offsets, completion, V, occupancy, capacity, cols, prefix=None,
            window=None, stream=None, fused=True):
        """fused: one pace_filter_step call; otherwise the four calls in sequence."""
        if fused:
            r = pace_filter_step(tags, offsets, completion, V, occupancy, capacity, cols, prefix, window,
                                 self.params, self.r_hat, self.score[: self.n], self.gen_sum[: self.n],
                                 self.gen_count[: self.n], self.keep[: self.n], self.reject_ids,
                                 [c[: self.n_tokens] for c in self.cols_out], self.offsets_out,
                                 self.kept_ids, self.n_kept_tokens, self.ws[3], stream)
            self.budget, self.r_hat = r["budget"], r["r_hat"]
            return self
        self.score_only(tags, offsets, completion, V, prefix, window, stream)
        self.budget, self.r_hat = pace_budget(occupancy, capacity, self.params, self.r_hat)
        pace_select(self.score[: self.n], self.budget, self.keep[: self.n], self.reject_ids,
                    self.ws[1], stream)
        pace_compact(offsets, self.keep[: self.n], cols, [c[: self.n_tokens] for c in self.cols_out],
                     self.offsets_out, self.kept_ids, self.n_kept_tokens, self.ws[2], stream,
                     n_tokens=self.n_tokens)
        return self
