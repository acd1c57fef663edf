"""CPU tests of the C ABI: the library loads, exports every entry point that
include/pace.h declares, and its host-only logic (defaults, workspace sizing,
the budget of Eq. (3)-(4), host-side argument checks) behaves as documented.
No GPU call is made here: every argument-error case returns before any
launch."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pace.h")


@pytest.fixture(scope="module")
def L():
    from paper_2609_36830_amd import _lib
    if not os.path.exists(_lib.library_path):
        from paper_2609_36830_amd import build
        build.build()
    return _lib.lib()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|void|const char \*)\s*\**\s*(pace_\w+)\s*\(", text, re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for f in ("pace_score", "pace_budget", "pace_select", "pace_compact", "pace_validate",
              "pace_filter_step", "pace_workspace_bytes", "pace_default_params", "pace_strerror"):
        assert f in names


def test_library_exports_every_declared_symbol(L):
    from paper_2609_36830_amd import _lib
    names = declared_functions()
    for f in names:
        assert hasattr(L, f), f
    assert sorted(n for n, _, _ in _lib.SIGNATURES) == names


def test_default_params(L):
    import paper_2609_36830_amd as pace
    p = pace.default_params()
    assert (p.w_wait, p.gamma, p.window_min, p.beta, p.r_max) == (1.0, 4, 32, 0.0, 0.9)


def test_strerror(L):
    assert L.pace_strerror(0) == b"ok"
    assert b"argument" in L.pace_strerror(-1)
    assert b"workspace" in L.pace_strerror(-2)


def test_workspace_sizes(L):
    import paper_2609_36830_amd as pace
    for which in (0, 1, 2, 3):
        for n, nt in ((0, 0), (1, 1), (4096, 50_000_000), (20000, 1000)):
            b = pace.pace_workspace_bytes(which, n, nt)
            assert b >= 256 and b % 256 == 0
    with pytest.raises(pace.PaceError):
        pace.pace_workspace_bytes(4, 1, 1)
    with pytest.raises(pace.PaceError):
        pace.pace_workspace_bytes(0, -1, 1)


def test_budget_bit_exact_vs_oracle(L):
    """pace_budget runs on the host: compare it with the oracle everywhere."""
    import paper_2609_36830_amd as pace
    rng = np.random.default_rng(11)
    cases = [(64, 48, 0.0), (4096, 1365, 0.0), (1024, 683, 0.0), (2048, 1575, 0.0), (100, 0, 0.0),
             (0, 0, 0.0), (1, 0, 0.5), (5, 5, 0.9)]
    for _ in range(3000):
        N = int(rng.integers(0, 100000))
        cases.append((N, int(rng.integers(0, N + 5)), float(rng.choice([0.0, 0.5, 0.9, 0.99, rng.random()]))))
    for N, Nt, beta in cases:
        rh_o = rh_g = float(rng.random()) if beta > 0 else 0.0
        for step in range(3):
            bo, rh_o = oracle.budget(N, Nt, rh_o, beta, 0.9)
            bg, rh_g = pace.pace_budget(N, Nt, pace.default_params(beta=beta), rh_g)
            assert bo == bg and rh_o == rh_g, (N, Nt, beta, step)


def test_budget_argument_errors(L):
    import paper_2609_36830_amd as pace
    for kw, N, Nt, rh in (({"beta": 1.0}, 10, 5, 0.0), ({"beta": -0.1}, 10, 5, 0.0),
                          ({"r_max": 1.5}, 10, 5, 0.0), ({}, -1, 5, 0.0), ({}, 10, -1, 0.0),
                          ({}, 10, 5, float("nan")), ({}, 10, 5, -1.0)):
        with pytest.raises(pace.PaceError) as e:
            pace.pace_budget(N, Nt, pace.default_params(**kw), rh)
        assert e.value.code == -1


FAKE = 0x100000   # aligned, never dereferenced: each call below fails its host checks first


def test_score_host_argument_errors(L):
    import paper_2609_36830_amd as pace
    p = pace.default_params()
    P = ctypes.byref(p)

    def call(tags=FAKE, off=FAKE, n=4, nt=100, comp=FAKE, V=10, pre=None, win=None, W=0, params=P,
             out=FAKE, ws=FAKE, wsb=0):
        return L.pace_score(tags, off, n, nt, comp, V, pre, win, W, params, out, None, None, ws, wsb, None)

    assert call(off=None) == -1
    assert call(n=-1) == -1
    assert call(out=None) == -1
    assert call(tags=FAKE + 2) == -1          # not 4-byte aligned
    assert call(V=-1) == -1
    assert call(V=2 ** 31 - 1) == -1
    assert call(win=None, W=5) == -1
    p.gamma = 5
    assert call() == -1
    p.gamma = 4
    assert call(win=FAKE, W=10000) == -1      # 10000^4 >= 2^53
    p.w_wait = float("nan")
    assert call() == -1
    p.w_wait = 1.0
    assert call(ws=None) == -2
    assert call(ws=FAKE + 64, wsb=1 << 30) == -2   # misaligned workspace
    assert call(wsb=16) == -2                   # too small


def test_window_power_bound_matches_oracle(L):
    """pace_score and the oracle accept and reject the same (window size,
    gamma) pairs: the exact form of Eq. (9) needs W^gamma < 2^53. An accepted
    pair gets as far as the workspace check (-2), a rejected one stops at the
    argument check (-1); the oracle returns a score or its argument error."""
    import paper_2609_36830_amd as pace
    from tests.test_oracle_pins import WINDOW_POWER_BOUNDS, _score_rc
    p = pace.default_params()

    def gpu_rc(W, gamma):
        p.gamma = gamma
        return L.pace_score(FAKE, FAKE, 1, 1, FAKE, 5, None, FAKE, W, ctypes.byref(p), FAKE, None, None,
                            FAKE, 0, None)

    grid = []
    for gam, Wmax in WINDOW_POWER_BOUNDS.items():
        grid += [(Wmax - 1, gam), (Wmax, gam), (Wmax + 1, gam), (Wmax + 2, gam)]
    grid += [(W, 4) for W in (1, 512, 4096, 55108, 55109, 55110, 65536)]
    grid += [(W, g) for g in (1, 2, 3) for W in (1, 512, 65536)]
    for W, gam in grid:
        ref = _score_rc(W, gam)
        accepted = not isinstance(ref, int)
        assert accepted or ref == oracle.ERR_ARG
        assert gpu_rc(W, gam) == (-2 if accepted else -1), (W, gam)
    # sizes no host array can hold: only the library's check is exercised
    for W, gam, acc in ((2 ** 53 - 1, 1, True), (2 ** 53, 1, False), (2 ** 40, 4, False), (2 ** 62, 2, False),
                        (2 ** 31, 3, False)):
        assert gpu_rc(W, gam) == (-2 if acc else -1), (W, gam)


def test_filter_step_host_argument_errors(L):
    """pace_filter_step rejects bad arguments before enqueuing, r_hat untouched."""
    import paper_2609_36830_amd as pace
    p = pace.default_params()
    rh = ctypes.c_double(0.25)
    b = ctypes.c_int64(-7)
    cols = (ctypes.c_void_p * 1)(FAKE)
    e4 = (ctypes.c_int32 * 1)(4)

    def call(occ=10, cap=5, ws=FAKE, wsb=1 << 30, keep=FAKE, rej=FAKE, beta=0.0, n=4):
        p.beta = beta
        return L.pace_filter_step(FAKE, FAKE, n, 100, FAKE, 10, None, None, 0, occ, cap, ctypes.byref(p),
                                  ctypes.byref(rh), ctypes.byref(b), FAKE, None, None, keep, rej, 1, cols, e4,
                                  cols, FAKE, FAKE, FAKE, ws, wsb, None)

    assert call(keep=None) == -1
    assert call(beta=1.5) == -1
    assert call(occ=-1) == -1
    assert call(occ=100, cap=0, n=4) == -1      # budget 90 > 4 trajectories
    assert call(rej=None) == -1
    assert call(ws=None) == -2
    assert call(wsb=64) == -2
    assert rh.value == 0.25 and b.value == -7


def test_filter_step_noalloc_limit(L):
    """The scratch variant refuses a pool whose workspace exceeds its fixed
    array, after the argument checks and before any launch."""
    import paper_2609_36830_amd as pace
    rh = ctypes.c_double(0.0)
    b = ctypes.c_int64(0)
    cols = (ctypes.c_void_p * 1)(FAKE)
    e4 = (ctypes.c_int32 * 1)(4)

    def call(n, nt, keep=FAKE):
        return L.pace_filter_step_noalloc(FAKE, FAKE, n, nt, FAKE, 10, None, None, 0, 10, 5, None,
                                          ctypes.byref(rh), ctypes.byref(b), FAKE, None, None, keep, FAKE, 1,
                                          cols, e4, cols, FAKE, FAKE, FAKE, None)

    assert pace.pace_workspace_bytes(3, 1 << 22, 1000) > pace.NOALLOC_SCRATCH_BYTES
    assert call(1 << 22, 1000) == pace.ERR_SCRATCH_LIMIT
    assert pace.pace_workspace_bytes(3, 4096, 4 * 10 ** 9) > pace.NOALLOC_SCRATCH_BYTES
    assert call(4096, 4 * 10 ** 9) == pace.ERR_SCRATCH_LIMIT
    assert call(1 << 22, 1000, keep=None) == -1          # argument errors come first
    assert L.pace_strerror(pace.ERR_SCRATCH_LIMIT) == b"pool too large for the fixed device scratch"


def test_select_and_compact_host_argument_errors(L):
    assert L.pace_select(FAKE, 10, 11, FAKE, FAKE, FAKE, 1 << 20, None) == -1     # budget > n
    assert L.pace_select(FAKE, 10, -1, FAKE, FAKE, FAKE, 1 << 20, None) == -1
    assert L.pace_select(FAKE, 10, 3, FAKE, None, FAKE, 1 << 20, None) == -1      # no reject ids
    assert L.pace_select(FAKE, 10, 3, FAKE, FAKE, FAKE, 0, None) == -2
    cols = (ctypes.c_void_p * 1)(FAKE)
    bad_e = (ctypes.c_int32 * 1)(3)
    ok_e = (ctypes.c_int32 * 1)(4)
    assert L.pace_compact(FAKE, 10, 100, FAKE, 1, cols, bad_e, cols, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == -1
    assert L.pace_compact(FAKE, 10, 100, FAKE, 9, cols, ok_e, cols, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == -1
    assert L.pace_compact(None, 10, 100, FAKE, 1, cols, ok_e, cols, FAKE, FAKE, FAKE, FAKE, 1 << 20, None) == -1
    assert L.pace_compact(FAKE, 10, 100, FAKE, 1, cols, ok_e, cols, FAKE, FAKE, FAKE, FAKE, 8, None) == -2
    assert L.pace_validate(FAKE, None, 10, 100, FAKE, 5, None, 0, FAKE, None) == -1


def test_time_next_kernel_arguments(L):
    assert L.pace_time_next_kernel(-1, None, None) == -1
    assert L.pace_time_next_kernel(7, None, None) == -1
    assert L.pace_time_next_kernel(0, FAKE, None) == -1
    assert L.pace_time_next_kernel(0, None, FAKE) == -1
    # arm then disarm: nothing is launched, so the fake handles are never used
    assert L.pace_time_next_kernel(3, FAKE, FAKE) == 0
    for phase in range(7):
        assert L.pace_time_next_kernel(phase, None, None) == 0


def test_group_host_argument_errors(L):
    assert L.pace_group_score(FAKE, 10, None, 3, FAKE, None) == -1
    assert L.pace_group_score(FAKE, 10, FAKE, -1, FAKE, None) == -1
    assert L.pace_group_score(FAKE, 10, FAKE + 4, 3, FAKE, None) == -1       # misaligned offsets
    assert L.pace_group_score(None, 10, FAKE, 3, FAKE, None) == -1
    assert L.pace_group_expand(FAKE, 3, 10, None, FAKE, None) == -1
    assert L.pace_group_expand(FAKE, 3, 10, FAKE, None, None) == -1
    assert L.pace_validate_groups(FAKE, 3, 10, None, None) == -1
    assert L.pace_validate_groups(FAKE, 3, -1, FAKE, None) == -1
    import paper_2609_36830_amd as pace
    p = pace.default_params()
    rh = ctypes.c_double(0.5)
    b = ctypes.c_int64(-3)
    cols = (ctypes.c_void_p * 1)(FAKE)
    e4 = (ctypes.c_int32 * 1)(4)

    def call(go=FAKE, ng=4, occ=6, cap=4, gscore=FAKE, ws=FAKE, wsb=1 << 30, grej=FAKE):
        return L.pace_group_filter_step(FAKE, FAKE, 20, 100, FAKE, 10, None, None, 0, go, ng, occ, cap,
                                        ctypes.byref(p), ctypes.byref(rh), ctypes.byref(b), FAKE, None, None,
                                        gscore, FAKE, grej, FAKE, 1, cols, e4, cols, FAKE, FAKE, FAKE, ws, wsb,
                                        None)

    assert call(go=None) == -1
    assert call(gscore=None) == -1
    assert call(occ=100, cap=0) == -1          # budget 90 > 4 groups
    assert call(grej=None) == -1               # budget 4 > 0 needs reject ids
    assert call(ws=None) == -2
    assert call(wsb=64) == -2
    assert rh.value == 0.5 and b.value == -3


def test_stream_admit_host_argument_errors(L):
    def call(n=10, r_hat=0.5, B=4, ring=FAKE, cap=512, state=FAKE, status=FAKE):
        return L.pace_stream_admit(FAKE, n, r_hat, None, B, ring, cap, state, status, FAKE, FAKE, FAKE, FAKE, None)

    assert call(cap=0) == -1
    assert call(cap=1025) == -1
    assert call(r_hat=float("nan")) == -1
    assert call(r_hat=-0.1) == -1
    assert call(B=-1) == -1
    assert call(n=-1) == -1
    assert call(ring=None) == -1
    assert call(state=None) == -1
    assert call(status=None) == -1


def test_stream_step_host_argument_errors(L):
    rh = ctypes.c_double(0.25)
    cols = (ctypes.c_void_p * 1)(FAKE)
    e4 = (ctypes.c_int32 * 1)(4)

    def call(cap=512, B=10, ws=FAKE, wsb=1 << 30, ring=FAKE):
        return L.pace_stream_step(FAKE, FAKE, 20, 100, FAKE, 10, None, None, 0, 30, 10, None, ctypes.byref(rh), B,
                                  ring, cap, FAKE, FAKE, None, None, FAKE, FAKE, FAKE, FAKE, FAKE, 1, cols, e4,
                                  cols, FAKE, FAKE, FAKE, ws, wsb, None)

    assert call(cap=0) == -1
    assert call(cap=2048) == -1
    assert call(B=-1) == -1
    assert call(ring=None) == -1
    assert call(ws=None) == -2
    assert call(wsb=64) == -2
    assert rh.value == 0.25


def test_prefix_score_host_argument_errors(L):
    assert L.pace_prefix_score(FAKE, FAKE, None, None, 3, 10, 1024, 32, FAKE, None) == -1
    assert L.pace_prefix_score(FAKE, FAKE, None, FAKE, -1, 10, 1024, 32, FAKE, None) == -1
    assert L.pace_prefix_score(FAKE, FAKE, None, FAKE, 3, 10, -1, 32, FAKE, None) == -1
    assert L.pace_prefix_score(FAKE, FAKE, None, FAKE, 3, 10, 1024, -1, FAKE, None) == -1
    assert L.pace_prefix_score(None, FAKE, None, FAKE, 3, 10, 1024, 32, FAKE, None) == -1
    assert L.pace_prefix_score(FAKE + 2, FAKE, None, FAKE, 3, 10, 1024, 32, FAKE, None) == -1
    assert L.pace_prefix_score(FAKE, FAKE, None, FAKE, 3, 10, 1024, 32, None, None) == -1


def test_stale_k_and_diagnostics_host_argument_errors(L):
    assert L.pace_stale_k(FAKE, FAKE, FAKE, 10, 5, -1, FAKE, None, None) == -1
    assert L.pace_stale_k(FAKE, FAKE, FAKE, 10, 5, 2 ** 31, FAKE, None, None) == -1
    assert L.pace_stale_k(None, FAKE, FAKE, 10, 5, 3, FAKE, None, None) == -1
    assert L.pace_stale_k(FAKE, FAKE, FAKE, 10, 5, 3, None, None, None) == -1
    assert L.pace_diagnostics(FAKE, FAKE, FAKE, FAKE, 10, FAKE, 5, FAKE, 0, FAKE, FAKE, None) == -1
    assert L.pace_diagnostics(FAKE, FAKE, FAKE, FAKE, 10, FAKE, 5, FAKE, 1025, FAKE, FAKE, None) == -1
    assert L.pace_diagnostics(FAKE, FAKE, FAKE, FAKE, 10, FAKE, 5, None, 8, FAKE, FAKE, None) == -1
    assert L.pace_diagnostics(FAKE, FAKE, FAKE, FAKE, 10, None, 5, FAKE, 8, FAKE, FAKE, None) == -1
