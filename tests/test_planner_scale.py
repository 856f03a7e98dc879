"""Planner complexity (Sec. 3.3: the dynamic program and Recover run in
time linear in the tree), on the CPU through the C ABI.

A chain of 10^6 segments (every segment a single child of the previous one)
and a star of 10^5 leaves under one root are planned within fixed time
bounds, and ten times more segments take at most about ten times longer
(a quadratic planner would take a hundred).  Lengths are drawn so that forks
fall at unaligned offsets and the star's leaves all replay part of a chunk.
"""
import ctypes as C
import time

import numpy as np
import pytest


@pytest.fixture(scope="module")
def L():
    from paper_2608_28158_amd import _lib
    return _lib.lib()


def plan_seconds(L, parent, seg_len, reps=3):
    from paper_2608_28158_amd import _lib
    parent = np.ascontiguousarray(parent, np.int32)
    seg_len = np.ascontiguousarray(seg_len, np.int64)
    best = None
    for _ in range(reps):
        h = C.c_void_p()
        t0 = time.perf_counter()
        rc = L.harts_plan(len(parent), parent.ctypes.data_as(_lib._I32),
                          seg_len.ctypes.data_as(_lib._I64), 64, C.byref(h))
        dt = time.perf_counter() - t0
        assert rc == _lib.HARTS_OK, _lib.last_error()
        info = _lib.PlanInfo()
        assert L.harts_plan_get_info(h, C.byref(info)) == _lib.HARTS_OK
        L.harts_plan_free(h)
        best = dt if best is None else min(best, dt)
    return best, info


def chain(n, rng):
    return np.arange(-1, n - 1), rng.integers(1, 8, size=n)


def star(n, rng):
    parent = np.zeros(n + 1, np.int64)
    parent[0] = -1
    seg_len = rng.integers(1, 200, size=n + 1)
    seg_len[0] = 1000                                  # forks 40 rows into a chunk
    return parent, seg_len


def test_chain_of_a_million_segments(L):
    rng = np.random.default_rng(0)
    t_small, _ = plan_seconds(L, *chain(10 ** 5, rng))
    t_big, info = plan_seconds(L, *chain(10 ** 6, rng))
    print(f"chain: 1e5 {t_small * 1e3:.1f} ms, 1e6 {t_big * 1e3:.1f} ms")
    assert info.n_rounds == 1 and info.n_seq == 1 and info.R == 0
    assert t_big < 3.0
    assert t_big < 25 * max(t_small, 1e-3)


def test_star_of_a_hundred_thousand_leaves(L):
    rng = np.random.default_rng(1)
    t_small, _ = plan_seconds(L, *star(10 ** 4, rng))
    t_big, info = plan_seconds(L, *star(10 ** 5, rng))
    print(f"star: 1e4 {t_small * 1e3:.1f} ms, 1e5 {t_big * 1e3:.1f} ms")
    # every leaf but the continued one starts a round later from S_960 and
    # replays rows 960..999 of the root (eq. mandatory-replay)
    assert info.n_rounds == 2 and info.n_seq == 10 ** 5
    assert info.R == (10 ** 5 - 1) * 40
    assert t_big < 2.0
    assert t_big < 25 * max(t_small, 1e-3)
