"""The C ABI on the CPU: libharts loads and exports every symbol that
include/harts.h declares, its host planner (Algorithm "minimum-call",
Sec. 3.3) is bit-exact against the oracle planner, and argument validation
returns the documented error codes before anything touches a device.

Nothing here launches a kernel; the library's device calls are exercised by
the GPU parity tests.
"""
import ctypes as C
import os
import re

import numpy as np
import pytest

from oracle.plan_ref import plan_ref
from workloads.trees import figure1_forest, forest_for_config

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def L():
    from paper_2608_28158_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        from paper_2608_28158_amd.build import build
        build()
    return _lib.lib()


def header_functions():
    text = open(os.path.join(ROOT, "include", "harts.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|void|const char\s*\*)\s+(harts_\w+)\s*\(",
                                 text, flags=re.M)))


def test_library_exports_every_declared_symbol(L):
    from paper_2608_28158_amd import _lib
    declared = header_functions()
    assert len(declared) >= 15
    assert sorted(_lib.EXPORTS) == declared
    for name in declared:
        assert getattr(L, name) is not None, name


# ---------------------------------------------------------------------------
# planner parity: every exported array equals the oracle planner's
# ---------------------------------------------------------------------------
ORACLE_NAME = {"tree_calls": "K_tree"}
SCALARS = ("n_seq", "n_slots", "n_trees", "n_bank", "n_leaves", "C", "S", "R")


def compare_plans(parent, seg_len, B):
    from paper_2608_28158_amd.plan import HartsPlan
    got = HartsPlan(parent, seg_len, B)
    ref = plan_ref(np.asarray(parent), np.asarray(seg_len), B)
    assert got["n_rounds"] == ref["K"]
    for k in SCALARS:
        assert got[k] == ref[k], k
    for name in got.arrays:
        a, b = got.arrays[name], np.asarray(ref[ORACLE_NAME.get(name, name)])
        assert a.shape == b.shape and np.array_equal(a, b.astype(a.dtype)), name
    got.close()


def random_forest(rng, n_seg, max_len):
    parent = [-1]
    for v in range(1, n_seg):
        parent.append(-1 if rng.random() < 0.1 else int(rng.integers(0, v)))
    seg_len = rng.integers(1, max_len + 1, size=n_seg)
    return np.array(parent, np.int32), seg_len.astype(np.int64)


def test_planner_matches_oracle_on_figure1(L):
    f = figure1_forest()
    for B in (64, 2, 3, 7):
        compare_plans(f.parent, f.seg_len, B)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_planner_matches_oracle_on_workloads(L, cfg):
    f, _, _ = forest_for_config(cfg)
    compare_plans(f.parent, f.seg_len, 64)


@pytest.mark.parametrize("B", [1, 2, 3, 4, 5, 8, 64])
def test_planner_matches_oracle_random(L, B):
    rng = np.random.default_rng(100 + B)
    for _ in range(60):
        n = int(rng.integers(1, 40))
        parent, seg_len = random_forest(rng, n, max_len=3 * B + 2)
        compare_plans(parent, seg_len, B)


def test_planner_figure1_worked_plan(L):
    """The hand-derived plan of Figure 1 (lengths of config 0, B = 64)."""
    from paper_2608_28158_amd.plan import HartsPlan
    f = figure1_forest()
    p = HartsPlan(f.parent, f.seg_len, 64)
    assert p["n_rounds"] == 2 and p["C"] == 481 and p["S"] == 958 and p["R"] == 29
    assert list(p["seg_mult"]) == [3, 2, 1, 1, 1]
    p.close()


# ---------------------------------------------------------------------------
# error paths (host validation only)
# ---------------------------------------------------------------------------
def plan_rc(L, parent, seg_len, chunk, n=None):
    parent = np.ascontiguousarray(parent, np.int32)
    seg_len = np.ascontiguousarray(seg_len, np.int64)
    h = C.c_void_p()
    rc = L.harts_plan(len(parent) if n is None else n,
                      parent.ctypes.data_as(C.POINTER(C.c_int32)),
                      seg_len.ctypes.data_as(C.POINTER(C.c_int64)), chunk, C.byref(h))
    if rc == 0:
        L.harts_plan_free(h)
    return rc


def test_plan_rejects_bad_forests(L):
    from paper_2608_28158_amd._lib import HARTS_EINVAL, HARTS_OK
    assert plan_rc(L, [-1, 0], [3, 4], 64) == HARTS_OK
    assert plan_rc(L, [-1, 0], [3, 4], 0) == HARTS_EINVAL          # chunk < 1
    assert plan_rc(L, [-1, 0], [3, 4], 64, n=0) == HARTS_EINVAL    # no segments
    assert plan_rc(L, [-1, 5], [3, 4], 64) == HARTS_EINVAL         # parent out of range
    assert plan_rc(L, [-1, 1], [3, 4], 64) == HARTS_EINVAL         # own parent
    assert plan_rc(L, [2, 0, 1], [3, 4, 5], 64) == HARTS_EINVAL    # cycle, no root
    assert plan_rc(L, [-1, 0], [3, 0], 64) == HARTS_EINVAL         # empty segment
    assert plan_rc(L, [-1, 0], [3, -2], 64) == HARTS_EINVAL        # negative length
    msg = L.harts_last_error()
    assert msg and len(msg) > 0
    h = C.c_void_p()
    assert L.harts_plan(2, None, None, 64, C.byref(h)) == HARTS_EINVAL


def test_device_calls_validate_before_launch(L):
    from paper_2608_28158_amd import _lib
    from paper_2608_28158_amd.plan import HartsPlan
    f = figure1_forest()
    p = HartsPlan(f.parent, f.seg_len, 64)
    sz = C.c_size_t()
    ws = L.harts_la_workspace_size
    assert ws(p.handle, 0, 0, _lib.HARTS_BF16, 16, 128, 128, 0, C.byref(sz)) == _lib.HARTS_OK
    assert sz.value > 0
    assert ws(p.handle, 0, 0, 7, 16, 128, 128, 0, C.byref(sz)) == _lib.HARTS_EUNSUPPORTED
    assert ws(p.handle, 0, 0, _lib.HARTS_BF16, 16, 96, 96, 0, C.byref(sz)) == _lib.HARTS_EUNSUPPORTED
    assert ws(p.handle, 0, 0, _lib.HARTS_F32, 16, 128, 128, 0, C.byref(sz)) == _lib.HARTS_EUNSUPPORTED
    assert ws(p.handle, 0, 0, _lib.HARTS_BF16, 16, 128, 64, 0, C.byref(sz)) == _lib.HARTS_EUNSUPPORTED
    assert ws(p.handle, 5, 0, _lib.HARTS_BF16, 16, 128, 128, 0, C.byref(sz)) == _lib.HARTS_EINVAL
    assert ws(p.handle, 0, 2, _lib.HARTS_BF16, 16, 128, 128, 0, C.byref(sz)) == _lib.HARTS_EINVAL
    assert ws(None, 0, 0, _lib.HARTS_BF16, 16, 128, 128, 0, C.byref(sz)) == _lib.HARTS_EINVAL
    # a plan with another chunk size cannot be executed on the device
    p2 = HartsPlan(f.parent, f.seg_len, 32)
    assert ws(p2.handle, 0, 0, _lib.HARTS_BF16, 16, 128, 128, 0, C.byref(sz)) == _lib.HARTS_EUNSUPPORTED
    # NULL tensors are rejected on the host (nothing is enqueued)
    null = C.c_void_p()
    rc = L.harts_la_fwd(p.handle, 0, null, _lib.HARTS_BF16, 16, 128, 128, C.c_float(0.1),
                        null, null, null, null, null, null, null, null, null, null,
                        C.c_size_t(0), null)
    assert rc == _lib.HARTS_EINVAL
    rc = L.harts_la_bwd(p.handle, 0, null, _lib.HARTS_BF16, 16, 128, 128, C.c_float(0.1),
                        null, null, null, null, null, null, null, null, null, null, null, null,
                        null, null, null, null, null, C.c_size_t(0), null)
    assert rc == _lib.HARTS_EINVAL
    # state gather: bad mode / sizes rejected, an empty gather is a no-op
    g = L.harts_state_gather
    assert g(null, null, 4, C.c_int64(16), null, 2, null) == _lib.HARTS_EINVAL
    assert g(null, null, -1, C.c_int64(16), null, 0, null) == _lib.HARTS_EINVAL
    assert g(null, null, 4, C.c_int64(6), null, 0, null) == _lib.HARTS_EINVAL
    assert g(null, null, 4, C.c_int64(16), null, 0, null) == _lib.HARTS_EINVAL
    assert g(null, null, 0, C.c_int64(16), null, 0, null) == _lib.HARTS_OK
    p.close()
    p2.close()


def test_device_calls_reject_plans_beyond_the_row_limit(L):
    """Device row tables hold physical row * 4 + kind in int32: a plan of
    2^29 or more packed rows plans on the host but every device call
    rejects it with HARTS_EUNSUPPORTED before launching anything."""
    from paper_2608_28158_amd import _lib
    from paper_2608_28158_amd.plan import HartsPlan
    sz = C.c_size_t()
    for n_rows, rc in (((1 << 29) - 64, _lib.HARTS_OK), (1 << 29, _lib.HARTS_EUNSUPPORTED)):
        p = HartsPlan([-1], [n_rows], 64)
        assert p["C"] + p["R"] == n_rows
        assert L.harts_la_workspace_size(p.handle, 0, 0, _lib.HARTS_BF16, 1, 64, 64, 0,
                                         C.byref(sz)) == rc
        p.close()


def test_set_blocks_recuts_rounds_by_head_count(L):
    """harts_plan_set_blocks: the largest block size (64, 48, ..., 8 chunks)
    that yields min_blocks blocks, min_blocks = ceil(896 / H) by default;
    the plan proper (rounds, sequences, rows) is untouched."""
    from paper_2608_28158_amd import _lib
    from paper_2608_28158_amd.plan import HartsPlan
    f, _, _ = forest_for_config(2)
    base = HartsPlan(f.parent, f.seg_len, 64)                  # set for 16 heads
    seen = {}
    for H, mb in ((16, 0), (32, 0), (8, 0), (16, 56), (16, 100000)):
        p = HartsPlan(f.parent, f.seg_len, 64, heads=H, min_blocks=mb)
        target = mb or -(-896 // H)
        for r, rd in enumerate(p.rounds):
            nc = rd["n_chunks"]
            assert rd["block_chunks"] in (64, 48, 32, 24, 16, 12, 8)
            assert rd["n_blk"] >= min(target, rd["n_blk"])
            if rd["block_chunks"] != 8:
                assert rd["n_blk"] >= target
            assert rd["n_blk"] >= rd["n_seq"] and rd["n_blk"] <= nc
        for key in ("seq_round", "seg_row", "replay_row", "seq_init_bank"):
            assert np.array_equal(p[key], base[key])
        seen[(H, mb)] = [rd["block_chunks"] for rd in p.rounds]
        p.close()
    assert seen[(16, 0)] == seen[(16, 56)]
    assert seen[(16, 100000)] == [8] * len(seen[(16, 0)])
    assert all(a >= b for a, b in zip(seen[(32, 0)], seen[(16, 0)]))
    h = base.handle
    assert L.harts_plan_set_blocks(h, 0, 0) == _lib.HARTS_EINVAL
    assert L.harts_plan_set_blocks(h, 16, -1) == _lib.HARTS_EINVAL
    assert L.harts_plan_set_blocks(None, 16, 0) == _lib.HARTS_EINVAL
    base.close()
