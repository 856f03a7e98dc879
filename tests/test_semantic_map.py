"""harts_semantic_map on the CPU: the library's compact-to-semantic map
(Sec. 3.5) equals the oracle's, position by position (rows translated to the
plan's physical order), and its per-row lists hold every position once, in
(target, position) order."""
import ctypes as C

import numpy as np
import pytest

from oracle.logprob import semantic_positions
from tests.harness import phys_index
from workloads.trees import figure1_forest, forest_for_config


def lib_map(plan, tokens_phys):
    from paper_2608_28158_amd import _lib
    L = _lib.lib()
    n_pos = plan["S"] - plan["n_leaves"]
    m = np.zeros(n_pos, np.int32)
    y = np.zeros(n_pos, np.int32)
    off = np.zeros(plan["C"] + 1, np.int64)
    pos = np.zeros(n_pos, np.int32)
    tok = np.ascontiguousarray(tokens_phys, np.int32)
    _lib.check(L.harts_semantic_map(plan.handle, tok.ctypes.data, n_pos, m.ctypes.data,
                                    y.ctypes.data, off.ctypes.data, pos.ctypes.data),
               "harts_semantic_map")
    return m, y, off, pos


CASES = [("figure 1", figure1_forest().parent, figure1_forest().seg_len),
         ("two trees", [-1, 0, 0, -1, 3, 3, 5], [65, 10, 80, 200, 1, 64, 3]),
         ("star", [-1] + [0] * 40, [100] + [3] * 40)]


@pytest.mark.parametrize("label,parent,seg_len", CASES, ids=[c[0] for c in CASES])
def test_semantic_map_matches_oracle(label, parent, seg_len):
    from paper_2608_28158_amd.plan import HartsPlan
    plan = HartsPlan(parent, seg_len, 64)
    C_ = int(np.sum(seg_len))
    r = np.random.default_rng(len(parent))
    tokens = r.integers(0, 1000, size=C_)
    phys = phys_index(seg_len, plan["seg_row"])
    tok_phys = np.empty(C_, np.int64)
    tok_phys[phys] = tokens
    m, y, off, pos = lib_map(plan, tok_phys)
    m_ref, y_ref = semantic_positions(parent, seg_len, tokens)
    assert np.array_equal(m, phys[m_ref]) and np.array_equal(y, y_ref)
    # per-row lists: a permutation of all positions, grouped by row, sorted by (y, s)
    assert off[0] == 0 and off[-1] == len(m) and np.all(np.diff(off) >= 0)
    assert np.array_equal(np.sort(pos), np.arange(len(m)))
    for c in range(C_):
        p = pos[off[c]:off[c + 1]]
        assert np.all(m[p] == c)
        keys = list(zip(y[p], p))
        assert keys == sorted(keys)


def test_semantic_map_on_the_64k_workload():
    from paper_2608_28158_amd.plan import HartsPlan
    f, _, _ = forest_for_config(2)
    plan = HartsPlan(f.parent, f.seg_len, 64)
    tokens = np.random.default_rng(9).integers(0, 157184, size=f.n_rows)
    phys = phys_index(f.seg_len, plan["seg_row"])
    tok_phys = np.empty(f.n_rows, np.int64)
    tok_phys[phys] = tokens
    m, y, off, pos = lib_map(plan, tok_phys)
    m_ref, y_ref = semantic_positions(f.parent, f.seg_len, tokens)
    assert np.array_equal(m, phys[m_ref]) and np.array_equal(y, y_ref)
    assert len(m) == plan["S"] - plan["n_leaves"]


def test_semantic_map_validates():
    from paper_2608_28158_amd import _lib
    from paper_2608_28158_amd.plan import HartsPlan
    f = figure1_forest()
    plan = HartsPlan(f.parent, f.seg_len, 64)
    L = _lib.lib()
    buf = np.zeros(4096, np.int64)
    p = buf.ctypes.data
    assert L.harts_semantic_map(plan.handle, p, 5, p, p, p, p) == _lib.HARTS_EINVAL
    assert L.harts_semantic_map(None, p, 955, p, p, p, p) == _lib.HARTS_EINVAL
    assert L.harts_semantic_map(plan.handle, None, 955, p, p, p, p) == _lib.HARTS_EINVAL


@pytest.mark.parametrize("label,parent,seg_len", CASES + [
    ("chain of one-token segments", [-1, 0, 1, 2, 3, 3, 5], [1, 1, 1, 1, 1, 4, 2])],
    ids=[c[0] for c in CASES] + ["tiny segments"])
@pytest.mark.parametrize("w", [2, 4, 8])
def test_conv_context_follows_each_trajectory(label, parent, seg_len, w):
    """harts_conv_context: a row's i-th predecessor is the row i positions
    earlier on its own trajectory (-1 before the start), the same on every
    trajectory through the row; the consumer lists are its transpose."""
    from oracle.forest import SegTree
    from paper_2608_28158_amd import _lib
    from paper_2608_28158_amd.plan import HartsPlan
    plan = HartsPlan(parent, seg_len, 64)
    C_ = int(np.sum(seg_len))
    k = w - 1
    pred = np.full(C_ * k, -7, np.int32)
    off = np.zeros(C_ + 1, np.int64)
    succ = np.zeros(C_ * k, np.int32)
    L = _lib.lib()
    _lib.check(L.harts_conv_context(plan.handle, w, pred.ctypes.data, off.ctypes.data,
                                    succ.ctypes.data), "harts_conv_context")
    pred = pred.reshape(C_, k)
    phys = phys_index(seg_len, plan["seg_row"])
    t = SegTree(parent, seg_len)
    want = {}
    for leaf in t.leaves:
        rows = t.trajectory_rows(leaf)
        for pos, row in enumerate(rows):
            exp = [int(phys[rows[pos - i]]) if pos - i >= 0 else -1 for i in range(1, w)]
            assert want.setdefault(int(phys[row]), exp) == exp
    for r in range(C_):
        assert list(pred[r]) == want[r]
    entries = []
    for r in range(C_):
        lst = [(int(c) & 7, int(c) >> 3) for c in succ[off[r]:off[r + 1]]]
        assert lst == sorted(lst)
        entries += [(s, i, r) for i, s in lst]
    expect = [(s, i, int(pred[s, i - 1])) for s in range(C_) for i in range(1, w)
              if pred[s, i - 1] >= 0]
    assert sorted(entries) == sorted(expect)
