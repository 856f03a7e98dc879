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


def lib_views(plan):
    from paper_2608_28158_amd import _lib
    L = _lib.lib()
    lay = _lib.AttnLayout()
    _lib.check(L.harts_attn_layout(plan.handle, C.byref(lay)), "harts_attn_layout")
    views = np.zeros((lay.n_views, 4), np.int32)
    kv_rows = np.zeros(lay.n_kv, np.int32)
    qt = np.zeros((lay.n_qtiles, 2), np.int32)
    kt = np.zeros((lay.n_kvtiles, 2), np.int32)
    off = np.zeros(plan["C"] + 1, np.int64)
    ent = np.zeros(lay.n_kv, np.int32)
    _lib.check(L.harts_attn_views(plan.handle, views.ctypes.data, kv_rows.ctypes.data, qt.ctypes.data,
                                  kt.ctypes.data, off.ctypes.data, ent.ctypes.data), "harts_attn_views")
    return views, kv_rows, qt, kt, off, ent


@pytest.mark.parametrize("label,parent,seg_len", CASES + [
    ("deep chain", [-1, 0, 1, 2, 3, 4], [70, 1, 130, 5, 64, 9])], ids=[c[0] for c in CASES] + ["deep chain"])
def test_attn_views_follow_each_trajectory(label, parent, seg_len):
    """Views of Sec. 4.2 (eq. asymmetric-qkv): per plan sequence, the query
    rows are its own rows and the key/value rows the trajectory positions
    0 .. h-1 before its first own token, then the own rows; 128-row tiles
    cover every query and key row once, heaviest first; the gradient lists
    invert kv_rows."""
    from oracle.compact import sequence_rows
    from oracle.forest import SegTree
    from paper_2608_28158_amd.plan import HartsPlan
    plan = HartsPlan(parent, seg_len, 64)
    t = SegTree(parent, seg_len)
    phys = phys_index(seg_len, plan["seg_row"])
    views, kv_rows, qt, kt, off, ent = lib_views(plan)
    C_ = int(np.sum(seg_len))
    assert len(views) == plan["n_seq"]
    seen_q = np.zeros(C_, np.int64)
    want_q, want_k = [], []
    for i in range(plan["n_seq"]):
        _, own = sequence_rows(t, plan, i)
        v0 = int(plan["chain_seg"][int(plan["seq_chain_off"][i])])
        anc = [t.row_of(v0, pos) for pos in range(t.s[v0])]
        q0, l, kvoff, h = (int(x) for x in views[i])
        assert l == len(own) and h == len(anc)
        assert np.array_equal(q0 + np.arange(l), phys[own])
        assert np.array_equal(kv_rows[kvoff:kvoff + h + l], phys[anc + own])
        seen_q[q0:q0 + l] += 1
        want_q += [(h + s, i, s) for s in range(0, l, 128)]
        want_k += [(l - max(0, s - h), i, s) for s in range(0, h + l, 128)]
    assert np.all(seen_q == 1)
    # heaviest first, equal work in view order
    order = lambda tiles: [(i, s) for _, i, s in sorted(tiles, key=lambda x: (-x[0], x[1], x[2]))]
    assert [tuple(x) for x in qt] == order(want_q) and [tuple(x) for x in kt] == order(want_k)
    assert off[0] == 0 and off[-1] == len(kv_rows) and np.all(np.diff(off) >= 1)
    for r in range(C_):
        e = ent[off[r]:off[r + 1]]
        assert np.all(np.diff(e) > 0) and np.all(kv_rows[e] == r)


def test_attn_views_on_the_64k_workload():
    from paper_2608_28158_amd.plan import HartsPlan
    f, _, cfg = forest_for_config(2)
    plan = HartsPlan(f.parent, f.seg_len, 64, heads=cfg["H"])
    views, kv_rows, qt, kt, off, ent = lib_views(plan)
    h = views[:, 3].astype(np.int64)
    l = views[:, 1].astype(np.int64)
    assert l.sum() == f.n_rows and len(kv_rows) == (h + l).sum()
    assert len(qt) == ((l + 127) // 128).sum() and len(kt) == ((h + l + 127) // 128).sum()
    assert np.array_equal(np.sort(kv_rows[ent]), np.sort(kv_rows)) and np.all(np.diff(kv_rows[ent]) >= 0)


def test_attn_entry_points_validate_before_any_launch():
    """Unsupported head sizes, NULL and misaligned pointers are rejected on
    the host (no device work is started, so this runs without a GPU)."""
    from paper_2608_28158_amd import _lib
    L = _lib.lib()
    buf = np.zeros(4096, np.int64)
    p = buf.ctypes.data
    f32 = C.c_float(0.1)
    assert L.harts_attn_fwd(p, p, 1, 2, 96, f32, p, p, p, p, p, None) == _lib.HARTS_EUNSUPPORTED
    assert L.harts_attn_fwd(p, p, 1, 0, 64, f32, p, p, p, p, p, None) == _lib.HARTS_EUNSUPPORTED
    assert L.harts_attn_fwd(p, p, 1, 2, 64, f32, None, p, p, p, p, None) == _lib.HARTS_EINVAL
    assert L.harts_attn_fwd(p, p, 1, 2, 64, f32, p + 2, p, p, p, p, None) == _lib.HARTS_EINVAL
    assert L.harts_attn_fwd(p, p, -1, 2, 64, f32, p, p, p, p, p, None) == _lib.HARTS_EINVAL
    assert L.harts_attn_fwd(p, p, 0, 2, 64, f32, p, p, p, p, p, None) == _lib.HARTS_OK
    assert L.harts_attn_bwd(p, p, 1, p, 1, 10, 2, 128, f32, p, p, p, p, p, p, p, None, p, p,
                            None) == _lib.HARTS_EINVAL
    assert L.harts_attn_bwd(p, p, 1, p, 1, 10, 2, 32, f32, p, p, p, p, p, p, p, p, p, p,
                            None) == _lib.HARTS_EUNSUPPORTED
    assert L.harts_attn_gather(p, p, -1, 10, 2, 64, p, None) == _lib.HARTS_EINVAL
    assert L.harts_attn_gather(p, None, 4, 10, 2, 64, p, None) == _lib.HARTS_EINVAL
    assert L.harts_attn_scatter(p, p, p, 10, 4, 2, 64, p + 4, None) == _lib.HARTS_EINVAL
    assert L.harts_attn_layout(None, None) == _lib.HARTS_EINVAL
