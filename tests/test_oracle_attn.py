"""Pins of the attention oracle (Sec. 4.2, eqs. asymmetric-qkv and
bottom-right): one sequence against torch's scaled_dot_product_attention
(a library routine), branch views with bottom-right alignment against the
trajectory-wise definition (and top-left alignment shown to differ),
gradients against finite differences."""
import numpy as np
import pytest
import torch

from oracle.attn import causal_attention, forest_attention, view_attention
from oracle.compact import sequence_rows
from oracle.forest import SegTree
from oracle.plan_ref import plan_ref
from workloads.trees import figure1_forest


def test_causal_attention_matches_sdpa():
    r = np.random.default_rng(0)
    q, k, v = (torch.tensor(r.standard_normal((37, 3, 16))) for _ in range(3))
    o = causal_attention(q, k, v, 0.25)
    ref = torch.nn.functional.scaled_dot_product_attention(
        q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1), is_causal=True, scale=0.25)
    assert torch.allclose(o, ref.transpose(0, 1), rtol=0, atol=1e-13)


def branch_views(parent, seg_len, B=64):
    """Per plan sequence: own rows and the h ancestor rows before them."""
    t = SegTree(parent, seg_len)
    p = plan_ref(parent, seg_len, B)
    out = []
    for i in range(p["n_seq"]):
        _, own = sequence_rows(t, p, i)
        first = own[0]
        v0 = next(v for v in range(t.n) if t.row0[v] == first)
        anc = [t.row_of(v0, pos) for pos in range(0, t.s[v0])]
        out.append((anc, own))
    return out


@pytest.mark.parametrize("case", [(figure1_forest().parent, figure1_forest().seg_len),
                                  ([-1, 0, 0, 1, 1, -1, 5], [70, 9, 30, 44, 20, 15, 3])])
def test_views_with_bottom_right_alignment_reproduce_trajectories(case):
    parent, seg_len = case
    r = np.random.default_rng(1)
    C = int(np.sum(seg_len))
    q, k, v = (r.standard_normal((C, 2, 8)) for _ in range(3))
    ref = forest_attention(parent, seg_len, q, k, v, 0.3)["o"]
    T = lambda a: torch.tensor(a)
    differs = False
    for anc, own in branch_views(parent, seg_len):
        kv = anc + own
        o = view_attention(T(q[own]), T(k[kv]), T(v[kv]), len(anc), 0.3).numpy()
        assert np.allclose(o, ref[own], rtol=0, atol=1e-13)
        if anc:     # top-left alignment (query i sees keys j <= i) would differ
            s = torch.einsum("qhd,khd->hqk", T(q[own]), T(k[kv])) * 0.3
            mask = torch.arange(len(kv))[None, :] <= torch.arange(len(own))[:, None]
            p = torch.softmax(s.masked_fill(~mask, float("-inf")), -1)
            top = torch.einsum("hqk,khd->qhd", p, T(v[kv])).numpy()
            differs = differs or not np.allclose(top, ref[own])
    assert differs


def test_gradients_finite_differences():
    parent, seg_len = [-1, 0, 0, 1], [3, 2, 4, 2]
    r = np.random.default_rng(2)
    C = sum(seg_len)
    q, k, v, dO = (r.standard_normal((C, 2, 4)) for _ in range(4))
    g = forest_attention(parent, seg_len, q, k, v, 0.5, dO=dO)
    loss = lambda qq, kk, vv: float(np.sum(forest_attention(parent, seg_len, qq, kk, vv, 0.5)["o"] * dO))
    h = 1e-6
    for name, arr in (("dq", q), ("dk", k), ("dv", v)):
        for _ in range(6):
            idx = tuple(int(r.integers(0, s)) for s in arr.shape)
            ap, am = arr.copy(), arr.copy()
            ap[idx] += h
            am[idx] -= h
            args_p = [ap if arr is x else x for x in (q, k, v)]
            args_m = [am if arr is x else x for x in (q, k, v)]
            fd = (loss(*args_p) - loss(*args_m)) / (2 * h)
            assert abs(fd - g[name][idx]) < 1e-7 * max(1.0, abs(fd))
