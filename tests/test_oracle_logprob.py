"""Pins of the compact-to-semantic log-probability oracle (Sec. 3.5,
eqs. mapped-logp, mapped-logp-grad) against things other than itself:
library log-softmax and cross-entropy routines, finite differences, the
softmax-gradient invariants, and the semantic map of the Figure 1 tree
worked out by hand."""
import numpy as np
import pytest
import scipy.special
import torch

from oracle.forest import SegTree
from oracle.logprob import log_softmax_row, logp_bwd, logp_fwd, semantic_positions
from workloads.trees import figure1_forest


def test_log_softmax_matches_scipy_and_normalises():
    r = np.random.default_rng(0)
    for scale in (0.1, 3.0, 80.0):
        z = r.standard_normal(1000) * scale
        ls = log_softmax_row(z)
        assert np.max(np.abs(ls - scipy.special.log_softmax(z))) < 1e-12 * max(1.0, scale)
        assert abs(np.sum(np.exp(ls)) - 1.0) < 1e-12


def test_figure1_semantic_map_by_hand():
    """Figure 1 (A=200, B=77, C=90, D=64, E=50; canonical rows A 0-199,
    B 200-276, C 277-366, D 367-430, E 431-480).  The last row of A
    precedes B's first row on two trajectories and C's on one; the last row
    of B precedes D's and E's first rows."""
    f = figure1_forest()
    tokens = np.arange(f.n_rows) * 7 % 1000          # distinct enough to trace
    m, y = semantic_positions(f.parent, f.seg_len, tokens)
    assert len(m) == (200 + 90) + (200 + 77 + 64) + (200 + 77 + 50) - 3
    nxt = {}
    for a, b in zip(m, y):
        nxt.setdefault(int(a), []).append(int(b))
    assert sorted(nxt[199]) == sorted([tokens[277], tokens[200], tokens[200]])
    assert sorted(nxt[276]) == sorted([tokens[367], tokens[431]])
    assert nxt[0] == [tokens[1]] * 3
    for last in (366, 430, 480):                      # leaf ends: terminal everywhere
        assert last not in nxt
    # positions per row = multiplicity, minus one at a leaf's last row
    t = SegTree(f.parent, f.seg_len)
    q = t.multiplicity()
    for v in range(t.n):
        for row in range(t.row0[v], t.row0[v] + t.len[v]):
            leaf_end = not t.kids[v] and row == t.row0[v] + t.len[v] - 1
            assert len(nxt.get(row, [])) == q[v] - leaf_end


def _expanded_ce(z, m, y):
    """torch's cross-entropy on the expanded S x V logits (library routine)."""
    zt = torch.tensor(np.asarray(z)[m], dtype=torch.float64, requires_grad=True)
    ce = torch.nn.functional.cross_entropy(zt, torch.tensor(y), reduction="none")
    return zt, ce


def test_forward_matches_expanded_cross_entropy():
    f = figure1_forest()
    r = np.random.default_rng(1)
    V = 97
    tokens = r.integers(0, V, size=f.n_rows)
    z = r.standard_normal((f.n_rows, V)) * 2.5
    m, y = semantic_positions(f.parent, f.seg_len, tokens)
    lam = logp_fwd(z, m, y)
    _, ce = _expanded_ce(z, m, y)
    assert np.max(np.abs(lam + ce.detach().numpy())) < 1e-12


def test_backward_matches_autograd_of_expanded_cross_entropy():
    f = figure1_forest()
    r = np.random.default_rng(2)
    V = 53
    tokens = r.integers(0, V, size=f.n_rows)
    z = r.standard_normal((f.n_rows, V))
    m, y = semantic_positions(f.parent, f.seg_len, tokens)
    g = r.standard_normal(len(m)) * (r.random(len(m)) < 0.7)   # an action mask
    dz = logp_bwd(z, m, y, g)
    zt, ce = _expanded_ce(z, m, y)
    (-(ce * torch.tensor(g))).sum().backward()
    ref = np.zeros_like(z)
    np.add.at(ref, m, zt.grad.numpy())
    assert np.max(np.abs(dz - ref)) < 1e-12


def test_backward_finite_differences_and_invariants():
    parent, seg_len = [-1, 0, 0, 1, 1, 0], [5, 3, 4, 2, 6, 1]
    r = np.random.default_rng(3)
    V = 11
    C = sum(seg_len)
    tokens = r.integers(0, V, size=C)
    z = r.standard_normal((C, V))
    m, y = semantic_positions(parent, seg_len, tokens)
    g = r.standard_normal(len(m))
    dz = logp_bwd(z, m, y, g)
    loss = lambda zz: float(np.dot(g, logp_fwd(zz, m, y)))
    h = 1e-6
    for _ in range(25):
        c, v = int(r.integers(0, C)), int(r.integers(0, V))
        zp, zm = z.copy(), z.copy()
        zp[c, v] += h
        zm[c, v] -= h
        fd = (loss(zp) - loss(zm)) / (2 * h)
        assert abs(fd - dz[c, v]) < 1e-7 * max(1.0, abs(fd))
    # every row's gradient sums to zero; rows no position maps to get none
    assert np.max(np.abs(dz.sum(axis=1))) < 1e-12
    unused = np.setdiff1d(np.arange(C), m)
    assert len(unused) > 0 and np.all(dz[unused] == 0)


@pytest.mark.parametrize("seed", [4, 5])
def test_shared_rows_give_one_logit_row_many_targets(seed):
    """At a fork, one compact row serves several positions with different
    targets: their lambdas come from one log-softmax row."""
    f = figure1_forest()
    r = np.random.default_rng(seed)
    V = 31
    tokens = r.integers(0, V, size=f.n_rows)
    z = r.standard_normal((f.n_rows, V))
    m, y = semantic_positions(f.parent, f.seg_len, tokens)
    lam = logp_fwd(z, m, y)
    ls = log_softmax_row(z[276])
    sel = np.nonzero(m == 276)[0]
    assert len(sel) == 2
    assert np.allclose(lam[sel], ls[y[sel]], rtol=0, atol=0)
