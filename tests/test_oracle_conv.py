"""Pins of the causal-convolution oracle (Sec. 4.2): one trajectory against
scipy's linear filter and torch's conv1d (library routines), the forest
gradients against torch autograd of the expanded trajectories, finite
differences, and the window of a row never reaching beyond its ancestors."""
import numpy as np
import pytest
import scipy.signal
import torch

from oracle.conv import conv_bwd, conv_fwd, conv_trajectory
from oracle.forest import SegTree
from workloads.trees import figure1_forest


def test_single_trajectory_matches_lfilter_and_conv1d():
    r = np.random.default_rng(0)
    x = r.standard_normal((50, 6))
    W = r.standard_normal((6, 4))
    y = conv_trajectory(x, W)
    for c in range(6):
        assert np.allclose(y[:, c], scipy.signal.lfilter(W[c], [1.0], x[:, c]), rtol=0, atol=1e-13)
    xt = torch.tensor(x.T[None], dtype=torch.float64)
    # conv1d correlates: flip the taps, pad w - 1 zeros on the left
    k = torch.tensor(W[:, ::-1].copy()[:, None, :], dtype=torch.float64)
    ref = torch.nn.functional.conv1d(torch.nn.functional.pad(xt, (3, 0)), k, groups=6)[0].T
    assert np.allclose(y, ref.numpy(), rtol=0, atol=1e-13)


def _expanded(parent, seg_len, x):
    t = SegTree(parent, seg_len)
    return t, [np.asarray(t.trajectory_rows(l)) for l in t.leaves]


@pytest.mark.parametrize("case", [(figure1_forest().parent, figure1_forest().seg_len),
                                  ([-1, 0, 1, 1, 2, 0], [2, 1, 3, 1, 5, 1])])
def test_forest_gradients_match_autograd(case):
    parent, seg_len = case
    r = np.random.default_rng(1)
    C = int(np.sum(seg_len))
    x = r.standard_normal((C, 5))
    W = r.standard_normal((5, 4))
    dy = r.standard_normal((C, 5))
    y = conv_fwd(parent, seg_len, x, W)
    dx, dW = conv_bwd(parent, seg_len, x, W, dy)
    t, trajs = _expanded(parent, seg_len, x)
    xt = torch.tensor(x, requires_grad=True)
    Wt = torch.tensor(W, requires_grad=True)
    owned = np.zeros(C, bool)
    loss = 0
    for rows in trajs:
        seq = xt[torch.tensor(rows)].T[None]
        k = Wt.flip(1)[:, None, :]
        yt = torch.nn.functional.conv1d(torch.nn.functional.pad(seq, (3, 0)), k, groups=5)[0].T
        assert np.allclose(yt.detach().numpy(), y[rows], atol=1e-12)
        mine = torch.tensor(~owned[rows])
        owned[rows] = True
        loss = loss + (yt * torch.tensor(dy[rows]) * mine[:, None]).sum()
    loss.backward()
    assert np.allclose(dx, xt.grad.numpy(), atol=1e-12)
    assert np.allclose(dW, Wt.grad.numpy(), atol=1e-12)


def test_finite_differences_and_ancestor_window():
    parent, seg_len = [-1, 0, 0, 1], [2, 2, 3, 4]
    r = np.random.default_rng(2)
    C = sum(seg_len)
    x = r.standard_normal((C, 3))
    W = r.standard_normal((3, 4))
    dy = r.standard_normal((C, 3))
    dx, dW = conv_bwd(parent, seg_len, x, W, dy)
    loss = lambda xx, WW: float(np.sum(conv_fwd(parent, seg_len, xx, WW) * dy))
    h = 1e-6
    for _ in range(12):
        a, c = int(r.integers(0, C)), int(r.integers(0, 3))
        xp, xm = x.copy(), x.copy()
        xp[a, c] += h
        xm[a, c] -= h
        assert abs((loss(xp, W) - loss(xm, W)) / (2 * h) - dx[a, c]) < 1e-7
        i = int(r.integers(0, 4))
        Wp, Wm = W.copy(), W.copy()
        Wp[c, i] += h
        Wm[c, i] -= h
        assert abs((loss(x, Wp) - loss(x, Wm)) / (2 * h) - dW[c, i]) < 1e-7
    # segment 2 (rows 4..6) forks from the root (rows 0, 1): its first row's
    # window is rows 4, 1, 0 and then zero -- never segment 1's rows 2, 3
    x2 = x.copy()
    x2[2:4] += 100.0
    y1, y2 = conv_fwd(parent, seg_len, x, W), conv_fwd(parent, seg_len, x2, W)
    assert np.array_equal(y1[4:7], y2[4:7])
    assert np.allclose(y1[4], W[:, 0] * x[4] + W[:, 1] * x[1] + W[:, 2] * x[0])
