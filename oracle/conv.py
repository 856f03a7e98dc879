"""Causal depthwise convolution with true-ancestor context (Sec. 4.2, "KDA
state reuse and causal convolution"), the plain definition in float64.
TEST INFRASTRUCTURE ONLY (see the package docstring).

Along every root-to-leaf trajectory, channel by channel,
    y_t[c] = sum_{i=0}^{w-1} W[c, i] x_{t-i}[c],   x_{t-i} = 0 before the
                                                   trajectory's first token.
A compact row's output is the one of any trajectory through it (they agree:
the window of a row reaches only its own ancestors); this oracle computes
every trajectory separately and checks that they agree.

Backward, per trajectory with the upstream gradient of a compact row given
to one trajectory through it (the smallest leaf id), summed over
trajectories into compact rows:
    dx_s[c] += W[c, i] dy_{s+i}[c]     for every i with s + i on the path,
    dW[c, i] += x_{t-i}[c] dy_t[c].
"""
from __future__ import annotations

import numpy as np

from .forest import SegTree


def conv_trajectory(x, W):
    """x: [n, Cch]; W: [Cch, w].  y[t] = sum_i W[:, i] x[t - i]."""
    x = np.asarray(x, np.float64)
    W = np.asarray(W, np.float64)
    n, w = x.shape[0], W.shape[1]
    y = np.zeros_like(x)
    for t in range(n):
        for i in range(w):
            if t - i >= 0:
                y[t] += W[:, i] * x[t - i]
    return y


def conv_fwd(parent, seg_len, x, W):
    t = SegTree(parent, seg_len)
    y = np.zeros(np.shape(x), np.float64)
    have = np.zeros(t.C, bool)
    for leaf in t.leaves:
        rows = np.asarray(t.trajectory_rows(leaf))
        yt = conv_trajectory(np.asarray(x)[rows], W)
        old = have[rows]
        if not np.array_equal(y[rows[old]], yt[old]):
            raise AssertionError("trajectories disagree on a shared row")
        y[rows[~old]] = yt[~old]
        have[rows] = True
    return y


def conv_bwd(parent, seg_len, x, W, dy):
    """(dx, dW) of sum <dy, y>, dy per compact row entering one trajectory."""
    t = SegTree(parent, seg_len)
    x = np.asarray(x, np.float64)
    W = np.asarray(W, np.float64)
    dy = np.asarray(dy, np.float64)
    w = W.shape[1]
    dx = np.zeros_like(x)
    dW = np.zeros_like(W)
    owned = np.zeros(t.C, bool)
    for leaf in t.leaves:
        rows = np.asarray(t.trajectory_rows(leaf))
        mine = ~owned[rows]
        owned[rows] = True
        g = np.where(mine[:, None], dy[rows], 0.0)
        xt = x[rows]
        n = len(rows)
        dxt = np.zeros_like(xt)
        for tt in range(n):
            for i in range(w):
                if tt - i >= 0:
                    dxt[tt - i] += W[:, i] * g[tt]
                    dW[:, i] += xt[tt - i] * g[tt]
        np.add.at(dx, rows, dxt)
    return dx, dW
