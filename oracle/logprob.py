"""Compact-to-semantic log-probabilities (Sec. 3.5), the plain definition in
float64.  TEST INFRASTRUCTURE ONLY (see the package docstring).

Semantic positions.  Trajectories are the root-to-leaf paths, in ascending
leaf id (the original batch order of this build), positions in order.  A
position s at trajectory index t < n - 1 is nonterminal: its next token y_s
is the token of the trajectory's row t + 1, and m(s) is its own compact row
(canonical rows: segments in id order).  A trajectory's last position has no
next token and is not in the set.

Log-probability (eq. mapped-logp):  lambda_s = z[m(s), y_s] - log sum_v
exp z[m(s), v], evaluated here per semantic position on its own row, i.e. the
trajectory-wise computation that the compact one must reproduce.

Gradient (eq. mapped-logp-grad): for upstream gradients g_s = dL/dlambda_s,
  dz[c, :] = sum over s with m(s) = c of g_s (onehot(y_s) - softmax(z[c, :])),
accumulated position by position.
"""
from __future__ import annotations

import numpy as np

from .forest import SegTree


def semantic_positions(parent, seg_len, tokens):
    """(m, y) over all nonterminal semantic positions, trajectories by
    ascending leaf id.  tokens: [C] int token id of every canonical row."""
    t = SegTree(parent, seg_len)
    m, y = [], []
    for leaf in t.leaves:
        rows = t.trajectory_rows(leaf)
        for a, b in zip(rows[:-1], rows[1:]):
            m.append(a)
            y.append(int(tokens[b]))
    return np.asarray(m, np.int64), np.asarray(y, np.int64)


def log_softmax_row(z_row):
    z = np.asarray(z_row, np.float64)
    mx = np.max(z)
    return z - (mx + np.log(np.sum(np.exp(z - mx))))


def logp_fwd(z, m, y):
    """lambda_s for every position, one vocabulary-wide log-softmax per
    semantic position (no reuse of compact rows)."""
    z = np.asarray(z, np.float64)
    out = np.empty(len(m))
    for s in range(len(m)):
        out[s] = log_softmax_row(z[m[s]])[y[s]]
    return out


def logp_bwd(z, m, y, g):
    """dz of L = sum_s g_s lambda_s, accumulated position by position."""
    z = np.asarray(z, np.float64)
    dz = np.zeros_like(z)
    for s in range(len(m)):
        p = np.exp(log_softmax_row(z[m[s]]))
        contrib = -g[s] * p
        contrib[y[s]] += g[s]
        dz[m[s]] += contrib
    return dz
