"""Token-by-token scalar-decay linear attention in float64 (the plain definition).

Per head h, with state S of shape [d_k, d_v]:

    S_t = exp(g_t) S_{t-1} + k_t v_t^T,      o_t = scale * S_t^T q_t,

inclusive of token t (decay applied before adding token t).  Over a forest
every root-to-leaf trajectory is run separately from its tree's initial state
(zero unless given, Sec. 3.4 "Round-wise execution": roots start from zero).
A compact row's output is the one computed on the trajectory of the smallest
leaf id that contains it; every other trajectory through the row must give
the bit-identical value, because it runs the same operations on the same
prefix (the claim of Sec. 2.2 that replay keeps the trajectory-wise path).

Backward, per trajectory, with Lam the adjoint of S_t (hand-derived from the
recurrence; checked against finite differences in the tests):

    Lam  = exp(g_{t+1}) Lam_{t+1} + scale q_t dO_t^T   (+ dS_final at the end)
    dq_t = scale S_t dO_t,  dk_t = Lam v_t,  dv_t = Lam^T k_t,
    dg_t = exp(g_t) <S_{t-1}, Lam>_F,        dS0 = exp(g_0) Lam_0.

Over a forest the upstream gradient of row c enters only the representative
trajectory of c, and per-trajectory gradients are summed into compact rows.
"""
from __future__ import annotations

import numpy as np

from .forest import SegTree


def la_fwd(q, k, v, g, S0, scale):
    """One trajectory.  q,k: [n,H,dk]; v: [n,H,dv]; g: [n,H]; S0: [H,dk,dv]."""
    q, k, v, g = (np.asarray(x, np.float64) for x in (q, k, v, g))
    S = np.array(S0, np.float64, copy=True)
    n, H, dv = v.shape
    o = np.zeros((n, H, dv))
    for t in range(n):
        S = np.exp(g[t])[:, None, None] * S + k[t][:, :, None] * v[t][:, None, :]
        o[t] = scale * np.einsum("hkv,hk->hv", S, q[t])
    return o, S


def la_bwd(q, k, v, g, S0, scale, dO, dS_final):
    """Gradients of sum <dO, o> + <dS_final, S_final> for one trajectory."""
    q, k, v, g, dO = (np.asarray(x, np.float64) for x in (q, k, v, g, dO))
    n = q.shape[0]
    states = [np.array(S0, np.float64, copy=True)]
    for t in range(n):
        states.append(np.exp(g[t])[:, None, None] * states[-1]
                      + k[t][:, :, None] * v[t][:, None, :])
    lam = np.array(dS_final, np.float64, copy=True)
    dq, dk, dv = np.zeros_like(q), np.zeros_like(k), np.zeros_like(v)
    dg = np.zeros_like(g)
    for t in range(n - 1, -1, -1):
        lam = lam + scale * q[t][:, :, None] * dO[t][:, None, :]
        dq[t] = scale * np.einsum("hkv,hv->hk", states[t + 1], dO[t])
        dk[t] = np.einsum("hkv,hv->hk", lam, v[t])
        dv[t] = np.einsum("hkv,hk->hv", lam, k[t])
        dg[t] = np.exp(g[t]) * np.einsum("hkv,hkv->h", states[t], lam)
        lam = np.exp(g[t])[:, None, None] * lam
    return dq, dk, dv, dg, lam


def forest_fwd(parent, seg_len, q, k, v, g, scale, S0_tree=None):
    """Expanded trajectory-wise forward over a forest (canonical rows).

    Returns o [C,H,dv] and S_final [n_leaves,H,dk,dv] (leaves by id)."""
    t = SegTree(parent, seg_len)
    C, H, dk = q.shape
    dv = v.shape[2]
    o = np.zeros((C, H, dv))
    have = np.zeros(C, bool)
    S_fin = np.zeros((len(t.leaves), H, dk, dv))
    for li, leaf in enumerate(t.leaves):
        rows = np.asarray(t.trajectory_rows(leaf))
        S0 = (np.zeros((H, dk, dv)) if S0_tree is None
              else S0_tree[t.tree[leaf]])
        ot, S = la_fwd(q[rows], k[rows], v[rows], g[rows], S0, scale)
        new = ~have[rows]
        if not np.array_equal(o[rows[~new]], ot[~new]):
            raise AssertionError("trajectories disagree on a shared row")
        o[rows[new]] = ot[new]
        have[rows] = True
        S_fin[li] = S
    return o, S_fin


def forest_bwd(parent, seg_len, q, k, v, g, scale, dO, dS_final,
               S0_tree=None):
    """Gradients over the expanded forest.  dO is per compact row; it enters
    only the representative (smallest-leaf-id) trajectory of each row."""
    t = SegTree(parent, seg_len)
    C, H, dk = q.shape
    dv = v.shape[2]
    dq, dk_, dv_ = np.zeros((C, H, dk)), np.zeros((C, H, dk)), np.zeros((C, H, dv))
    dg = np.zeros((C, H))
    dS0 = np.zeros((len(t.roots), H, dk, dv))
    owned = np.zeros(C, bool)
    for li, leaf in enumerate(t.leaves):
        rows = np.asarray(t.trajectory_rows(leaf))
        mine = ~owned[rows]
        owned[rows] = True
        dOt = np.where(mine[:, None, None], dO[rows], 0.0)
        tr = t.tree[leaf]
        S0 = np.zeros((H, dk, dv)) if S0_tree is None else S0_tree[tr]
        a, b, c, d, lam = la_bwd(q[rows], k[rows], v[rows], g[rows], S0, scale,
                                 dOt, dS_final[li])
        np.add.at(dq, rows, a)
        np.add.at(dk_, rows, b)
        np.add.at(dv_, rows, c)
        np.add.at(dg, rows, d)
        dS0[tr] += lam
    return dq, dk_, dv_, dg, dS0
