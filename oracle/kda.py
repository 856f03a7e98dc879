"""KDA: linear attention with per-channel decay and the delta rule (Sec. 2.2,
eq. chunk-state), the plain definitions in float64.  TEST INFRASTRUCTURE
ONLY (see the package docstring).

Token recurrence, per head, state S in R^{dk x dv} (the KDA update whose
chunk-level form the paper prints as eq. chunk-state):

    S'  = Diag(exp(g_t)) S_{t-1}                 (per-channel decay, g_t <= 0)
    S_t = S' + beta_t k_t (v_t - S'^T k_t)^T     ((I - beta k k^T) S' + beta k v^T)
    o_t = scale * S_t^T q_t

Chunk form (eq. chunk-state), chunk of B tokens, start state S, local
cumulative log-decays G_i = g_1 + ... + g_i (per channel), Gamma_i = exp(G_i):
    A[i, j] = beta_i sum_d k_i[d] k_j[d] exp(G_i[d] - G_j[d])   (j < i)
    U       = (I + A)^{-1} Diag(beta) (V - (K * Gamma) S)       (= U' - W S)
    O       = scale ((Q * Gamma) S + M U),
              M[i, j] = sum_d q_i[d] k_j[d] exp(G_i[d] - G_j[d])  (j <= i)
    S_next  = Diag(Gamma_B) S + (K * exp(G_B - G))^T U
with U' = (I + A)^{-1} Diag(beta) V and W = (I + A)^{-1} Diag(beta) (K * Gamma).

Over a rollout forest: every root-to-leaf trajectory runs the recurrence from
its tree's initial state; a compact row's output is that of any trajectory
through it; gradients by reverse mode of exactly this program (the upstream
gradient of a compact row enters the trajectory of the smallest leaf id
through it, dS_final of a leaf enters its own trajectory).
"""
from __future__ import annotations

import numpy as np
import torch

from .forest import SegTree


def kda_recurrent(q, k, v, g, beta, scale, S0):
    """One sequence, torch float64.  q, k, g [n, H, dk]; v [n, H, dv];
    beta [n, H]; S0 [H, dk, dv].  Returns (o [n, H, dv], S_n)."""
    S = S0
    out = []
    for t in range(q.shape[0]):
        Sp = torch.exp(g[t])[:, :, None] * S                       # Diag(exp g) S
        pred = torch.einsum("hkv,hk->hv", Sp, k[t])                # S'^T k
        S = Sp + beta[t][:, None, None] * k[t][:, :, None] * (v[t] - pred)[:, None, :]
        out.append(scale * torch.einsum("hkv,hk->hv", S, q[t]))
    return torch.stack(out), S


def kda_chunkwise(q, k, v, g, beta, scale, S0, B):
    """The same sequence by chunks of B tokens in the form of eq. chunk-state
    (zero-padded last chunk: padding has g = 0, beta = 0, k = q = v = 0)."""
    n, H, dk = q.shape
    dv = v.shape[2]
    pad = (-n) % B
    P = lambda x: torch.cat([x, x.new_zeros((pad,) + x.shape[1:])]) if pad else x
    q, k, v, g, beta = P(q), P(k), P(v), P(g), P(beta)
    S = S0
    outs = []
    tri_strict = torch.tril(torch.ones(B, B, dtype=torch.bool), -1)
    tri = torch.tril(torch.ones(B, B, dtype=torch.bool))
    eye = torch.eye(B, dtype=q.dtype)
    for c0 in range(0, n + pad, B):
        sl = slice(c0, c0 + B)
        Q, K, V, Gs, b = q[sl], k[sl], v[sl], g[sl], beta[sl]      # [B, H, .]
        G = torch.cumsum(Gs, dim=0)                                 # [B, H, dk]
        diff = (G[:, None] - G[None, :]).masked_fill(~tri[:, :, None, None], float("-inf"))
        D = torch.exp(diff)                                         # [i, j, H, dk], 0 above the diagonal
        A = torch.einsum("ihd,jhd,ijhd->hij", K, K, D) * b.T[:, :, None]
        A = A * tri_strict
        M = torch.einsum("ihd,jhd,ijhd->hij", Q, K, D) * tri
        L = eye + A                                                 # [H, B, B]
        R = b.T[:, :, None] * (V.transpose(0, 1) - torch.einsum("ihd,hdv->hiv", K * torch.exp(G), S))
        U = torch.linalg.solve_triangular(L, R, upper=False, unitriangular=True)   # [H, B, dv]
        O = torch.einsum("ihd,hdv->hiv", Q * torch.exp(G), S) + torch.einsum("hij,hjv->hiv", M, U)
        outs.append(scale * O.transpose(0, 1))
        GB = G[-1]                                                  # [H, dk]
        S = torch.exp(GB)[:, :, None] * S + torch.einsum("ihd,hiv->hdv", K * torch.exp(GB[None] - G), U)
    return torch.cat(outs)[:n], S


def kda_forest(parent, seg_len, q, k, v, g, beta, scale, S0_tree, dO=None, dS_final=None):
    """Trajectory-wise KDA over a forest (canonical rows).  q, k, g [C, H, dk],
    v [C, H, dv], beta [C, H], S0_tree [n_trees, H, dk, dv].  Returns o
    [C, H, dv] and S_final [n_leaves, H, dk, dv] (leaves by ascending id)
    and, with dO (and optionally dS_final), the gradients dq, dk, dv, dg,
    dbeta and dS0_tree."""
    t = SegTree(parent, seg_len)
    as64 = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.float64)
    grad = dO is not None
    xs = [as64(a).clone().requires_grad_(grad) for a in (q, k, v, g, beta, S0_tree)]
    qq, kk, vv, gg, bb, S0 = xs
    C = qq.shape[0]
    o = torch.zeros(C, qq.shape[1], vv.shape[2], dtype=torch.float64)
    have = torch.zeros(C, dtype=torch.bool)
    finals = []
    loss = 0.0
    gO = as64(dO) if grad else None
    gS = as64(dS_final) if grad and dS_final is not None else None
    for li, leaf in enumerate(t.leaves):
        rows = torch.as_tensor(t.trajectory_rows(leaf), dtype=torch.long)
        ot, St = kda_recurrent(qq[rows], kk[rows], vv[rows], gg[rows], bb[rows], scale, S0[t.tree[leaf]])
        new = ~have[rows]
        if not grad and not torch.equal(o[rows[~new]], ot[~new]):
            raise AssertionError("trajectories disagree on a shared row")
        o = o.index_put((rows[new],), ot[new].detach())
        finals.append(St.detach())
        if grad:
            loss = loss + (ot[new] * gO[rows[new]]).sum()
            if gS is not None:
                loss = loss + (St * gS[li]).sum()
        have[rows] = True
    out = {"o": o.numpy(), "S_final": torch.stack(finals).numpy()}
    if grad:
        loss.backward()
        for name, x in zip(("dq", "dk", "dv", "dg", "dbeta", "dS0_tree"), xs):
            out[name] = x.grad.numpy()
    return out
