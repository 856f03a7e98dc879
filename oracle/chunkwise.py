"""Chunkwise form of the scalar-decay recurrence (torch float64 on the CPU).

Sec. 2.2 describes the training path: a sequence is cut into execution chunks
of B tokens from its start; inside a chunk everything is computed in parallel
and the state is carried from chunk to chunk.  For chunk c with initial state
S and in-chunk inclusive prefix sums G_i = g_0 + ... + g_i (per head):

    A      = (Q K^T) * exp(G_i - G_j) * [j <= i]
    O      = scale * (A V + (Q * exp(G)) S)
    S_next = exp(G_{B-1}) S + (K * exp(G_{B-1} - G))^T V

A partial last chunk is zero-padded to B rows (q = k = v = 0, g = 0), so every
chunk has one shape and one order of operations; padding adds nothing to the
state and its outputs are dropped.  Written with torch so that reverse-mode
differentiation of the same program gives gradients.
"""
from __future__ import annotations

import torch


def chunk_fwd(q, k, v, g, S, scale, B):
    """One sequence.  q,k: [n,H,dk]; v: [n,H,dv]; g: [n,H]; S: [H,dk,dv].

    Returns (o [n,H,dv], boundary states list [S_0, S_1, ..., S_nc]) where
    S_c is the state at the start of chunk c and S_nc the final state."""
    n, H, dk = q.shape
    dv = v.shape[2]
    nc = -(-n // B)
    pad = nc * B - n
    if pad:
        def z(x):
            return torch.cat([x, x.new_zeros((pad,) + x.shape[1:])], 0)
        q, k, v, g = z(q), z(k), z(v), z(g)
    causal = torch.tril(torch.ones(B, B, dtype=torch.bool))
    states = [S]
    outs = []
    for c in range(nc):
        sl = slice(c * B, (c + 1) * B)
        Q = q[sl].transpose(0, 1)                  # [H,B,dk]
        K = k[sl].transpose(0, 1)
        V = v[sl].transpose(0, 1)                  # [H,B,dv]
        G = torch.cumsum(g[sl], dim=0).transpose(0, 1)   # [H,B]
        diff = G[:, :, None] - G[:, None, :]
        D = torch.where(causal, torch.exp(torch.where(causal, diff,
                                                      torch.zeros_like(diff))),
                        torch.zeros_like(diff))
        A = (Q @ K.transpose(1, 2)) * D
        O = scale * (A @ V + (Q * torch.exp(G)[:, :, None]) @ S)
        GL = G[:, -1:]                              # [H,1]
        S = (torch.exp(GL)[:, :, None] * S
             + (K * torch.exp(GL - G)[:, :, None]).transpose(1, 2) @ V)
        states.append(S)
        outs.append(O.transpose(0, 1))
    o = torch.cat(outs, 0)[:n]
    return o, states
