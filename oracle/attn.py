"""Full attention over a rollout forest with asymmetric packed Q/KV views
(Sec. 4.2, "MLA execution with asymmetric packed Q/KV views"), the plain
definition in float64.  TEST INFRASTRUCTURE ONLY (see the package docstring).

Definition: along every root-to-leaf trajectory, causal softmax attention,
    o_t = sum_{j <= t} softmax_j(scale q_t . k_j) v_j,
per head.  A compact row's output is that of any trajectory through it (its
keys are its own ancestors and itself).  Gradients: the upstream gradient of
a compact row enters one trajectory through it, and per-trajectory gradients
are summed into compact rows (autograd of exactly this program).

Views: the query row of a branch holds its l own tokens, its key/value row
the h ancestor tokens followed by the same l tokens (eq. asymmetric-qkv);
query i may see key j iff j <= h + i, bottom-right alignment (eq.
bottom-right).  ``view_attention`` computes one branch that way; the tests
check that views reproduce the trajectory-wise definition.
"""
from __future__ import annotations

import numpy as np
import torch

from .forest import SegTree


def causal_attention(q, k, v, scale):
    """One sequence, torch float64: q, k, v [n, H, d] -> o [n, H, d]."""
    n = q.shape[0]
    s = torch.einsum("qhd,khd->hqk", q, k) * scale
    mask = torch.ones(n, n, dtype=torch.bool).tril()
    s = s.masked_fill(~mask, float("-inf"))
    p = torch.softmax(s, dim=-1)
    return torch.einsum("hqk,khd->qhd", p, v)


def view_attention(q_own, k_view, v_view, h, scale):
    """One branch: l own queries against h + l view keys, bottom-right
    causal: query i sees keys j <= h + i."""
    l = q_own.shape[0]
    kv = k_view.shape[0]
    assert kv == h + l
    s = torch.einsum("qhd,khd->hqk", q_own, k_view) * scale
    i = torch.arange(l)[:, None]
    j = torch.arange(kv)[None, :]
    s = s.masked_fill(~(j <= h + i), float("-inf"))
    p = torch.softmax(s, dim=-1)
    return torch.einsum("hqk,khd->qhd", p, v_view)


def forest_attention(parent, seg_len, q, k, v, scale, dO=None):
    """Trajectory-wise attention over a forest (canonical rows).  Returns o
    [C, H, d] and, with dO, (dq, dk, dv) by reverse mode of the same
    program, dO of a row entering its smallest-leaf-id trajectory."""
    t = SegTree(parent, seg_len)
    as64 = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.float64)
    qq, kk, vv = (as64(a).clone().requires_grad_(dO is not None) for a in (q, k, v))
    C = qq.shape[0]
    o = torch.zeros_like(qq)
    have = torch.zeros(C, dtype=torch.bool)
    loss = 0.0
    gO = as64(dO) if dO is not None else None
    for leaf in t.leaves:
        rows = torch.as_tensor(t.trajectory_rows(leaf), dtype=torch.long)
        ot = causal_attention(qq[rows], kk[rows], vv[rows], scale)
        new = ~have[rows]
        if dO is None:
            old = ~new
            if not torch.equal(o[rows[old]], ot[old].detach()):
                raise AssertionError("trajectories disagree on a shared row")
        o = o.index_put((rows[new],), ot[new].detach())
        if dO is not None:
            loss = loss + (ot[new] * gO[rows[new]]).sum()
        have[rows] = True
    out = {"o": o.detach().numpy()}
    if dO is not None:
        loss.backward()
        out.update(dq=qq.grad.numpy(), dk=kk.grad.numpy(), dv=vv.grad.numpy())
    return out
