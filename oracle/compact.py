"""Compact (tree-packed) execution of a plan, in float64 on the CPU.

Runs the rounds produced by ``plan_ref`` (Algorithm "minimum-call", Sec. 3.3)
with the chunkwise form of ``chunkwise.chunk_fwd``:

* each sequence starts at its anchor from its initial state, which is either
  its tree's initial state or a boundary state written by an earlier round
  (eq. chunkla-interface: a call returns the requested chunk-boundary states
  and the final state of every sequence);
* the fixed replay interval [anchor, first segment start) is read from the
  ancestor's compact rows and only updates the state (Sec. 3.3 "Fixed replay"
  and Sec. 3.4 "Round-wise execution"); only own rows produce outputs;
* a shared boundary state is one tensor read by every consumer, so
  differentiation sums all consumer gradients into it (Sec. 3.4,
  "Differentiable boundary states").

Gradients are obtained by reverse-mode differentiation (torch.autograd) of
exactly this program, which is the definition of the backward pass; the
tests tie it to the hand-derived trajectory-wise backward and to finite
differences.  Rows are canonical (segments in id order).
"""
from __future__ import annotations

import torch

from .chunkwise import chunk_fwd
from .forest import SegTree
from .plan_ref import plan_ref


def sequence_rows(t: SegTree, plan, i):
    """Canonical (replay_rows, own_rows) of sequence i of the plan."""
    a, b = int(plan["seq_chain_off"][i]), int(plan["seq_chain_off"][i + 1])
    chain = [int(x) for x in plan["chain_seg"][a:b]]
    first = chain[0]
    rep = [t.row_of(first, p) for p in range(int(plan["seq_anchor"][i]),
                                             t.s[first])]
    own = []
    for v in chain:
        own.extend(range(t.row0[v], t.row0[v] + t.len[v]))
    return rep, own


def compact_fwd(parent, seg_len, B, q, k, v, g, scale, S0_tree, plan=None):
    """Forward over all rounds.  q,k,v,g canonical torch float64 tensors,
    S0_tree [n_trees,H,dk,dv].  Returns dict with o, S_final, seq_S0 (the
    initial-state tensor of every sequence, one node each), bank."""
    t = SegTree(parent, seg_len)
    if plan is None:
        plan = plan_ref(parent, seg_len, B)
    C, H, dk = q.shape
    dv = v.shape[2]
    bank = [None] * plan["n_bank"]
    for tr in range(plan["n_trees"]):
        bank[tr] = S0_tree[tr]
    o = torch.zeros(C, H, dv, dtype=q.dtype)
    S_final = [None] * plan["n_leaves"]
    seq_S0 = []
    for i in range(plan["n_seq"]):
        rep, own = sequence_rows(t, plan, i)
        rows = torch.as_tensor(rep + own, dtype=torch.long)
        init = int(plan["seq_init_bank"][i])
        S_init = bank[init] * 1.0            # own graph node per consumer
        seq_S0.append(S_init)
        o_seq, states = chunk_fwd(q[rows], k[rows], v[rows], g[rows], S_init,
                                  scale, B)
        own_t = torch.as_tensor(own, dtype=torch.long)
        o = o.index_put((own_t,), o_seq[len(rep):])
        r0, r1 = int(plan["seq_req_off"][i]), int(plan["seq_req_off"][i + 1])
        for j in range(r0, r1):
            bank[int(plan["req_bank"][j])] = states[int(plan["req_chunk"][j])]
        S_final[int(plan["seq_final_leaf"][i])] = states[-1]
    return dict(o=o, S_final=torch.stack(S_final), seq_S0=seq_S0, bank=bank,
                plan=plan)


def compact_fwd_bwd(parent, seg_len, B, q, k, v, g, scale, dO, dS_final,
                    S0_tree, plan=None):
    """Forward plus gradients of <dO, o> + <dS_final, S_final> (float64).

    Returns numpy arrays: o, S_final, dq, dk, dv, dg, dS0_tree and dS0_seq
    [n_seq,H,dk,dv] (the gradient at every sequence's initial state)."""
    as64 = lambda x: torch.as_tensor(x, dtype=torch.float64)
    leaves = [as64(x).clone().requires_grad_(True) for x in (q, k, v, g, S0_tree)]
    qq, kk, vv, gg, SS = leaves
    out = compact_fwd(parent, seg_len, B, qq, kk, vv, gg, scale, SS, plan)
    loss = ((out["o"] * as64(dO)).sum()
            + (out["S_final"] * as64(dS_final)).sum())
    grads = torch.autograd.grad(loss, leaves + out["seq_S0"])
    np_ = lambda x: x.detach().numpy()
    return dict(o=np_(out["o"]), S_final=np_(out["S_final"]),
                dq=np_(grads[0]), dk=np_(grads[1]), dv=np_(grads[2]),
                dg=np_(grads[3]), dS0_tree=np_(grads[4]),
                dS0_seq=torch.stack(grads[5:]).numpy(), plan=out["plan"])
