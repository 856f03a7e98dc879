"""Reference minimum-call planner: Algorithm "minimum-call" of Sec. 3.3.

Written from the paper's statement of the dynamic program (eqs. leaf-calls,
tin, tpre with the early-start condition eq. early-start) and of the Recover
procedure; plain recursive Python, no tricks.

Conventions where the paper leaves a choice (the library follows the same):

* children are visited in ascending segment id ("a fixed child order");
* sequences are created in Recover's order (the direct continuation is
  recursed into before the side children are launched, side children in
  child order), trees in ascending root id; sequence ids are assigned by a
  stable sort of that creation order on the round number;
* a side branch launched in the same round reuses its parent sequence's
  initial-state source; one launched in the next round consumes the boundary
  state S_{b_v} requested from the parent's sequence;
* requested states are deduplicated by (producer sequence, boundary position)
  and numbered by that pair; the state bank holds one initial state per tree
  first, then the requested slots;
* physical rows: sequences in id order, chain segments in order;
* a sequence's final state goes to the leaf ending its chain (leaf index =
  rank of the leaf among all leaves by id).
"""
from __future__ import annotations

import sys

import numpy as np

from .forest import SegTree, anchor


def dp_calls(t: SegTree, B: int):
    """T_pre and T_in for every segment (eqs. leaf-calls, tin, tpre)."""
    T_pre = [0] * t.n
    T_in = [0] * t.n
    for v in t.postorder():
        ch = t.kids[v]
        if not ch:
            T_pre[v] = T_in[v] = 1
            continue
        best = None
        for o in ch:
            others = [T_pre[u] for u in ch if u != o]
            h = max(others) if others else 0      # max of an empty set is 0
            cand = max(T_in[o], 1 + h)
            best = cand if best is None else min(best, cand)
        T_in[v] = best
        if t.e[v] < anchor(t.s[v], B) + B:        # early start (strict)
            T_pre[v] = max(T_pre[u] for u in ch)
        else:
            T_pre[v] = T_in[v]
    return T_pre, T_in


class _Seq:
    def __init__(self, tree, rnd, anchor_pos, init, creation):
        self.tree = tree
        self.round = rnd
        self.anchor = anchor_pos
        self.init = init          # ("tree", t) or ("slot", producer _Seq, pos)
        self.chain = []
        self.creation = creation
        self.id = -1


def plan_ref(parent, seg_len, B: int):
    """Plan a forest.  Returns a dict of plain Python / numpy results."""
    if B < 1:
        raise ValueError("chunk size must be >= 1")
    t = SegTree(parent, seg_len)
    T_pre, T_in = dp_calls(t, B)
    seqs = []
    requests = []                 # (producer _Seq, position)
    seg_seq = [None] * t.n

    def new_seq(tree, rnd, a, init):
        q = _Seq(tree, rnd, a, init, len(seqs))
        seqs.append(q)
        return q

    def recover(v, ready, K, r, q):
        q.chain.append(v)
        seg_seq[v] = q
        ch = t.kids[v]
        if not ch:
            return
        same = ready and (t.e[v] < anchor(t.s[v], B) + B)
        delta = 0 if same else 1
        K_side = K - delta
        need = {o: (T_pre[o] if same else T_in[o]) for o in ch}
        f = sum(1 for u in ch if T_pre[u] > K_side)
        o = None
        for c in ch:
            if need[c] <= K and f - (1 if T_pre[c] > K_side else 0) == 0:
                o = c
                break
        assert o is not None, "round budget infeasible"
        recover(o, same, K, r, q)
        b_v = anchor(t.e[v], B)
        for u in ch:
            if u == o:
                continue
            if same:
                assert b_v == q.anchor
                qu = new_seq(q.tree, r, b_v, q.init)
            else:
                requests.append((q, b_v))
                qu = new_seq(q.tree, r + 1, b_v, ("slot", q, b_v))
            recover(u, True, K_side, r + delta, qu)

    old_limit = sys.getrecursionlimit()
    sys.setrecursionlimit(max(old_limit, 4 * t.n + 1000))
    try:
        K_tree = []
        for ti, root in enumerate(t.roots):
            K_root = T_pre[root]
            K_tree.append(K_root)
            q0 = new_seq(ti, 1, 0, ("tree", ti))
            recover(root, True, K_root, 1, q0)
    finally:
        sys.setrecursionlimit(old_limit)
    K = max(K_tree)

    order = sorted(seqs, key=lambda q: (q.round, q.creation))
    for i, q in enumerate(order):
        q.id = i
    assert all(1 <= q.round <= K for q in order)

    slot_keys = sorted({(p.id, pos) for p, pos in requests})
    slot_of = {key: j for j, key in enumerate(slot_keys)}
    n_trees = len(t.roots)

    def bank_of(init):
        if init[0] == "tree":
            return init[1]
        return n_trees + slot_of[(init[1].id, init[2])]

    # physical rows
    seg_row = [0] * t.n
    row = 0
    seq_row, seq_n_own = [], []
    for q in order:
        seq_row.append(row)
        n_own = 0
        for v in q.chain:
            seg_row[v] = row
            row += t.len[v]
            n_own += t.len[v]
        seq_n_own.append(n_own)

    # replay rows (physical) and requests per sequence
    replay_rows, seq_n_replay, seq_replay_off = [], [], []
    req_chunk, req_bank, seq_req_off = [], [], []
    req_by_seq = {}
    for (pid, pos), j in slot_of.items():
        req_by_seq.setdefault(pid, []).append((pos, j))
    for q in order:
        first = q.chain[0]
        seq_replay_off.append(len(replay_rows))
        n_rep = t.s[first] - q.anchor
        assert 0 <= n_rep < B
        v = t.parent[first]
        rows = []
        for p in range(q.anchor, t.s[first]):
            w = first
            while not (t.s[w] <= p < t.e[w]):
                w = t.parent[w]
            rows.append(seg_row[w] + p - t.s[w])
        replay_rows.extend(rows)
        seq_n_replay.append(n_rep)
        seq_req_off.append(len(req_chunk))
        for pos, j in sorted(req_by_seq.get(q.id, [])):
            assert (pos - q.anchor) % B == 0 and pos > q.anchor
            req_chunk.append((pos - q.anchor) // B)
            req_bank.append(n_trees + j)
    seq_req_off.append(len(req_chunk))
    seq_replay_off.append(len(replay_rows))

    round_seq_off = [0] * (K + 1)
    for q in order:
        round_seq_off[q.round] += 1
    for r in range(1, K + 1):
        round_seq_off[r] += round_seq_off[r - 1]

    chain_seg, seq_chain_off = [], []
    for q in order:
        seq_chain_off.append(len(chain_seg))
        chain_seg.extend(q.chain)
    seq_chain_off.append(len(chain_seg))

    i64 = lambda x: np.asarray(x, dtype=np.int64)
    i32 = lambda x: np.asarray(x, dtype=np.int32)
    R = len(replay_rows)
    return dict(
        K=K, n_seq=len(order), n_slots=len(slot_keys), n_trees=n_trees,
        n_bank=n_trees + len(slot_keys), n_leaves=len(t.leaves),
        C=t.C, S=t.semantic_positions(), R=R, chunk=B,
        K_tree=i32(K_tree),
        seg_start=i64(t.s), seg_end=i64(t.e), seg_row=i64(seg_row),
        seg_seq=i32([seg_seq[v].id for v in range(t.n)]),
        seg_mult=i64(t.multiplicity()), seg_tpre=i32(T_pre), seg_tin=i32(T_in),
        seg_tree=i32(t.tree), leaf_seg=i32(t.leaves),
        round_seq_off=i32(round_seq_off),
        seq_round=i32([q.round for q in order]),
        seq_tree=i32([q.tree for q in order]),
        seq_first_seg=i32([q.chain[0] for q in order]),
        seq_final_leaf=i32([t.leaf_index[q.chain[-1]] for q in order]),
        seq_init_bank=i32([bank_of(q.init) for q in order]),
        seq_anchor=i64([q.anchor for q in order]),
        seq_n_replay=i64(seq_n_replay), seq_replay_off=i64(seq_replay_off),
        seq_row=i64(seq_row), seq_n_own=i64(seq_n_own),
        seq_chain_off=i32(seq_chain_off), chain_seg=i32(chain_seg),
        seq_req_off=i32(seq_req_off), req_chunk=i32(req_chunk),
        req_bank=i32(req_bank),
        slot_seq=i32([k[0] for k in slot_keys]),
        slot_pos=i64([k[1] for k in slot_keys]),
        replay_row=i64(replay_rows),
    )
