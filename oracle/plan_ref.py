"""Reference minimum-call planner (Sec. 3.3, Algorithm "minimum-call").

Written from the paper's definitions, in a structure of its own:

* the minimum call counts of every subtree, T_pre and T_in, straight from
  eqs. leaf-calls, tin and tpre with the early-start condition eq.
  early-start (e_v < a_v + B), children visited in postorder;
* recovery as a feasibility test against one deadline per tree: the tree's
  rounds are 1 .. D with D = T_pre(root), and every segment of it must finish
  by round D.  A segment v reached in round r continues its sequence with the
  first child (in child order) whose own subtree still finishes by D when
  continued in the same sequence, provided every other child, started as a
  side branch in the earliest round its anchor state S_{b_v} allows, also
  finishes by D.  (The printed procedure's round budgets K_round and K_side
  are this deadline counted from r and from the side branches' start round.)

A side branch starts in round r itself when v's entry anchor state was ready
before round r and v crosses no chunk boundary (e_v < a_v + B), from v's
sequence's own initial state; otherwise in round r + 1 from S_{b_v},
requested from v's sequence.  The direct child inherits "ready" exactly in
the first case: its entry state is then the same ready anchor state.

Conventions where the paper leaves a choice (the library follows the same):

* children are visited in ascending segment id ("a fixed child order");
* sequences are created in the order of a depth-first recovery that finishes
  the direct continuation's subtree before launching a segment's side
  branches, side branches in child order (each with its whole subtree), and
  trees in ascending root id; sequence ids are a stable sort of that creation
  order on the round number;
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

import numpy as np

from .forest import SegTree, anchor


def early_start(t: SegTree, v: int, B: int) -> bool:
    """eq. early-start: v ends before the chunk boundary after its entry
    anchor a_v, so it produces no new boundary state (b_v = a_v)."""
    return t.e[v] < anchor(t.s[v], B) + B


def dp_calls(t: SegTree, B: int):
    """T_pre and T_in for every segment (eqs. leaf-calls, tin, tpre)."""
    T_pre = [0] * t.n
    T_in = [0] * t.n
    for v in t.postorder():
        ch = t.kids[v]
        if not ch:                                    # eq. leaf-calls
            T_pre[v] = T_in[v] = 1
            continue
        # eq. tin: the direct child o keeps the call; every other child
        # waits one round for its anchor state (max over an empty set = 0)
        T_in[v] = min(max(T_in[o], 1 + max([T_pre[u] for u in ch if u != o], default=0))
                      for o in ch)
        # eq. tpre
        T_pre[v] = max(T_pre[u] for u in ch) if early_start(t, v, B) else T_in[v]
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

    def grow(q, first, ready, deadline, todo):
        """Extend sequence q from segment `first` (entered with its anchor
        state ready before q's round, or not) down its chain of direct
        continuations; queue every side branch on `todo` so that the side
        branches of deeper chain segments are launched first."""
        v, r = first, q.round
        launches = []
        while True:
            q.chain.append(v)
            seg_seq[v] = q
            ch = t.kids[v]
            if not ch:
                break
            same_round = ready and early_start(t, v, B)
            side_round = r if same_round else r + 1
            # finishing by the deadline: a subtree entering round x with a
            # count of T rounds ends in round x + T - 1
            side_ok = [side_round + T_pre[u] - 1 <= deadline for u in ch]
            direct = None
            for o in ch:
                need = T_pre[o] if same_round else T_in[o]
                if r + need - 1 <= deadline and all(ok for u, ok in zip(ch, side_ok) if u != o):
                    direct = o
                    break
            assert direct is not None, "no child meets the tree's deadline"
            launches.append((v, same_round, side_round,
                             [u for u in ch if u != direct]))
            v, ready = direct, same_round
        # deepest segment's side branches first; within a segment, child order
        for v, same_round, side_round, sides in launches:
            todo.extend((v, same_round, side_round, u) for u in reversed(sides))

    K_tree = []
    for ti, root in enumerate(t.roots):
        D = T_pre[root]                  # the root's zero state is ready before round 1
        K_tree.append(D)
        todo = []
        grow(new_seq(ti, 1, 0, ("tree", ti)), root, True, D, todo)
        while todo:
            v, same_round, side_round, u = todo.pop()
            q = seg_seq[v]
            b_v = anchor(t.e[v], B)
            if same_round:               # b_v = a_v: the sequence's own initial state
                assert b_v == q.anchor
                qu = new_seq(ti, side_round, b_v, q.init)
            else:
                requests.append((q, b_v))
                qu = new_seq(ti, side_round, b_v, ("slot", q, b_v))
            grow(qu, u, True, D, todo)
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
