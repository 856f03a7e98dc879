"""Brute-force minimum call count under the execution model of Sec. 3.3.

Independent of the dynamic program: enumerate, for every internal segment,
which child (or none) directly continues its input sequence; build the
sequences; give every sequence the earliest round its initial state allows:

* a root sequence runs in round 1 from its tree's initial state;
* a side child u of v needs S_{b_v}, b_v = a(e_v).  If b_v is the start
  anchor of v's sequence, that state is the sequence's own initial state and
  u can run in the same round; otherwise the state is produced inside v's
  call and u runs one round later (a state produced inside a call initialises
  another sequence only after the call returns).

The call count of a choice is its largest round; the minimum over all
choices is the minimum-call count the planner must reach.
"""
from __future__ import annotations

import itertools

from .forest import SegTree, anchor


def rounds_for_choice(t: SegTree, B: int, direct):
    """direct[v] = chosen child or -1 (for leaves ignored).  Returns
    (max round, list of sequences as (round, anchor, chain))."""
    seqs = []
    stack = []
    for r in t.roots:
        stack.append((r, 1, 0))            # (first segment, round, anchor)
    while stack:
        first, rnd, a = stack.pop()
        chain = [first]
        v = first
        while t.kids[v] and direct[v] >= 0:
            v = direct[v]
            chain.append(v)
        seqs.append((rnd, a, chain))
        for w in chain:
            for u in t.kids[w]:
                if u == direct[w]:
                    continue
                b = anchor(t.e[w], B)
                stack.append((u, rnd if b == a else rnd + 1, b))
    return max(s[0] for s in seqs), seqs


def min_calls(parent, seg_len, B: int):
    """Minimum over all direct-continuation choices (exponential)."""
    t = SegTree(parent, seg_len)
    internal = [v for v in range(t.n) if t.kids[v]]
    options = [t.kids[v] + [-1] for v in internal]
    best = None
    for pick in itertools.product(*options):
        direct = [-1] * t.n
        for v, c in zip(internal, pick):
            direct[v] = c
        k, _ = rounds_for_choice(t, B, direct)
        best = k if best is None else min(best, k)
    return best
