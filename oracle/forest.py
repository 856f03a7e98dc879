"""Segment-tree bookkeeping for the oracle (Sec. 2.1 and Sec. 3.3).

Segment v covers trajectory positions [s_v, e_v): s_v is its parent's end
(0 for a root) and e_v = s_v + len_v.  Positions restart at 0 in every tree,
so every tree has its own chunk grid.  Canonical compact rows: segments in id
order, tokens in order (row of position p in v = row0[v] + p - s_v).
"""
from __future__ import annotations

import numpy as np


def anchor(p: int, B: int) -> int:
    """Resume anchor a(p) = B * floor(p / B) (eq. resume-anchor)."""
    return B * (p // B)


class SegTree:
    """Validated forest with positions, children, trees and canonical rows."""

    def __init__(self, parent, seg_len):
        parent = [int(x) for x in parent]
        seg_len = [int(x) for x in seg_len]
        n = len(parent)
        if n == 0 or len(seg_len) != n:
            raise ValueError("empty forest or length mismatch")
        for v in range(n):
            if not (-1 <= parent[v] < n) or parent[v] == v:
                raise ValueError(f"bad parent of segment {v}")
            if seg_len[v] <= 0:
                raise ValueError(f"segment {v} has length {seg_len[v]}")
        self.n = n
        self.parent = parent
        self.len = seg_len
        self.kids = [[] for _ in range(n)]
        self.roots = []
        for v in range(n):
            (self.kids[parent[v]] if parent[v] >= 0 else self.roots).append(v)
        # preorder from the roots; a cycle leaves segments unreached
        self.pre = []
        self.tree = [-1] * n
        self.s = [0] * n
        self.e = [0] * n
        for t, r in enumerate(self.roots):
            stack = [r]
            while stack:
                v = stack.pop()
                self.tree[v] = t
                self.s[v] = self.e[parent[v]] if parent[v] >= 0 else 0
                self.e[v] = self.s[v] + seg_len[v]
                self.pre.append(v)
                stack.extend(reversed(self.kids[v]))
        if len(self.pre) != n:
            raise ValueError("parent array has a cycle")
        self.row0 = [0] * n
        acc = 0
        for v in range(n):
            self.row0[v] = acc
            acc += seg_len[v]
        self.C = acc
        self.leaves = [v for v in range(n) if not self.kids[v]]
        self.leaf_index = {v: i for i, v in enumerate(self.leaves)}

    def postorder(self):
        return list(reversed(self.pre))  # children after parents, reversed

    def path(self, v):
        """Segments root -> v."""
        out = []
        while v >= 0:
            out.append(v)
            v = self.parent[v]
        return out[::-1]

    def row_of(self, v, p):
        """Canonical compact row of trajectory position p on the path to v."""
        while not (self.s[v] <= p < self.e[v]):
            v = self.parent[v]
            if v < 0:
                raise ValueError("position not on path")
        return self.row0[v] + p - self.s[v]

    def trajectory_rows(self, leaf):
        rows = []
        for w in self.path(leaf):
            rows.extend(range(self.row0[w], self.row0[w] + self.len[w]))
        return rows

    def multiplicity(self):
        """q_v = number of leaves under v (eq. multiplicity, per segment)."""
        q = [0] * self.n
        for v in self.postorder():
            q[v] = 1 if not self.kids[v] else sum(q[u] for u in self.kids[v])
        return q

    def semantic_positions(self):
        """S = total length of all root-to-leaf trajectories."""
        return sum(self.e[l] for l in self.leaves)

    def mandatory_replay(self, B):
        """R = sum over internal v of (|ch(v)| - 1) (e_v mod B)
        (eq. mandatory-replay)."""
        return sum((len(self.kids[v]) - 1) * (self.e[v] % B)
                   for v in range(self.n) if self.kids[v])


def rows_to_array(rows):
    return np.asarray(rows, dtype=np.int64)
