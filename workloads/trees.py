"""Seeded synthetic rollout forests.

A forest is given the way the planner consumes it: ``parent[v]`` (-1 for a
root) and ``seg_len[v]`` (> 0) for every segment v, a segment being a
fork-free run of tokens (Sec. 3.3, "Execution model").  Children of a segment
are ordered by ascending id, trees by the ascending id of their roots.

The shapes stand in for the paper's SWE-bench-derived rollout trees, which are
not available: microbatch capacity 65,536, a long shared task prefix and
several retries per task (Sec. 1, Sec. 5.1, Table "planner").  Every draw is
seeded; a rejected microbatch is redrawn from sub-seed (seed, j+1).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

CHUNK = 64

# Workload table.  Sizes follow the five benchmark configurations of the
# build: the Figure-1 tree, random spine trees, and agentic trees scaled by a
# single length factor ``lam`` so that the compact-row total hits its target.
CONFIGS = {
    0: dict(kind="fig1", H=4, d=64, dtype="f32", seed=0),
    1: dict(kind="spine", n_trees=4, H=16, d=128, dtype="bf16", seed=1,
            c_range=(12288, 20480)),
    2: dict(kind="agentic", n_trees=8, lam=0.21, target=65536, H=16, d=128,
            dtype="bf16", seed=2),
    3: dict(kind="agentic", n_trees=32, lam=0.104, target=131072,
            depth_cap=6, H=32, d=128, dtype="bf16", seed=3),
    4: dict(kind="agentic", n_trees=4, lam=0.21, target=32768, H=16, d=128,
            dtype="bf16", seed=4),
}


@dataclass
class Forest:
    parent: np.ndarray          # int32 [n_seg], -1 marks a root
    seg_len: np.ndarray         # int64 [n_seg], every entry > 0
    meta: dict = field(default_factory=dict)

    @property
    def n_seg(self) -> int:
        return int(self.parent.shape[0])

    @property
    def n_rows(self) -> int:
        """Compact rows C: every token of every segment, stored once."""
        return int(self.seg_len.sum())

    def children(self):
        ch = [[] for _ in range(self.n_seg)]
        for v, p in enumerate(self.parent.tolist()):
            if p >= 0:
                ch[p].append(v)
        return ch

    def leaves(self):
        ch = self.children()
        return [v for v in range(self.n_seg) if not ch[v]]


def _concat(trees):
    """Concatenate per-tree (parent, len) lists into one forest (ids shifted)."""
    parent, seg_len = [], []
    for p_list, l_list in trees:
        base = len(parent)
        parent += [(-1 if p < 0 else p + base) for p in p_list]
        seg_len += list(l_list)
    return np.asarray(parent, np.int32), np.asarray(seg_len, np.int64)


def figure1_forest() -> Forest:
    """The Figure-1 tree: A -> {B -> {D, E}, C} with unaligned forks.

    ids: A=0, B=1, C=2, D=3, E=4; lengths A=200, B=77, C=90, D=64, E=50.
    """
    parent = np.array([-1, 0, 0, 1, 1], np.int32)
    seg_len = np.array([200, 77, 90, 64, 50], np.int64)
    return Forest(parent, seg_len, dict(kind="fig1", names="ABCDE"))


def _spine_tree(rng):
    depth = int(rng.integers(2, 5))             # U{2,3,4} spine levels
    parent = [-1]
    spine = 0
    for _ in range(depth - 1):
        fan = int(rng.integers(1, 5))           # U{1..4} children
        kids = []
        for _ in range(fan):
            parent.append(spine)
            kids.append(len(parent) - 1)
        spine = kids[0]                          # first child continues the spine
    n = len(parent)
    has_child = [False] * n
    for p in parent:
        if p >= 0:
            has_child[p] = True
    seg_len = [0] * n
    end = [0] * n
    for v in range(n):                           # parents precede children
        start = end[parent[v]] if parent[v] >= 0 else 0
        while True:
            length = int(rng.integers(16, 2049))  # U[16, 2048]
            if not has_child[v] or (start + length) % CHUNK != 0:
                break                            # forks avoid chunk boundaries
        seg_len[v] = length
        end[v] = start + length
    return parent, seg_len


def spine_forest(seed: int, n_trees: int = 4, c_range=(12288, 20480),
                 max_tries: int = 10000):
    """Random spine trees; redraw the microbatch until C lies in ``c_range``.

    Returns (forest, rng) with ``rng`` positioned after the tree draws.
    """
    for j in range(max_tries):
        rng = np.random.default_rng([seed, j])
        trees = [_spine_tree(rng) for _ in range(n_trees)]
        parent, seg_len = _concat(trees)
        c = int(seg_len.sum())
        if c_range[0] <= c <= c_range[1]:
            return Forest(parent, seg_len, dict(kind="spine", seed=seed,
                                                subseed=j)), rng
    raise RuntimeError("spine_forest: no accepted draw")


def _canonical(parent, seg_len):
    """Merge fork-free chains and renumber in preorder (children by old id)."""
    n = len(parent)
    kids = [[] for _ in range(n)]
    roots = []
    for v in range(n):
        (kids[parent[v]] if parent[v] >= 0 else roots).append(v)
    new_parent, new_len = [], []
    stack = [(r, -1) for r in reversed(roots)]
    while stack:
        v, p_new = stack.pop()
        length = seg_len[v]
        while len(kids[v]) == 1:                 # a segment has no inner fork
            v = kids[v][0]
            length += seg_len[v]
        me = len(new_parent)
        new_parent.append(p_new)
        new_len.append(length)
        for c in reversed(kids[v]):
            stack.append((c, me))
    return new_parent, new_len


def _depth_of(parent, v):
    d = 1
    while parent[v] >= 0:
        v = parent[v]
        d += 1
    return d


def _agentic_tree(rng, lam, depth_cap=None):
    """One agentic rollout tree: a long task prefix, then retries.

    Root prefix ~ U_int[8192, 32768] * lam.  A first branch follows it; every
    further leaf forks from the most recently added leaf at a uniform offset
    inside that leaf's own segment (offset 0 forks at the segment's start),
    the way a retry restarts from some point of the failed attempt.  Branch
    lengths are LogNormal(ln(1500 lam), 1).
    """
    def branch_len():
        return max(1, int(round(rng.lognormal(np.log(1500.0 * lam), 1.0))))

    parent = [-1]
    seg_len = [max(1, int(round(int(rng.integers(8192, 32769)) * lam)))]
    n_leaves = int(rng.integers(3, 13))          # U{3..12}
    parent.append(0)
    seg_len.append(branch_len())
    last = 1
    for _ in range(n_leaves - 1):
        off = int(rng.integers(0, seg_len[last]))
        if off > 0 and depth_cap is not None:
            if _depth_of(parent, last) + 1 > depth_cap:
                off = 0                          # a deeper fork is rejected
        if off == 0:
            fork_at = parent[last]
        else:                                    # split `last` at `off`
            head = len(parent)
            parent.append(parent[last])
            seg_len.append(off)
            parent[last] = head
            seg_len[last] -= off
            fork_at = head
        parent.append(fork_at)
        seg_len.append(branch_len())
        last = len(parent) - 1
    return _canonical(parent, seg_len)


def agentic_forest(seed: int, n_trees: int, lam: float, target: int,
                   depth_cap=None, tol: float = 0.05, max_tries: int = 10000):
    """``n_trees`` agentic trees; redraw until |C - target| <= tol * target."""
    for j in range(max_tries):
        rng = np.random.default_rng([seed, j])
        trees = [_agentic_tree(rng, lam, depth_cap) for _ in range(n_trees)]
        parent, seg_len = _concat(trees)
        c = int(seg_len.sum())
        if abs(c - target) <= tol * target:
            return Forest(parent, seg_len,
                          dict(kind="agentic", seed=seed, subseed=j, lam=lam,
                               depth_cap=depth_cap)), rng
    raise RuntimeError("agentic_forest: no accepted draw")


def forest_for_config(idx: int):
    """(forest, rng, cfg) for a workload; ``rng`` continues with tensor draws."""
    cfg = dict(CONFIGS[idx])
    if cfg["kind"] == "fig1":
        return figure1_forest(), np.random.default_rng(cfg["seed"]), cfg
    if cfg["kind"] == "spine":
        f, rng = spine_forest(cfg["seed"], cfg["n_trees"], cfg["c_range"])
        return f, rng, cfg
    f, rng = agentic_forest(cfg["seed"], cfg["n_trees"], cfg["lam"],
                            cfg["target"], cfg.get("depth_cap"))
    return f, rng, cfg


def trajectory_tokens(forest: Forest, rng, vocab: int = 157184):
    """Token sequences of every root-to-leaf trajectory (leaves by ascending
    id): one seeded token id per compact row, read along each path, so that
    trajectories of one tree share exactly their common prefix."""
    tok = rng.integers(0, vocab, size=forest.n_rows).astype(np.int32)
    row0 = np.concatenate([[0], np.cumsum(forest.seg_len)[:-1]])
    out = []
    for leaf in forest.leaves():
        path, v = [], leaf
        while v >= 0:
            path.append(v)
            v = int(forest.parent[v])
        out.append(np.concatenate([tok[row0[w]:row0[w] + forest.seg_len[w]] for w in reversed(path)]))
    return out
