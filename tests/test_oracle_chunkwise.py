"""Self-checks of the oracle's chunkwise and compact forms (CPU only).

1. chunkwise == recurrent for B in {1, 2, 3, 4, 64} (B = 1 is the recurrence);
2. compact execution of the plan == trajectory-wise chunkwise execution,
   bitwise, at every shared token and for every leaf's final state, and
   == the recurrence to 1e-12;
3. gradients of the compact program == the hand-derived trajectory-wise
   backward, and the gradient at every sequence's initial state == its
   trajectory-wise definition (adjoint at the anchor summed over the
   trajectories that depend on that initial state).
"""
import numpy as np
import pytest
import torch

from oracle import recurrent
from oracle.chunkwise import chunk_fwd
from oracle.compact import compact_fwd, compact_fwd_bwd
from oracle.forest import SegTree
from oracle.plan_ref import plan_ref

t64 = lambda x: torch.as_tensor(np.asarray(x), dtype=torch.float64)


def _inputs(C, H, dk, dv, n_leaves, n_trees, seed):
    r = np.random.default_rng(seed)
    q = r.standard_normal((C, H, dk))
    k = r.standard_normal((C, H, dk))
    q /= np.linalg.norm(q, axis=-1, keepdims=True)
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = r.standard_normal((C, H, dv))
    g = r.uniform(-0.1, -0.001, size=(C, H))
    dO = r.standard_normal((C, H, dv))
    dSf = r.standard_normal((n_leaves, H, dk, dv))
    S0 = r.standard_normal((n_trees, H, dk, dv)) * 0.5
    return q, k, v, g, dO, dSf, S0


def _random_forest(r, n, B, max_trees=2):
    parent = [-1]
    for v in range(1, n):
        parent.append(-1 if (r.random() < 0.15 and
                             parent.count(-1) < max_trees) else int(r.integers(0, v)))
    seg_len = [int(x) for x in r.integers(1, 2 * B + 2, size=n)]
    return parent, seg_len


def _rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


@pytest.mark.parametrize("B", [1, 2, 3, 4, 64])
def test_chunkwise_equals_recurrent(B):
    n, H, dk, dv = 150, 2, 5, 4
    q, k, v, g, _, _, S0 = _inputs(n, H, dk, dv, 1, 1, seed=B)
    o_ref, S_ref = recurrent.la_fwd(q, k, v, g, S0[0], 0.4)
    o, states = chunk_fwd(t64(q), t64(k), t64(v), t64(g), t64(S0[0]), 0.4, B)
    assert _rel(o.numpy(), o_ref) <= 1e-12
    assert _rel(states[-1].numpy(), S_ref) <= 1e-12
    # boundary state at every chunk start equals the recurrence's state there
    for c in range(1, len(states) - 1):
        _, Sc = recurrent.la_fwd(q[:c * B], k[:c * B], v[:c * B], g[:c * B],
                                 S0[0], 0.4)
        assert _rel(states[c].numpy(), Sc) <= 1e-12


FORESTS = [
    ([-1, 0, 0, 1, 1], [200, 77, 90, 64, 50], 64),     # Figure 1 workload
    ([-1, 0, 0, 1, 1], [63, 2, 10, 20, 30], 64),       # Figure 2 workload
    ([-1, 0, 0, 0], [158, 40, 50, 60], 64),            # Figure 3 workload
]


def _compare_compact_to_trajectories(parent, seg_len, B, seed, H=2, dk=4, dv=3):
    t = SegTree(parent, seg_len)
    q, k, v, g, dO, dSf, S0 = _inputs(t.C, H, dk, dv, len(t.leaves),
                                      len(t.roots), seed)
    out = compact_fwd(parent, seg_len, B, t64(q), t64(k), t64(v), t64(g), 0.5,
                      t64(S0))
    o_c = out["o"].numpy()
    Sf_c = out["S_final"].numpy()
    for li, leaf in enumerate(t.leaves):
        rows = t.trajectory_rows(leaf)
        o_t, st = chunk_fwd(t64(q[rows]), t64(k[rows]), t64(v[rows]),
                            t64(g[rows]), t64(S0[t.tree[leaf]]), 0.5, B)
        assert np.array_equal(o_c[rows], o_t.numpy()), "compact != trajectory"
        assert np.array_equal(Sf_c[li], st[-1].numpy())
    o_r, Sf_r = recurrent.forest_fwd(parent, seg_len, q, k, v, g, 0.5, S0)
    assert _rel(o_c, o_r) <= 1e-12
    assert _rel(Sf_c, Sf_r) <= 1e-12


@pytest.mark.parametrize("parent,seg_len,B", FORESTS)
def test_compact_equals_trajectorywise_figures(parent, seg_len, B):
    _compare_compact_to_trajectories(parent, seg_len, B, seed=sum(seg_len))


@pytest.mark.parametrize("B", [2, 3, 4])
def test_compact_equals_trajectorywise_random(B):
    r = np.random.default_rng(100 + B)
    for trial in range(12):
        n = int(r.integers(1, 8))
        parent, seg_len = _random_forest(r, n, B)
        _compare_compact_to_trajectories(parent, seg_len, B, seed=trial)


def _traj_dS0_seq(parent, seg_len, B, plan, q, k, v, g, S0, scale, dO, dSf):
    """Trajectory-wise gradient at each sequence's initial state."""
    t = SegTree(parent, seg_len)
    n_seq = plan["n_seq"]
    owner = np.zeros(t.C, np.int64)
    leaf_of_seq = []
    for i in range(n_seq):
        a, b = plan["seq_chain_off"][i], plan["seq_chain_off"][i + 1]
        chain = [int(x) for x in plan["chain_seg"][a:b]]
        for w in chain:
            owner[t.row0[w]:t.row0[w] + t.len[w]] = i
        leaf_of_seq.append(chain[-1])
    anc = []
    for i in range(n_seq):
        bnk = int(plan["seq_init_bank"][i])
        anc.append(-1 if bnk < plan["n_trees"]
                   else int(plan["slot_seq"][bnk - plan["n_trees"]]))

    def depends(w, u):
        while w >= 0:
            if w == u:
                return True
            w = anc[w]
        return False

    out = np.zeros((n_seq,) + S0.shape[1:])
    for u in range(n_seq):
        A = int(plan["seq_anchor"][u])
        for i in range(n_seq):
            if not depends(i, u):
                continue
            leaf = leaf_of_seq[i]
            rows = np.asarray(t.trajectory_rows(leaf))
            keep = np.array([depends(int(owner[c]), u) and
                             leaf_of_seq[int(owner[c])] == leaf for c in rows])
            _, SA = recurrent.la_fwd(q[rows[:A]], k[rows[:A]], v[rows[:A]],
                                     g[rows[:A]], S0[t.tree[leaf]], scale)
            dOm = np.where(keep[:, None, None], dO[rows], 0.0)[A:]
            sl = rows[A:]
            *_, lam = recurrent.la_bwd(q[sl], k[sl], v[sl], g[sl], SA, scale,
                                       dOm, dSf[t.leaf_index[leaf]])
            out[u] += lam
    return out


def _compare_grads(parent, seg_len, B, seed, H=2, dk=3, dv=4):
    t = SegTree(parent, seg_len)
    q, k, v, g, dO, dSf, S0 = _inputs(t.C, H, dk, dv, len(t.leaves),
                                      len(t.roots), seed)
    res = compact_fwd_bwd(parent, seg_len, B, q, k, v, g, 0.6, dO, dSf, S0)
    ref = recurrent.forest_bwd(parent, seg_len, q, k, v, g, 0.6, dO, dSf, S0)
    for name, r_ in zip(["dq", "dk", "dv", "dg", "dS0_tree"], ref):
        assert _rel(res[name], r_) <= 1e-11, name
    ds = _traj_dS0_seq(parent, seg_len, B, res["plan"], q, k, v, g, S0, 0.6,
                       dO, dSf)
    assert _rel(res["dS0_seq"], ds) <= 1e-11


@pytest.mark.parametrize("parent,seg_len,B", FORESTS)
def test_compact_gradients_figures(parent, seg_len, B):
    _compare_grads(parent, seg_len, B, seed=len(seg_len))


@pytest.mark.parametrize("B", [2, 3, 4])
def test_compact_gradients_random(B):
    r = np.random.default_rng(200 + B)
    for trial in range(8):
        n = int(r.integers(1, 8))
        parent, seg_len = _random_forest(r, n, B)
        _compare_grads(parent, seg_len, B, seed=trial)


def test_handoff_gradient_closed_form_fig1():
    """Figure 1 workload: sequence [E] starts at 256 from slot S_256 and
    replays [256, 277).  Its initial-state gradient is the adjoint entering
    its first own token (277) from E's subtree only, carried back over the
    replay by exp(sum of g over [256, 277))."""
    parent, seg_len, B = FORESTS[0]
    t = SegTree(parent, seg_len)
    q, k, v, g, dO, dSf, S0 = _inputs(t.C, 2, 3, 4, 3, 1, seed=42)
    res = compact_fwd_bwd(parent, seg_len, B, q, k, v, g, 0.6, dO, dSf, S0)
    plan = res["plan"]
    iE = [i for i in range(plan["n_seq"]) if plan["seq_first_seg"][i] == 4][0]
    rows_E = list(range(t.row0[4], t.row0[4] + t.len[4]))
    *_, adj = recurrent.la_bwd(q[rows_E], k[rows_E], v[rows_E], g[rows_E],
                               np.zeros((2, 3, 4)), 0.6, dO[rows_E],
                               dSf[t.leaf_index[4]])
    rep_rows = [t.row_of(4, p) for p in range(256, 277)]
    decay = np.exp(g[rep_rows].sum(axis=0))           # per head
    assert _rel(res["dS0_seq"][iE], decay[:, None, None] * adj) <= 1e-11
