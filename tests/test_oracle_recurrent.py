"""Pins for the oracle's token-by-token recurrence (CPU only).

Nothing here re-types the recurrence: the forward is checked against the
closed (parallel) form of the scalar-decay linear attention and its special
cases, the backward against central finite differences and against an
identity that follows from rescaling q and k.
"""
import numpy as np
import pytest

from oracle import recurrent
from oracle.forest import SegTree


def _rand(n, H, dk, dv, seed, g_lo=-0.5, g_hi=-0.001):
    r = np.random.default_rng(seed)
    q = r.standard_normal((n, H, dk))
    k = r.standard_normal((n, H, dk))
    v = r.standard_normal((n, H, dv))
    g = r.uniform(g_lo, g_hi, size=(n, H))
    S0 = r.standard_normal((H, dk, dv)) * 0.3
    return q, k, v, g, S0


def parallel_form(q, k, v, g, S0, scale):
    """o_t = scale * [ sum_{s<=t} exp(sum_{s<r<=t} g_r) (q_t.k_s) v_s
                       + exp(sum_{r<=t} g_r) S0^T q_t ]  (unrolled recurrence)."""
    n, H, _ = q.shape
    G = np.cumsum(g, axis=0)                         # G_t = sum_{r<=t} g_r
    o = np.zeros((n, H, v.shape[2]))
    for h in range(H):
        for t in range(n):
            acc = np.exp(G[t, h]) * (S0[h].T @ q[t, h])
            for s in range(t + 1):
                acc = acc + np.exp(G[t, h] - G[s, h]) * (q[t, h] @ k[s, h]) * v[s, h]
            o[t, h] = scale * acc
    return o


def test_forward_matches_parallel_form():
    q, k, v, g, S0 = _rand(37, 3, 5, 4, seed=1)
    o, S = recurrent.la_fwd(q, k, v, g, S0, 0.7)
    ref = parallel_form(q, k, v, g, S0, 0.7)
    assert np.max(np.abs(o - ref)) <= 1e-12 * np.max(np.abs(ref))
    # final state in closed form
    G = np.cumsum(g, axis=0)
    Sref = np.exp(G[-1])[:, None, None] * S0
    for s in range(len(g)):
        Sref += (np.exp(G[-1] - G[s])[:, None, None]
                 * k[s][:, :, None] * v[s][:, None, :])
    assert np.max(np.abs(S - Sref)) <= 1e-12 * np.max(np.abs(Sref))


def test_zero_decay_is_causal_linear_attention():
    q, k, v, _, _ = _rand(20, 2, 4, 3, seed=2)
    g = np.zeros((20, 2))
    o, _ = recurrent.la_fwd(q, k, v, g, np.zeros((2, 4, 3)), 1.3)
    for h in range(2):
        scores = np.tril(q[:, h] @ k[:, h].T)         # (q_t . k_s) for s <= t
        ref = 1.3 * scores @ v[:, h]
        assert np.allclose(o[:, h], ref, rtol=0, atol=1e-12)


def test_constant_decay_is_retnet_form():
    q, k, v, _, _ = _rand(25, 2, 4, 3, seed=3)
    gam = np.array([-0.05, -0.3])
    g = np.tile(gam, (25, 1))
    o, _ = recurrent.la_fwd(q, k, v, g, np.zeros((2, 4, 3)), 0.5)
    t = np.arange(25)
    for h in range(2):
        Dm = np.where(t[:, None] >= t[None, :],
                      np.exp(gam[h] * (t[:, None] - t[None, :])), 0.0)
        ref = 0.5 * ((q[:, h] @ k[:, h].T) * Dm) @ v[:, h]
        assert np.allclose(o[:, h], ref, rtol=0, atol=1e-12)


def _loss(q, k, v, g, S0, scale, dO, dSf):
    o, S = recurrent.la_fwd(q, k, v, g, S0, scale)
    return np.sum(o * dO) + np.sum(S * dSf)


@pytest.mark.parametrize("seed", [4, 5])
def test_backward_matches_finite_differences(seed):
    q, k, v, g, S0 = _rand(9, 2, 3, 4, seed=seed)
    r = np.random.default_rng(seed + 100)
    dO = r.standard_normal(q.shape[:2] + (4,))
    dSf = r.standard_normal(S0.shape)
    scale = 0.8
    dq, dk, dv, dg, dS0 = recurrent.la_bwd(q, k, v, g, S0, scale, dO, dSf)
    args = dict(q=q, k=k, v=v, g=g, S0=S0)
    grads = dict(q=dq, k=dk, v=dv, g=dg, S0=dS0)
    h = 1e-6
    for name in args:
        x = args[name]
        for _ in range(6):
            idx = tuple(r.integers(0, s) for s in x.shape)
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            ap, am = dict(args), dict(args)
            ap[name], am[name] = xp, xm
            fd = (_loss(scale=scale, dO=dO, dSf=dSf, **ap)
                  - _loss(scale=scale, dO=dO, dSf=dSf, **am)) / (2 * h)
            assert abs(fd - grads[name][idx]) <= 1e-7 * max(1.0, abs(fd)), name


def test_dg_rescaling_identity():
    """Adding e to g_t equals scaling q_u by e^e and k_u by e^-e for u >= t
    and the final state by e^e, so
    dg_t = sum_{u>=t} (q_u.dq_u - k_u.dk_u) + <dS_final, S_final>."""
    q, k, v, g, S0 = _rand(15, 3, 4, 5, seed=6)
    r = np.random.default_rng(7)
    dO = r.standard_normal((15, 3, 5))
    dSf = r.standard_normal(S0.shape)
    dq, dk, _, dg, _ = recurrent.la_bwd(q, k, v, g, S0, 0.9, dO, dSf)
    _, S = recurrent.la_fwd(q, k, v, g, S0, 0.9)
    term = np.sum(q * dq, -1) - np.sum(k * dk, -1)
    rev = np.cumsum(term[::-1], axis=0)[::-1]
    ref = rev + np.einsum("hkv,hkv->h", dSf, S)[None, :]
    assert np.max(np.abs(dg - ref)) <= 1e-11 * np.max(np.abs(ref))


def test_forest_rows_shared_bitwise_and_single_path_is_plain_run():
    parent = [-1, 0, 0, 1, 1]
    seg_len = [7, 5, 6, 3, 4]
    C = sum(seg_len)
    q, k, v, g, _ = _rand(C, 2, 3, 3, seed=8)
    S0 = np.random.default_rng(9).standard_normal((1, 2, 3, 3))
    o, Sf = recurrent.forest_fwd(parent, seg_len, q, k, v, g, 0.6, S0)
    t = SegTree(parent, seg_len)
    for li, leaf in enumerate(t.leaves):
        rows = t.trajectory_rows(leaf)
        ot, S = recurrent.la_fwd(q[rows], k[rows], v[rows], g[rows], S0[0], 0.6)
        assert np.array_equal(o[rows], ot)       # bitwise on every row
        assert np.array_equal(Sf[li], S)


def test_forest_backward_matches_finite_differences():
    parent = [-1, 0, 0, 1, 1]
    seg_len = [4, 3, 2, 3, 2]
    C = sum(seg_len)
    q, k, v, g, _ = _rand(C, 1, 2, 3, seed=10)
    r = np.random.default_rng(11)
    S0 = r.standard_normal((1, 1, 2, 3))
    dO = r.standard_normal((C, 1, 3))
    dSf = r.standard_normal((3, 1, 2, 3))
    scale = 0.7
    grads = recurrent.forest_bwd(parent, seg_len, q, k, v, g, scale, dO, dSf, S0)

    def loss(q, k, v, g, S0):
        o, Sf = recurrent.forest_fwd(parent, seg_len, q, k, v, g, scale, S0)
        return np.sum(o * dO) + np.sum(Sf * dSf)

    args = [q, k, v, g, S0]
    h = 1e-6
    for i, x in enumerate(args):
        for _ in range(5):
            idx = tuple(r.integers(0, s) for s in x.shape)
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            ap, am = list(args), list(args)
            ap[i], am[i] = xp, xm
            fd = (loss(*ap) - loss(*am)) / (2 * h)
            assert abs(fd - grads[i][idx]) <= 1e-7 * max(1.0, abs(fd))
