"""Pins of the KDA oracle (Sec. 2.2, eq. chunk-state): the decay alone in
closed form, the delta rule as one gradient step of the squared retrieval
error (torch autograd), exact retrieval of the value just written, the
chunk form of eq. chunk-state against the token recurrence, gradients
against finite differences, and the forest's shared rows."""
import numpy as np
import pytest
import torch

from oracle.forest import SegTree
from oracle.kda import kda_chunkwise, kda_forest, kda_recurrent

T = lambda a: torch.as_tensor(np.asarray(a), dtype=torch.float64)


def inputs(n, H, dk, dv, seed, gmin=-0.5):
    r = np.random.default_rng(seed)
    q = r.standard_normal((n, H, dk))
    k = r.standard_normal((n, H, dk))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    v = r.standard_normal((n, H, dv))
    g = r.uniform(gmin, 0.0, (n, H, dk))
    beta = r.uniform(0.05, 1.0, (n, H))
    S0 = r.standard_normal((H, dk, dv))
    return [T(x) for x in (q, k, v, g, beta, S0)]


def test_without_writes_only_the_decay_acts():
    q, k, v, g, beta, S0 = inputs(9, 2, 5, 3, 0)
    o, S = kda_recurrent(q, k, v, g, beta * 0, 0.7, S0)
    G = torch.cumsum(g, 0)                                   # per-channel log-decay so far
    for t in range(9):
        St = torch.exp(G[t])[:, :, None] * S0
        assert torch.allclose(o[t], 0.7 * torch.einsum("hkv,hk->hv", St, q[t]), rtol=0, atol=1e-13)
    assert torch.allclose(S, torch.exp(G[-1])[:, :, None] * S0, rtol=0, atol=1e-13)


def test_delta_rule_is_one_gradient_step_on_the_retrieval_error():
    q, k, v, g, beta, S0 = inputs(1, 3, 6, 4, 1)
    _, S1 = kda_recurrent(q, k, v, g, beta, 1.0, S0)
    for h in range(3):
        Sp = (torch.exp(g[0, h])[:, None] * S0[h]).clone().requires_grad_(True)
        loss = 0.5 * ((Sp.T @ k[0, h] - v[0, h]) ** 2).sum()
        (grad,) = torch.autograd.grad(loss, Sp)
        assert torch.allclose(S1[h], Sp.detach() - beta[0, h] * grad, rtol=0, atol=1e-13)


def test_a_full_write_retrieves_the_value_just_written():
    q, k, v, g, beta, S0 = inputs(12, 2, 8, 5, 2)
    o, _ = kda_recurrent(k, k, v, g, torch.ones_like(beta), 1.0, S0)   # q = k, beta = 1, |k| = 1
    assert torch.allclose(o, v, rtol=0, atol=1e-12)


@pytest.mark.parametrize("B", [1, 2, 3, 16, 64])
def test_chunk_form_matches_the_recurrence(B):
    q, k, v, g, beta, S0 = inputs(70, 2, 8, 6, 3 + B)
    o, S = kda_recurrent(q, k, v, g, beta, 0.4, S0)
    oc, Sc = kda_chunkwise(q, k, v, g, beta, 0.4, S0, B)
    assert torch.allclose(oc, o, rtol=0, atol=1e-11)
    assert torch.allclose(Sc, S, rtol=0, atol=1e-11)


def test_gradients_finite_differences():
    parent, seg_len = [-1, 0, 0, 1], [3, 2, 4, 2]
    C = sum(seg_len)
    q, k, v, g, beta, _ = inputs(C, 2, 4, 3, 4)
    r = np.random.default_rng(5)
    S0 = T(r.standard_normal((1, 2, 4, 3)))
    dO = T(r.standard_normal((C, 2, 3)))
    dSf = T(r.standard_normal((2, 2, 4, 3)))
    args = [x.numpy() for x in (q, k, v, g, beta)] + [S0.numpy()]
    res = kda_forest(parent, seg_len, *args[:5], 0.6, args[5], dO=dO.numpy(), dS_final=dSf.numpy())

    def loss(xs):
        out = kda_forest(parent, seg_len, *xs[:5], 0.6, xs[5])
        return float(np.sum(out["o"] * dO.numpy()) + np.sum(out["S_final"] * dSf.numpy()))

    h = 1e-6
    for slot, name in enumerate(("dq", "dk", "dv", "dg", "dbeta", "dS0_tree")):
        for _ in range(5):
            idx = tuple(int(r.integers(0, s)) for s in args[slot].shape)
            xp = [a.copy() for a in args]
            xm = [a.copy() for a in args]
            xp[slot][idx] += h
            xm[slot][idx] -= h
            fd = (loss(xp) - loss(xm)) / (2 * h)
            assert abs(fd - res[name][idx]) < 1e-7 * max(1.0, abs(fd)), (name, idx)


def test_forest_rows_agree_across_trajectories_and_a_path_is_a_plain_run():
    parent, seg_len = [-1, 0, 0, 1, -1], [5, 3, 4, 2, 6]
    C = sum(seg_len)
    q, k, v, g, beta, _ = inputs(C, 2, 4, 3, 6)
    S0 = T(np.random.default_rng(7).standard_normal((2, 2, 4, 3)))
    out = kda_forest(parent, seg_len, q, k, v, g, beta, 0.5, S0)   # raises if shared rows disagree
    t = SegTree(parent, seg_len)
    for li, leaf in enumerate(t.leaves):
        rows = t.trajectory_rows(leaf)
        o, S = kda_recurrent(q[rows], k[rows], v[rows], g[rows], beta[rows], 0.5, S0[t.tree[leaf]])
        assert np.allclose(out["o"][rows], o.numpy(), rtol=0, atol=1e-13)
        assert np.allclose(out["S_final"][li], S.numpy(), rtol=0, atol=1e-13)
