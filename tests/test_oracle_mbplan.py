"""Pins of the prefix-aware microbatch planner oracle (Sec. 3.2) against
things other than itself: compact work counted as distinct prefixes (the
trie's nodes, by brute force), the cut identity eq. cut-prefix-loss, the
insertion delta eq. greedy-insertion-delta recounted on the trie, the exact
contiguous DP against enumeration of every contiguous partition, the K range
of eqs. k-lower-bound and k-search-range on hand-computed values, and the
feasibility guarantees of every returned plan."""
import itertools

import numpy as np
import pytest

from oracle.mbplan import (Groups, Lex, assign, exact_dp, k_range, natural_partition,
                           plan_microbatches, trie_nodes)


def random_trajs(r, n, vocab=4, max_base=6, max_tail=6):
    """Trajectories sharing prefixes: a few stems, each extended."""
    stems = [list(r.integers(0, vocab, size=int(r.integers(1, max_base)))) for _ in range(3)]
    out = []
    for _ in range(n):
        s = stems[int(r.integers(0, len(stems)))]
        cut = int(r.integers(0, len(s) + 1))
        out.append(s[:cut] + list(r.integers(0, vocab, size=int(r.integers(1, max_tail)))))
    return out


@pytest.mark.parametrize("seed", range(6))
def test_interval_work_cut_loss_and_subset_work(seed):
    r = np.random.default_rng(seed)
    trajs = random_trajs(r, 12)
    lx = Lex(trajs)
    seqs = [lx.trajs[i] for i in lx.order]
    N = len(trajs)
    for a in range(N):
        for b in range(a, N):
            assert lx.W(a, b) == trie_nodes(seqs[a:b + 1])           # eq. compact-trie-cost
            for t in range(a + 1, b + 1):                             # eq. cut-prefix-loss
                assert lx.W(a, t - 1) + lx.W(t, b) - lx.W(a, b) == lx.L[t]
    for _ in range(40):
        k = int(r.integers(1, N + 1))
        ranks = sorted(r.choice(N, k, replace=False).tolist())
        assert lx.work(ranks) == trie_nodes([seqs[x] for x in ranks])


@pytest.mark.parametrize("seed", range(4))
def test_insertion_delta_recounted_on_the_trie(seed):
    r = np.random.default_rng(10 + seed)
    trajs = random_trajs(r, 14)
    lx = Lex(trajs)
    seqs = [lx.trajs[i] for i in lx.order]
    g = Groups(lx)
    for _ in range(60):
        k = int(r.integers(1, 8))
        ms = sorted(r.choice(len(trajs), k, replace=False).tolist())
        x = int(r.choice([i for i in range(len(trajs)) if i not in ms]))
        g.members = [ms]
        before = trie_nodes([seqs[i] for i in ms])
        after = trie_nodes([seqs[i] for i in ms + [x]])
        assert g.delta(0, x) == after - before                     # eq. greedy-insertion-delta


def contiguous_partitions(N, K):
    for cuts in itertools.combinations(range(1, N), K - 1):
        bounds = (0,) + cuts + (N,)
        yield [(bounds[i], bounds[i + 1] - 1) for i in range(K)]


@pytest.mark.parametrize("seed", range(5))
def test_exact_dp_against_enumeration(seed):
    r = np.random.default_rng(20 + seed)
    trajs = random_trajs(r, 9)
    lx = Lex(trajs)
    T = int(r.integers(8, 20))
    N = len(trajs)
    Ks = list(range(1, N + 1))
    got = exact_dp(lx, T, Ks)
    for K in Ks:
        best = None
        for parts in contiguous_partitions(N, K):
            ws = [lx.W(a, b) for a, b in parts]
            if max(ws) > T:
                continue
            key = (sum(ws), max(ws))
            best = key if best is None or key < best else best
        if best is None:
            assert K not in got
        else:
            ws = [lx.W(a, b) for a, b in got[K]]
            assert (sum(ws), max(ws)) == best


def test_k_range_by_hand():
    # G = 100, T = 30, D = 2: K_min = 2 * max(1, ceil(100 / 60)) = 4;
    # K0 = 5, N = 9: K_max = max(4, min(2 * 3, 2 * 4)) = 6
    assert k_range(100, 30, 2, 5, 9) == [4, 6]
    # everything fits one microbatch: K_min = D
    assert k_range(10, 30, 4, 1, 8) == [4]
    # K_max capped by the trajectory count: min(2 * 5, 2 * 2) = 4 < K_min = 6
    assert k_range(150, 30, 2, 9, 5) == [6]


def test_natural_partition_splits_at_the_lowest_valley():
    # two families sharing nothing, each internally sharing a long prefix:
    # the split falls between the families
    a = [1] * 8
    b = [2] * 8
    trajs = [a + [3], a + [4], a + [5], b + [3], b + [4]]
    lx = Lex(trajs)
    parts = natural_partition(lx, 12)
    assert parts == [(0, 2), (3, 4)]
    assert lx.W(0, 2) == 11 and lx.W(3, 4) == 10


def check_plan(trajs, D, T, p):
    N = len(trajs)
    K = p["K"]
    assert K % D == 0 and K == len(p["members"])
    seen = sorted(i for ms in p["members"] for i in ms)
    assert seen == list(range(N))                                  # exact coverage
    for gi, ms in enumerate(p["members"]):
        assert ms and trie_nodes([trajs[i] for i in ms]) <= T      # capacity
        for i in ms:
            assert p["group"][i] == gi
    per = [0] * D
    for d in p["replica"]:
        per[d] += 1
    assert per == [K // D] * D                                     # K/D per replica
    w = [trie_nodes([trajs[i] for i in ms]) for ms in p["members"]]
    slots = {}
    cum = [0] * D
    for gi in range(K):
        slots.setdefault(p["slot"][gi], []).append(w[gi])
        cum[p["replica"][gi]] += w[gi]
    assert all(len(v) == D for v in slots.values())
    assert p["J"] == (sum(w), sum(max(v) for v in slots.values()), max(cum))


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("D", [1, 2, 4])
def test_plans_are_feasible_and_beat_the_natural_partition(seed, D):
    r = np.random.default_rng(100 + seed)
    trajs = random_trajs(r, int(r.integers(D, 16)), max_tail=8)
    T = max(len(t) for t in trajs) + int(r.integers(0, 20))
    p = plan_microbatches(trajs, D, T)
    check_plan(trajs, D, T, p)
    lx = Lex(trajs)
    P0 = natural_partition(lx, T)
    if D == 1:      # the natural partition is an exact-search candidate's competitor
        assert p["J"][0] <= sum(lx.W(a, b) for a, b in P0)


@pytest.mark.parametrize("seed", range(4))
def test_heuristic_mode_plans_are_feasible(seed):
    """The scalable path (evolution from the natural partition, anchors
    refined) with the exact-search threshold lowered to 6."""
    r = np.random.default_rng(200 + seed)
    trajs = random_trajs(r, 24, max_tail=8)
    T = max(len(t) for t in trajs) + 8
    for D in (1, 2):
        p = plan_microbatches(trajs, D, T, n0=6)
        check_plan(trajs, D, T, p)


def test_assignment_balances_slots_by_hand():
    # works 9, 7, 5, 3 with D = 2: slots {9, 7} and {5, 3}; replica 0 takes
    # 9 then 3 (less cumulative work after slot 0 is replica 1's 7 -> 5)
    trajs = [[0] * 9, [1] * 7, [2] * 5, [3] * 3]
    lx = Lex(trajs)
    groups = [[lx.rank[i]] for i in range(4)]
    J, rep, slot = assign(lx, groups, 2)
    assert slot == [0, 0, 1, 1]
    assert rep[0] == 0 and rep[1] == 1 and rep[2] == 1 and rep[3] == 0
    assert J == (24, 9 + 5, 12)


def test_rejects_infeasible_inputs():
    with pytest.raises(ValueError):
        plan_microbatches([[1, 2, 3]], 1, 2)          # a trajectory above capacity
    with pytest.raises(ValueError):
        plan_microbatches([[1], [2]], 4, 10)          # fewer trajectories than replicas
