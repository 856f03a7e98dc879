"""Prefix-aware microbatch and data-parallel planning (Sec. 3.2), plain
Python.  TEST INFRASTRUCTURE ONLY (see the package docstring).

Input: N trajectories (token sequences), DP degree D and microbatch capacity
T in compact tokens.  A microbatch's work is the node count of the compact
trie of its members (eq. compact-trie-cost).  Candidate plans are ranked by
J = (total work, sum over slots of the heaviest microbatch of the slot,
heaviest replica's total) (eq. prefix-plan-objective).

Steps, in the paper's order:
  1. lexicographic order, adjacent LCPs, interval work W(a, b);
  2. the natural partition: split intervals above T at their lowest
     adjacent-LCP valley (ties: smaller larger side, then smaller
     difference);
  3. the K range (eqs. k-lower-bound, k-search-range);
  4. exact contiguous DP per K when N <= N0 (eq. contiguous-dp), else
     merge/split evolution of the natural partition at sampled K;
  5. trie-aware greedy (eq. greedy-insertion-delta): 4 orders x 2 policies,
     small-microbatch elimination, K aligned to D by singleton splits, one
     candidate kept (fewest microbatches, then least work);
  6. local refinement: boundary refinement of contiguous anchors, sparse
     repair (moves, then swaps, within H lexicographic positions);
  7. DP-replica assignment and slots, then the lexicographic choice by J.

Where the paper leaves a tie or a detail open, the choice is written next to
the step (and listed with the readings of the paper); the library follows
the same choices.
"""
from __future__ import annotations

N0 = 512        # exact search up to this many trajectories
Q_MAX = 32      # sampled K budget of the heuristic search
H_REF = 8       # refinement window in lexicographic positions
B_REF = 3       # anchors refined in heuristic mode


def lcp(a, b):
    n = min(len(a), len(b))
    i = 0
    while i < n and a[i] == b[i]:
        i += 1
    return i


def trie_nodes(seqs):
    """Compact work by definition: distinct non-empty prefixes."""
    return len({tuple(s[:k]) for s in seqs for k in range(1, len(s) + 1)})


class Lex:
    """Trajectories in lexicographic order (stable by index)."""

    def __init__(self, trajs):
        self.trajs = [list(t) for t in trajs]
        self.order = sorted(range(len(trajs)), key=lambda i: (self.trajs[i], i))
        self.rank = [0] * len(trajs)
        for r, i in enumerate(self.order):
            self.rank[i] = r
        self.len = [len(self.trajs[i]) for i in self.order]          # by rank
        self.L = [0] + [lcp(self.trajs[self.order[r - 1]], self.trajs[self.order[r]])
                        for r in range(1, len(trajs))]

    def lcp_ranks(self, r1, r2):
        """LCP of the trajectories at lexicographic ranks r1 != r2: the
        minimum adjacent LCP between them."""
        a, b = min(r1, r2), max(r1, r2)
        return min(self.L[a + 1:b + 1])

    def W(self, a, b):
        """Work of the contiguous ranks a..b (eq. compact-trie-cost)."""
        return sum(self.len[a:b + 1]) - sum(self.L[a + 1:b + 1])

    def work(self, ranks):
        rs = sorted(ranks)
        return sum(self.len[r] for r in rs) - sum(self.lcp_ranks(rs[i - 1], rs[i])
                                                  for i in range(1, len(rs)))


def natural_partition(lx, T):
    """Intervals (a, b) of ranks; an interval above T is split before the
    rank t with the lowest adjacent LCP; ties: smaller max(W left, W right),
    then smaller |W left - W right|, then smaller t."""
    out = []

    def rec(a, b):
        if lx.W(a, b) <= T or a == b:
            out.append((a, b))
            return
        best = None
        for t in range(a + 1, b + 1):
            wl, wr = lx.W(a, t - 1), lx.W(t, b)
            key = (lx.L[t], max(wl, wr), abs(wl - wr), t)
            if best is None or key < best:
                best = key
        t = best[3]
        rec(a, t - 1)
        rec(t, b)

    rec(0, len(lx.len) - 1)
    return out


def k_range(G, T, D, K0, N):
    kmin = D * max(1, -(-G // (T * D)))
    kmax = max(kmin, min(D * -(-K0 // D), D * (N // D)))
    return list(range(kmin, kmax + 1, D))


def exact_dp(lx, T, Ks):
    """eq. contiguous-dp: for every K in Ks the minimum-work partition of
    the ranks into K contiguous, capacity-feasible microbatches; ties: the
    smaller maximum microbatch work, then the smaller split point s."""
    N = len(lx.len)
    kmax = max(Ks)
    INF = None
    F = [[INF] * (N + 1) for _ in range(kmax + 1)]     # (total, max work)
    arg = [[-1] * (N + 1) for _ in range(kmax + 1)]
    F[0][0] = (0, 0)
    for k in range(1, kmax + 1):
        for e in range(1, N + 1):
            best, bs = None, -1
            for s in range(0, e):
                if F[k - 1][s] is None:
                    continue
                w = lx.W(s, e - 1)
                if w > T:
                    continue
                tot, mx = F[k - 1][s]
                cand = (tot + w, max(mx, w))
                if best is None or cand < best:
                    best, bs = cand, s
            F[k][e], arg[k][e] = best, bs
    out = {}
    for K in Ks:
        if F[K][N] is None:
            continue
        parts, e = [], N
        for k in range(K, 0, -1):
            s = arg[k][e]
            parts.append((s, e - 1))
            e = s
        out[K] = list(reversed(parts))
    return out


def sampled_ks(Ks):
    """At most Q_MAX values: every K when they fit; otherwise both ends,
    the Q_MAX/2 smallest and evenly spaced values over the rest."""
    if len(Ks) <= Q_MAX:
        return list(Ks)
    head = Ks[:Q_MAX // 2]
    rest = Ks[Q_MAX // 2:]
    m = Q_MAX - len(head)
    pick = {rest[round(i * (len(rest) - 1) / (m - 1))] for i in range(m)}
    return sorted(set(head) | pick)


def evolve(lx, T, parts, K):
    """Merge (K < K0) or split (K > K0) contiguous microbatches until there
    are K.  A merge of neighbours saves the LCP at their boundary (eq.
    cut-prefix-loss): the largest saving among capacity-feasible merges,
    ties by the smaller boundary rank.  A split costs the LCP at the cut:
    the smallest cost, ties by the smaller max side work, then the smaller
    cut rank.  None if no legal step remains."""
    parts = list(parts)
    while len(parts) > K:
        best = None
        for i in range(len(parts) - 1):
            (a, _), (_, b) = parts[i], parts[i + 1]
            if lx.W(a, b) > T:
                continue
            key = (-lx.L[parts[i + 1][0]], parts[i + 1][0])
            if best is None or key < best[0]:
                best = (key, i)
        if best is None:
            return None
        i = best[1]
        parts[i:i + 2] = [(parts[i][0], parts[i + 1][1])]
    while len(parts) < K:
        best = None
        for i, (a, b) in enumerate(parts):
            for t in range(a + 1, b + 1):
                key = (lx.L[t], max(lx.W(a, t - 1), lx.W(t, b)), t)
                if best is None or key < best[0]:
                    best = (key, i, t)
        if best is None:
            return None
        _, i, t = best
        a, b = parts[i]
        parts[i:i + 1] = [(a, t - 1), (t, b)]
    return parts


class Groups:
    """Microbatches as sorted rank lists with their work."""

    def __init__(self, lx):
        self.lx = lx
        self.members = []

    def work(self, g):
        return self.lx.work(self.members[g])

    def delta(self, g, r):
        """eq. greedy-insertion-delta: the work added by inserting rank r."""
        ms = self.members[g]
        lx = self.lx
        p = max((x for x in ms if x < r), default=None)
        q = min((x for x in ms if x > r), default=None)
        d = lx.len[r]
        if p is not None:
            d -= lx.lcp_ranks(p, r)
        if q is not None:
            d -= lx.lcp_ranks(r, q)
        if p is not None and q is not None:
            d += lx.lcp_ranks(p, q)
        return d


def greedy(lx, T, D, order, policy):
    g = Groups(lx)
    for r in order:
        best = None
        for i in range(len(g.members)):
            dc = g.delta(i, r)
            w = g.work(i)
            if w + dc > T:
                continue
            key = (-(w + dc), i) if policy == "best-fit" else (-(lx.len[r] - dc), i)
            if best is None or key < best[0]:
                best = (key, i)
        if best is None:
            g.members.append([r])
        else:
            g.members[best[1]] = sorted(g.members[best[1]] + [r])
    # eliminate small microbatches: in ascending work (ties by index), move
    # every member to the feasible other microbatch of least added work
    # (ties by index); keep the result only if all members fit
    changed = True
    while changed and len(g.members) > 1:
        changed = False
        for i in sorted(range(len(g.members)), key=lambda i: (g.work(i), i)):
            trial = [list(m) for m in g.members]
            ok = True
            for r in g.members[i]:
                best = None
                for j in range(len(trial)):
                    if j == i:
                        continue
                    tg = Groups(lx)
                    tg.members = trial
                    dc = tg.delta(j, r)
                    if tg.work(j) + dc > T:
                        continue
                    if best is None or (dc, j) < best:
                        best = (dc, j)
                if best is None:
                    ok = False
                    break
                trial[best[1]] = sorted(trial[best[1]] + [r])
            if ok:
                del trial[i]
                g.members = trial
                changed = True
                break
    # align K to D with singleton splits of the least added work (the shared
    # prefix of the trajectory split off); ties by group index, then rank
    while len(g.members) % D:
        best = None
        for i, ms in enumerate(g.members):
            if len(ms) < 2:
                continue
            for r in ms:
                rest = [x for x in ms if x != r]
                cost = lx.work(rest) + lx.len[r] - lx.work(ms)
                if best is None or (cost, i, r) < best:
                    best = (cost, i, r)
        if best is None:
            return None
        _, i, r = best
        g.members[i] = [x for x in g.members[i] if x != r]
        g.members.append([r])
    return g.members


def greedy_orders(lx):
    N = len(lx.len)
    asc = list(range(N))
    desc = asc[::-1]
    by_len = sorted(asc, key=lambda r: (-lx.len[r], r))

    def u(r):
        s = 0
        if r > 0:
            s = max(s, lx.L[r])
        if r + 1 < N:
            s = max(s, lx.L[r + 1])
        return lx.len[r] - s

    by_u = sorted(asc, key=lambda r: (-u(r), r))
    return [asc, desc, by_len, by_u]


def sparse_repair(lx, T, groups):
    groups = [sorted(m) for m in groups]
    where = {r: i for i, ms in enumerate(groups) for r in ms}
    for _ in range(4):
        best = None
        for r in range(len(lx.len)):
            a = where[r]
            if len(groups[a]) < 2:
                continue
            near = {where[x] for x in range(max(0, r - H_REF), min(len(lx.len), r + H_REF + 1))
                    if x != r and where[x] != a}
            for b in sorted(near):
                na = [x for x in groups[a] if x != r]
                nb = sorted(groups[b] + [r])
                wb = lx.work(nb)
                if wb > T:
                    continue
                gain = lx.work(groups[a]) + lx.work(groups[b]) - lx.work(na) - wb
                if gain > 0 and (best is None or (-gain, r, b) < best[0]):
                    best = ((-gain, r, b), ("move", r, b))
        if best is None:
            for r in range(len(lx.len)):
                for s in range(r + 1, min(len(lx.len), r + H_REF + 1)):
                    a, b = where[r], where[s]
                    if a == b:
                        continue
                    na = sorted([x for x in groups[a] if x != r] + [s])
                    nb = sorted([x for x in groups[b] if x != s] + [r])
                    wa, wb = lx.work(na), lx.work(nb)
                    if wa > T or wb > T:
                        continue
                    gain = lx.work(groups[a]) + lx.work(groups[b]) - wa - wb
                    if gain > 0 and (best is None or (-gain, r, s) < best[0]):
                        best = ((-gain, r, s), ("swap", r, s))
        if best is None:
            break
        op = best[1]
        if op[0] == "move":
            _, r, b = op
            a = where[r]
            groups[a] = [x for x in groups[a] if x != r]
            groups[b] = sorted(groups[b] + [r])
            where[r] = b
        else:
            _, r, s = op
            a, b = where[r], where[s]
            groups[a] = sorted([x for x in groups[a] if x != r] + [s])
            groups[b] = sorted([x for x in groups[b] if x != s] + [r])
            where[r], where[s] = b, a
    return groups


def boundary_refine(lx, T, parts):
    """Move each cut between neighbouring contiguous microbatches within
    H_REF ranks: the position of least (pair work, pair max work), ties by
    the smaller cut; at most two sweeps, stopping when a sweep moves none."""
    parts = list(parts)
    for _ in range(2):
        moved = False
        for i in range(len(parts) - 1):
            (a, c0), (_, b) = parts[i], parts[i + 1]
            cut = c0 + 1
            best = None
            for t in range(max(a + 1, cut - H_REF), min(b, cut + H_REF) + 1):
                wl, wr = lx.W(a, t - 1), lx.W(t, b)
                if wl > T or wr > T:
                    continue
                key = (wl + wr, max(wl, wr), t)
                if best is None or key < best:
                    best = key
            if best is not None and best[2] != cut:
                t = best[2]
                parts[i], parts[i + 1] = (a, t - 1), (t, b)
                moved = True
        if not moved:
            break
    return parts


def assign(lx, groups, D):
    """Slots of D microbatches in descending work (ties by group index);
    within a slot the heavier microbatch goes to the replica with less
    cumulative work (ties by replica index).  Returns (J, replica, slot)."""
    K = len(groups)
    w = [lx.work(m) for m in groups]
    order = sorted(range(K), key=lambda i: (-w[i], i))
    cum = [0] * D
    replica, slot = [0] * K, [0] * K
    slot_max = 0
    for j in range(K // D):
        blk = order[j * D:(j + 1) * D]
        reps = sorted(range(D), key=lambda d: (cum[d], d))
        for gi, d in zip(blk, reps):
            replica[gi], slot[gi] = d, j
            cum[d] += w[gi]
        slot_max += max(w[gi] for gi in blk)
    J = (sum(w), slot_max, max(cum))
    return J, replica, slot


def plan_microbatches(trajs, D, T, n0=N0):
    """The plan of Sec. 3.2 (exact contiguous search up to n0 trajectories,
    the paper's N0 = 512).  Returns dict(K, J, label, group[i] (microbatch
    of trajectory i), replica[g], slot[g], members[g])."""
    N = len(trajs)
    if D < 1 or T < 1 or N < D:
        raise ValueError("need D >= 1, T >= 1 and at least D trajectories")
    if any(len(t) > T or len(t) == 0 for t in trajs):
        raise ValueError("every trajectory must be non-empty and fit the capacity")
    lx = Lex(trajs)
    P0 = natural_partition(lx, T)
    G = lx.W(0, N - 1)
    Ks = k_range(G, T, D, len(P0), N)
    ranks = lambda parts: [list(range(a, b + 1)) for a, b in parts]
    cands = []                                    # (label, groups as rank lists)
    evolved = []                                  # (label, contiguous parts)
    if N <= n0:
        for K, parts in exact_dp(lx, T, Ks).items():
            cands.append((f"exact K={K}", ranks(parts)))
    else:
        for K in sampled_ks(Ks):
            parts = evolve(lx, T, P0, K)
            if parts is not None:
                evolved.append((f"evolved K={K}", parts))
                cands.append((f"evolved K={K}", ranks(parts)))
    greedy_best = None
    for order in greedy_orders(lx):
        for policy in ("best-fit", "max-shared"):
            gs = greedy(lx, T, D, order, policy)
            if gs is None:
                continue
            key = (len(gs), sum(lx.work(m) for m in gs))
            if greedy_best is None or key < greedy_best[0]:
                greedy_best = (key, gs)
    # refinement: exact mode refines only the greedy candidate; heuristic
    # mode also refines at most B_REF anchors among the evolved candidates:
    # the one at the greedy K, the lowest-work one, and the one whose K is
    # closest to the greedy K (each chosen among those not yet picked, ties
    # by generation order)
    if evolved:
        kg = greedy_best[0][0] if greedy_best is not None else None
        works = [sum(lx.W(a, b) for a, b in p) for _, p in evolved]
        picks = []
        if kg is not None:
            at_kg = [i for i, (_, p) in enumerate(evolved) if len(p) == kg]
            picks += at_kg[:1]
        rest = [i for i in range(len(evolved)) if i not in picks]
        if rest:
            picks.append(min(rest, key=lambda i: (works[i], i)))
        rest = [i for i in range(len(evolved)) if i not in picks]
        if kg is not None and rest:
            picks.append(min(rest, key=lambda i: (abs(len(evolved[i][1]) - kg), i)))
        for i in picks[:B_REF]:
            label, parts = evolved[i]
            parts = boundary_refine(lx, T, parts)
            cands.append((label + " refined", sparse_repair(lx, T, ranks(parts))))
    if greedy_best is not None:
        cands.append(("greedy refined", sparse_repair(lx, T, greedy_best[1])))
    best = None
    for label, groups in cands:
        if len(groups) % D or any(lx.work(m) > T for m in groups):
            continue
        J, rep, slot = assign(lx, groups, D)
        if best is None or J < best[0]:
            best = (J, label, groups, rep, slot)
    if best is None:
        raise ValueError("no feasible plan")
    J, label, groups, rep, slot = best
    group = [0] * N
    for gi, ms in enumerate(groups):
        for r in ms:
            group[lx.order[r]] = gi
    return dict(K=len(groups), J=J, label=label, group=group, replica=rep, slot=slot,
                members=[[lx.order[r] for r in ms] for ms in groups])
