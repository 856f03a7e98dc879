"""Pins for the reference planner ``oracle.plan_ref`` (CPU only).

* hand-derived plans of the paper's worked examples (tests/golden);
* brute-force minimality of the call count over every increasing-label tree
  with up to 7 segments (and forests), B in {2, 3, 4};
* the plan's rounds are the earliest legal rounds of its own choices;
* closed forms and invariants: eq. mandatory-replay and its independence of
  the direct-child choice, sum_v q_v len_v = S, every compact row is an own
  row of exactly one sequence, forest call count = max over trees, splitting
  a segment at a non-fork point keeps K and R.
"""
import itertools
import json
import os

import numpy as np
import pytest

from oracle.bruteforce import min_calls, rounds_for_choice
from oracle.forest import SegTree
from oracle.plan_ref import plan_ref


def _load(golden_dir, name):
    with open(os.path.join(golden_dir, name)) as f:
        return json.load(f)


def _chains(p):
    off = p["seq_chain_off"]
    return [[int(x) for x in p["chain_seg"][off[i]:off[i + 1]]]
            for i in range(p["n_seq"])]


def _requests(p):
    off = p["seq_req_off"]
    return [[[int(p["req_chunk"][j]), int(p["req_bank"][j])]
             for j in range(off[i], off[i + 1])] for i in range(p["n_seq"])]


def test_figure1_plan(golden_dir):
    gd = _load(golden_dir, "fig1_plan.json")
    p = plan_ref(gd["parent"], gd["seg_len"], gd["chunk"])
    for key in ["K", "C", "S", "R"]:
        assert p[key] == gd[key], key
    for key in ["seg_start", "seg_end", "seg_mult", "seg_tpre", "seg_tin",
                "seg_row", "seg_seq", "seq_round", "seq_anchor", "seq_n_replay",
                "seq_row", "seq_n_own", "seq_init_bank", "seq_final_leaf",
                "slot_seq", "slot_pos", "replay_row"]:
        assert p[key].tolist() == gd[key], key
    assert _chains(p) == gd["seq_chain"]
    assert _requests(p) == gd["seq_requests"]


def test_figure2_plan(golden_dir):
    gd = _load(golden_dir, "fig2_plan.json")
    p = plan_ref(gd["parent"], gd["seg_len"], gd["chunk"])
    assert p["K"] == gd["K"] and p["R"] == gd["R"]
    assert _chains(p) == gd["seq_chain"]
    for key in ["seq_round", "seq_anchor", "seq_n_replay", "seq_init_bank",
                "slot_pos"]:
        assert p[key].tolist() == gd[key], key
    assert _requests(p) == gd["seq_requests"]


def test_figure2b_boundary_cases(golden_dir):
    gd = _load(golden_dir, "fig2b_cases.json")
    for case in gd["cases"]:
        L = gd["leaf_len"]
        p = plan_ref([-1, 0, 0], [case["fork"], L, L], gd["chunk"])
        assert p["K"] == case["K"]
        side = [i for i in range(p["n_seq"]) if p["seq_first_seg"][i] == 2][0]
        assert p["seq_round"][side] == case["side_round"]
        assert p["seq_anchor"][side] == case["side_anchor"]
        assert p["seq_n_replay"][side] == case["side_replay"]


def test_figure3_plan(golden_dir):
    gd = _load(golden_dir, "fig3_plan.json")
    for form in gd["forms"]:
        p = plan_ref(form["parent"], form["seg_len"], gd["chunk"])
        assert p["K"] == form["K"] and p["R"] == form["R"]
        assert _chains(p) == form["seq_chain"]
        for key in ["seq_round", "seq_anchor", "seq_n_replay",
                    "seq_init_bank", "slot_pos"]:
            assert p[key].tolist() == form[key], key


def test_appendix_replay_arithmetic(golden_dir):
    """Only the printed arithmetic: per-call replay lists add up to the
    printed call totals and to R; the trees are not recoverable."""
    gd = _load(golden_dir, "appendix_cases.json")
    for case in gd["cases"]:
        assert len(case["per_call"]) == case["calls"]
        assert [sum(c) for c in case["per_call"]] == case["printed_call_totals"]
        assert sum(case["printed_call_totals"]) == case["R"]
        assert all(0 <= r < 64 for c in case["per_call"] for r in c)


def _increasing_trees(n):
    """All rooted trees on n labelled segments with parent[v] < v."""
    for choice in itertools.product(*[range(v) for v in range(1, n)]):
        yield [-1] + list(choice)


def _check_plan_against_model(parent, seg_len, B, p):
    t = SegTree(parent, seg_len)
    direct = [-1] * t.n
    for ch in _chains(p):
        for a, b in zip(ch[:-1], ch[1:]):
            direct[a] = b
    # every internal segment has a direct continuation and chains end at leaves
    for ch in _chains(p):
        assert not t.kids[ch[-1]]
    k_model, seqs = rounds_for_choice(t, B, direct)
    assert k_model == p["K"]
    model_round = {tuple(c): (r, a) for r, a, c in seqs}
    for i, ch in enumerate(_chains(p)):
        r, a = model_round[tuple(ch)]
        assert p["seq_round"][i] == r and p["seq_anchor"][i] == a
    # every compact row is an own row of exactly one sequence
    cover = np.zeros(t.C, np.int64)
    for ch in _chains(p):
        for v in ch:
            cover[t.row0[v]:t.row0[v] + t.len[v]] += 1
    assert np.all(cover == 1)
    # physical rows: a permutation of segments, contiguous per sequence
    rows = sorted((int(p["seg_row"][v]), v) for v in range(t.n))
    acc = 0
    for r0, v in rows:
        assert r0 == acc
        acc += t.len[v]
    # init states are produced earlier (slot producers run in earlier rounds)
    for i in range(p["n_seq"]):
        b = int(p["seq_init_bank"][i])
        if b >= p["n_trees"]:
            prod = int(p["slot_seq"][b - p["n_trees"]])
            assert p["seq_round"][prod] < p["seq_round"][i]


@pytest.mark.parametrize("B", [2, 3, 4])
def test_bruteforce_minimal_all_small_trees(B):
    r = np.random.default_rng(B)
    count = 0
    for n in range(1, 8):
        shapes = list(_increasing_trees(n))      # all (n-1)! shapes, 720 at n = 7
        for parent in shapes:
            for _ in range(4 if n < 7 else 1):
                seg_len = [int(x) for x in r.integers(1, 2 * B + 2, size=n)]
                p = plan_ref(parent, seg_len, B)
                assert p["K"] == min_calls(parent, seg_len, B), (parent, seg_len)
                _check_plan_against_model(parent, seg_len, B, p)
                count += 1
    assert count > 1000


@pytest.mark.parametrize("B", [2, 3, 4])
def test_bruteforce_minimal_forests(B):
    r = np.random.default_rng(50 + B)
    for _ in range(150):
        n = int(r.integers(2, 8))
        parent = [-1]
        for v in range(1, n):
            parent.append(-1 if r.random() < 0.25 else int(r.integers(0, v)))
        seg_len = [int(x) for x in r.integers(1, 2 * B + 2, size=n)]
        p = plan_ref(parent, seg_len, B)
        assert p["K"] == min_calls(parent, seg_len, B)
        assert p["K"] == max(p["K_tree"])
        _check_plan_against_model(parent, seg_len, B, p)


def test_mandatory_replay_closed_form_and_choice_independence():
    r = np.random.default_rng(7)
    for _ in range(200):
        B = int(r.integers(2, 9))
        n = int(r.integers(1, 7))
        parent = [-1] + [int(r.integers(0, v)) for v in range(1, n)]
        seg_len = [int(x) for x in r.integers(1, 3 * B, size=n)]
        t = SegTree(parent, seg_len)
        p = plan_ref(parent, seg_len, B)
        R_formula = sum((len(t.kids[v]) - 1) * (t.e[v] % B)
                        for v in range(n) if t.kids[v])
        assert p["R"] == R_formula
        assert int(np.sum(p["seq_n_replay"])) == R_formula
        # any direct-continuation choice replays the same total
        internal = [v for v in range(n) if t.kids[v]]
        for pick in itertools.product(*[t.kids[v] for v in internal]):
            direct = [-1] * n
            for v, c in zip(internal, pick):
                direct[v] = c
            _, seqs = rounds_for_choice(t, B, direct)
            total = sum(t.s[c[0]] - a for _, a, c in seqs)
            assert total == R_formula


def test_multiplicity_sums_to_semantic_positions():
    r = np.random.default_rng(8)
    for _ in range(100):
        n = int(r.integers(1, 12))
        parent = [-1] + [int(r.integers(0, v)) for v in range(1, n)]
        seg_len = [int(x) for x in r.integers(1, 100, size=n)]
        p = plan_ref(parent, seg_len, 16)
        assert int(np.sum(p["seg_mult"] * np.asarray(seg_len))) == p["S"]
    # Figure 1 caption: q_B = 2
    p = plan_ref([-1, 0, 0, 1, 1], [200, 77, 90, 64, 50], 64)
    assert p["seg_mult"][1] == 2


def test_split_at_non_fork_point_keeps_K_and_R():
    r = np.random.default_rng(9)
    for _ in range(200):
        B = int(r.integers(2, 9))
        n = int(r.integers(1, 8))
        parent = [-1] + [int(r.integers(0, v)) for v in range(1, n)]
        seg_len = [int(x) for x in r.integers(2, 4 * B, size=n)]
        v = int(r.integers(0, n))
        cut = int(r.integers(1, seg_len[v]))
        # new segment n takes the tail of v and v's children
        parent2 = [(n if (p == v) else p) for p in parent] + [v]
        seg_len2 = list(seg_len) + [seg_len[v] - cut]
        seg_len2[v] = cut
        p1 = plan_ref(parent, seg_len, B)
        p2 = plan_ref(parent2, seg_len2, B)
        assert (p1["K"], p1["R"]) == (p2["K"], p2["R"])


def test_invalid_inputs_raise():
    with pytest.raises(ValueError):
        plan_ref([-1, 0], [5, 0], 4)          # zero-length segment
    with pytest.raises(ValueError):
        plan_ref([1, 0], [5, 5], 4)           # cycle, no root
    with pytest.raises(ValueError):
        plan_ref([-1, 0, 2], [5, 5, 5], 4)    # self-parent
    with pytest.raises(ValueError):
        plan_ref([-1, 5], [5, 5], 4)          # parent out of range
    with pytest.raises(ValueError):
        plan_ref([-1], [5], 0)                # chunk size
