"""The KDA host tables on the CPU (Sec. 2.2 with the handoffs of Sec. 3.4):
their structure against the plan, and their meaning: executing them in
float64 (per sequence, replay rows then own rows from the sequence's bank
entry, requested chunk-start states written to the bank, outputs of own rows
kept) with the oracle's token recurrence reproduces the trajectory-wise
oracle, on plans of one to four rounds."""
import ctypes as C

import numpy as np
import pytest
import torch

from oracle.kda import kda_forest, kda_recurrent
from oracle.plan_ref import plan_ref
from tests.harness import phys_index
from workloads.trees import figure1_forest

CASES = [
    ("figure 1", figure1_forest().parent, figure1_forest().seg_len),
    ("binary 3 levels", [-1, 0, 0, 1, 1, 2, 2], [150, 100, 90, 130, 70, 80, 60]),
    ("two trees K3 + K1", [-1, 0, 0, 1, 1, 2, 2, -1, 7], [150, 100, 90, 130, 70, 80, 60, 40, 300]),
    ("binary 4 levels", [-1, 0, 0, 1, 1, 2, 2, 3, 3, 4, 4, 5, 5, 6, 6],
     [120, 70, 66, 90, 100, 65, 130, 80, 75, 90, 68, 77, 101, 66, 140]),
]


def tables(plan):
    from paper_2608_28158_amd import _lib
    L = _lib.lib()
    sz = _lib.KdaSizes()
    _lib.check(L.harts_kda_layout(plan.handle, C.byref(sz)), "harts_kda_layout")
    t = dict(rows=np.zeros(sz.n_chunks * 64, np.int32), seq=np.zeros((sz.n_seq, 8), np.int32),
             req=np.zeros((max(sz.n_req, 1), 2), np.int32), grp=np.zeros((sz.n_groups, 4), np.int32),
             gseq=np.zeros(sz.n_seq, np.int32), slot=np.zeros(sz.n_chunks * 64, np.int32),
             mrow=np.zeros(max(sz.n_multi, 1), np.int32), moff=np.zeros(sz.n_multi + 1, np.int64))
    _lib.check(L.harts_kda_tables(plan.handle, *(t[k].ctypes.data for k in
                                                 ("rows", "seq", "req", "grp", "gseq", "slot", "mrow", "moff"))),
               "harts_kda_tables")
    return sz, t


@pytest.mark.parametrize("label,parent,seg_len", CASES, ids=[c[0] for c in CASES])
def test_tables_follow_the_plan(label, parent, seg_len):
    from paper_2608_28158_amd.plan import HartsPlan
    plan = HartsPlan(parent, seg_len, 64)
    sz, t = tables(plan)
    assert sz.n_rounds == plan["n_rounds"]
    c = 0
    for i in range(plan["n_seq"]):
        rnd, c0, nc, init, ro, nr, leaf, _ = (int(x) for x in t["seq"][i])
        assert rnd == plan["seq_round"][i] - 1 and c0 == c and init == plan["seq_init_bank"][i]
        assert leaf == plan["seq_final_leaf"][i]
        a, b = plan["seq_replay_off"][i], plan["seq_replay_off"][i + 1]
        own = plan["seq_row"][i] + np.arange(plan["seq_n_own"][i])
        want = np.concatenate([plan["replay_row"][a:b] * 2, own * 2 + 1])
        assert nc == -(-len(want) // 64)
        got = t["rows"][c0 * 64:(c0 + nc) * 64]
        assert np.array_equal(got[:len(want)], want) and np.all(got[len(want):] == -1)
        assert ro == plan["seq_req_off"][i] and nr == plan["seq_req_off"][i + 1] - ro
        for j in range(ro, ro + nr):
            assert t["req"][j, 0] == plan["req_chunk"][j] and t["req"][j, 1] == plan["req_bank"][j]
            assert 0 <= t["req"][j, 0] <= nc
        c += nc
    assert c == sz.n_chunks
    # the state passes' order (last column): each round's sequences once,
    # by descending chunk count, ties by id
    for rnd in range(sz.n_rounds):
        ids = np.nonzero(t["seq"][:, 0] == rnd)[0]
        order = t["seq"][ids, 7]
        assert sorted(order) == list(ids)
        assert order.tolist() == sorted(ids, key=lambda i: (-t["seq"][i, 2], i))
    # groups: every round's sequences once, by initial bank entry, in order
    seen = []
    for rnd, bank, first, n in t["grp"]:
        members = t["gseq"][first:first + n]
        assert np.all(plan["seq_init_bank"][members] == bank) and np.all(t["seq"][members, 0] == rnd)
        assert np.all(np.diff(members) > 0)
        seen += list(members)
    assert sorted(seen) == list(range(plan["n_seq"]))
    # gradient slots: every real packed row of a compact row with no other
    # packed row writes directly (-1); the compact rows with replay copies,
    # ascending, hold consecutive slots in ascending packed order
    real = np.nonzero(t["rows"] >= 0)[0]
    owner = t["rows"][real] // 2
    count = np.bincount(owner, minlength=plan["C"])
    assert np.all(count >= 1)
    assert np.all(np.bincount(owner[(t["rows"][real] & 1) == 1], minlength=plan["C"]) == 1)   # one own row each
    multi = np.nonzero(count > 1)[0]
    assert sz.n_multi == len(multi) == len(np.unique(plan["replay_row"]))
    assert np.array_equal(t["mrow"][:sz.n_multi], multi)
    assert t["moff"][0] == 0 and np.array_equal(np.diff(t["moff"]), count[multi]) and t["moff"][-1] == sz.n_slots
    assert np.all(t["slot"][real][count[owner] == 1] == -1)
    for m, r in enumerate(multi):
        p = real[owner == r]                              # ascending packed positions
        assert np.array_equal(t["slot"][p], np.arange(t["moff"][m], t["moff"][m + 1]))


def execute_tables(plan, t, q, k, v, g, beta, S0_tree, scale):
    """The tables run in float64 with the oracle's token recurrence."""
    bank = [None] * plan["n_bank"]
    for i in range(plan["n_trees"]):
        bank[i] = S0_tree[i]
    o = torch.zeros_like(v)
    finals = [None] * plan["n_leaves"]
    for rnd in range(plan["n_rounds"]):
        for i in np.nonzero(t["seq"][:, 0] == rnd)[0]:
            _, c0, nc, init, ro, nr, leaf, _ = (int(x) for x in t["seq"][i])
            reqs = [tuple(int(x) for x in t["req"][j]) for j in range(ro, ro + nr)]
            S = bank[init]
            for cc in range(nc + 1):
                for rc, b in reqs:
                    if rc == cc:
                        bank[b] = S.clone()
                if cc == nc:
                    break
                for e in t["rows"][(c0 + cc) * 64:(c0 + cc + 1) * 64]:
                    if e < 0:
                        continue
                    r = int(e) // 2
                    ot, S = kda_recurrent(q[[r]], k[[r]], v[[r]], g[[r]], beta[[r]], scale, S)
                    if e & 1:
                        o[r] = ot[0]
            finals[leaf] = S
    return o, torch.stack(finals)


@pytest.mark.parametrize("label,parent,seg_len", CASES, ids=[c[0] for c in CASES])
def test_executing_the_tables_reproduces_every_trajectory(label, parent, seg_len):
    from paper_2608_28158_amd.plan import HartsPlan
    plan = HartsPlan(parent, seg_len, 64)
    assert plan["n_rounds"] == plan_ref(parent, seg_len, 64)["K"]
    _, t = tables(plan)
    Cn, H, d = int(np.sum(seg_len)), 2, 3
    r = np.random.default_rng(len(parent))
    q, k, v = (r.standard_normal((Cn, H, d)) for _ in range(3))
    k /= np.linalg.norm(k, axis=-1, keepdims=True)
    g = r.uniform(-0.2, 0.0, (Cn, H, d))
    beta = r.uniform(0.1, 1.0, (Cn, H))
    S0 = r.standard_normal((plan["n_trees"], H, d, d))
    ref = kda_forest(parent, seg_len, q, k, v, g, beta, 0.5, S0)
    phys = phys_index(seg_len, plan["seg_row"])
    T = lambda a: torch.as_tensor(a, dtype=torch.float64)

    def to_phys(a):
        out = np.empty_like(a)
        out[phys] = a
        return T(out)

    o, Sf = execute_tables(plan, t, *(to_phys(a) for a in (q, k, v, g, beta)), T(S0), 0.5)
    assert np.allclose(o.numpy()[phys], ref["o"], rtol=0, atol=1e-12)
    assert np.allclose(Sf.numpy(), ref["S_final"], rtol=0, atol=1e-12)


def test_tables_reject_plans_of_another_chunk():
    from paper_2608_28158_amd import _lib
    from paper_2608_28158_amd.plan import HartsPlan
    plan = HartsPlan([-1, 0], [40, 20], 32)
    sz = _lib.KdaSizes()
    assert _lib.lib().harts_kda_layout(plan.handle, C.byref(sz)) == _lib.HARTS_EUNSUPPORTED


def test_kda_entry_points_reject_bad_arguments():
    """Argument checks of the device entry points, which return before any
    GPU call: unsupported dtype or width, missing tables, misaligned gradient
    outputs, bad reduction arguments; empty work returns HARTS_OK."""
    from paper_2608_28158_amd import _lib
    L = _lib.lib()
    buf = np.zeros(4096, np.float32)
    p = buf.ctypes.data + (16 - buf.ctypes.data % 16) % 16         # 16-byte aligned host address
    tabs = np.zeros(64, np.int32).ctypes.data

    def bwd(dtype=_lib.HARTS_BF16, d=128, slot=tabs, dq=p):
        ptrs = [p] * 10
        return L.harts_kda_bwd(tabs, tabs, tabs, slot, 0, 1, 0, 1, dtype, 2, d, C.c_float(1.0),
                               p, p, p, p, p, p, p, p, p, p, dq, p, p, p, p, *ptrs[:5], None)

    assert bwd(dtype=7) == _lib.HARTS_EUNSUPPORTED
    assert bwd(d=96) == _lib.HARTS_EUNSUPPORTED
    assert bwd(slot=None) == _lib.HARTS_EINVAL
    assert bwd(dq=p + 4) == _lib.HARTS_EINVAL
    assert b"16-byte aligned" in L.harts_last_error()
    red = lambda n, w, dt=_lib.HARTS_F32, src=p: L.harts_kda_reduce(src, tabs, tabs, n, w, dt, p, None)
    assert red(0, 8) == _lib.HARTS_OK                              # nothing to sum: no launch
    assert red(3, 0) == _lib.HARTS_EINVAL
    assert red(3, 8, dt=5) == _lib.HARTS_EINVAL
    assert red(3, 8, src=None) == _lib.HARTS_EINVAL
    assert L.harts_kda_bank_add(tabs, 0, 0, tabs, 16, p, p, None) == _lib.HARTS_OK
    assert L.harts_kda_bank_add(tabs, 0, -1, tabs, 16, p, p, None) == _lib.HARTS_EINVAL
