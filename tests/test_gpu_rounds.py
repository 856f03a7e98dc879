"""GPU parity on plans of three or more rounds, through the C ABI.

Algorithm "minimum-call" (Sec. 3.3) needs K >= 3 sequential calls whenever a
side branch itself holds a subtree that needs two (eqs. tin, tpre); Appendix A
Case I is such a plan.  Those plans chain the differentiable handoffs of
Sec. 3.4: a sequence that starts from a requested boundary state requests one
itself, and its dS0 reaches the producer's producer two rounds back.  Every
case below asserts, from the library's own plan, that such a chained handoff
is present, then compares every tensor (o, S_final, dq, dk, dv, dg, dS0 of
the trees and of every sequence) with the fp64 oracle.

Forests: full binary trees of 3, 4 and 5 levels (K = levels when no fork
falls inside its parent's first chunk), nested forks that each cross a chunk
boundary, the same with sequences cut into several blocks, and seeded random
forests of which only the draws with K >= 3 are kept.
"""
import numpy as np
import pytest
import torch

from oracle.plan_ref import plan_ref
from tests.test_gpu_parity import compare
from workloads import draw_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2608_28158_amd import _lib
    _lib.lib()


def full_binary(levels, rng, lo=65, hi=200):
    parent, frontier = [-1], [0]
    for _ in range(levels - 1):
        nxt = []
        for u in frontier:
            for _ in range(2):
                parent.append(u)
                nxt.append(len(parent) - 1)
        frontier = nxt
    return parent, [int(x) for x in rng.integers(lo, hi, size=len(parent))]


def handoff_depth(plan):
    """(sequences that start from a slot and request slots themselves,
    longest chain of slot handoffs) of a library plan."""
    nt = plan["n_trees"]
    init = plan["seq_init_bank"]
    roff = plan["seq_req_off"]
    depth = {}
    chained = 0
    for i in range(plan["n_seq"]):       # producers precede consumers in id order
        b = int(init[i])
        depth[i] = 0 if b < nt else depth[int(plan["slot_seq"][b - nt])] + 1
        if b >= nt and roff[i + 1] > roff[i]:
            chained += 1
    return chained, max(depth.values())


def random_k3_forests(seed, count, max_len):
    """Seeded random forests, keeping only those whose plan has K >= 3."""
    r = np.random.default_rng(seed)
    out = []
    while len(out) < count:
        n = int(r.integers(5, 14))
        parent = [-1] + [int(r.integers(max(0, v - 3), v)) for v in range(1, n)]
        seg_len = [int(x) for x in r.integers(1, max_len, size=n)]
        if plan_ref(parent, seg_len, 64)["K"] >= 3:
            out.append((parent, seg_len))
    return out


def run_case(parent, seg_len, H, d, dtype, seed, label, min_rounds=3, min_blocks=0):
    from paper_2608_28158_amd.plan import HartsPlan
    plan = HartsPlan(parent, seg_len, 64, heads=H, min_blocks=min_blocks)
    chained, depth = handoff_depth(plan)
    print(f"[gpu] {label}: K={plan['n_rounds']} chained={chained} handoff depth={depth}",
          flush=True)
    assert plan["n_rounds"] >= min_rounds
    assert chained >= 1 and depth >= 2, "the case must chain handoffs"
    r = np.random.default_rng(seed)
    n_leaves = len([v for v in range(len(parent)) if v not in parent])
    x = draw_inputs(int(sum(seg_len)), n_leaves, H, d, d, r, dtype,
                    n_trees=list(parent).count(-1), s0_scale=0.3)
    compare(parent, seg_len, x, H, d, dtype, label=label, min_blocks=min_blocks)


BINARY = [(3, 10), (4, 11), (5, 12)]


@pytest.mark.parametrize("levels,seed", BINARY, ids=[f"{lv}-levels" for lv, _ in BINARY])
def test_full_binary_fp32_d64(levels, seed):
    parent, seg_len = full_binary(levels, np.random.default_rng(seed))
    run_case(parent, seg_len, 2, 64, "f32", seed, f"binary{levels} f32 d64", min_rounds=levels)


@pytest.mark.parametrize("levels,seed", BINARY[:2], ids=[f"{lv}-levels" for lv, _ in BINARY[:2]])
def test_full_binary_bf16_d128(levels, seed):
    parent, seg_len = full_binary(levels, np.random.default_rng(seed))
    run_case(parent, seg_len, 3, 128, "bf16", seed, f"binary{levels} bf16 d128",
             min_rounds=levels)


def test_binary_three_calls_fp32_and_bf16():
    """A 7-segment binary tree whose plan takes three calls (the shape of
    Appendix A Case I's call count)."""
    parent, seg_len = [-1, 0, 0, 1, 1, 2, 2], [150, 100, 90, 130, 70, 80, 60]
    assert plan_ref(parent, seg_len, 64)["K"] == 3
    run_case(parent, seg_len, 2, 64, "f32", 21, "binary7 f32 d64")
    run_case(parent, seg_len, 2, 128, "bf16", 22, "binary7 bf16 d128")


BOUNDARY_FORKS = [
    [129, 127, 63, 70, 1, 65, 200],   # forks one past, on, and on a boundary
    [127, 129, 65, 1, 64, 63, 3],     # one before, on, one past; 63 replay rows
    [128, 128, 129, 5, 7, 66, 64],    # on, on, one past
]


@pytest.mark.parametrize("seg_len", BOUNDARY_FORKS, ids=["past-on-on", "before-on-past", "on-on-past"])
def test_three_calls_with_forks_at_boundaries(seg_len):
    """Three-call binary trees whose forks sit on chunk boundaries or one
    row either side of one: slot-initialised sequences with 0, 1 or 63
    replay rows that request boundary states themselves."""
    parent = [-1, 0, 0, 1, 1, 2, 2]
    run_case(parent, seg_len, 2, 64, "f32", 31, "boundary forks f32 d64")
    run_case(parent, seg_len, 2, 128, "bf16", 32, "boundary forks bf16 d128")


@pytest.mark.parametrize("dtype,d", [("f32", 64), ("bf16", 128)])
def test_multiblock_chained_handoffs(dtype, d):
    """Long segments cut into 8-chunk blocks: slot-initialised sequences of
    several blocks, with requested boundaries inside them (the adjoint chain
    injects dbank into a sequence that itself started from a slot)."""
    parent, seg_len = full_binary(4, np.random.default_rng(41), lo=300, hi=900)
    from paper_2608_28158_amd.plan import HartsPlan
    plan = HartsPlan(parent, seg_len, 64, min_blocks=100000)
    assert any(r["n_blk"] > r["n_seq"] for r in plan.rounds[1:])
    run_case(parent, seg_len, 2, d, dtype, 42, f"multi-block binary4 {dtype} d{d}", min_rounds=4,
             min_blocks=100000)


def test_random_k3_forests_fp32():
    for i, (parent, seg_len) in enumerate(random_k3_forests(77, 4, 260)):
        run_case(parent, seg_len, 2, 64, "f32", 100 + i, f"random-K3 {i} f32 d64")


def test_random_k3_forests_bf16_d128():
    for i, (parent, seg_len) in enumerate(random_k3_forests(78, 2, 260)):
        run_case(parent, seg_len, 2, 128, "bf16", 200 + i, f"random-K3 {i} bf16 d128")


def test_two_trees_three_and_one_rounds():
    """A forest whose trees need different numbers of calls: the shallow
    tree's sequences all run in round 1."""
    p3, l3 = [-1, 0, 0, 1, 1, 2, 2], [150, 100, 90, 130, 70, 80, 60]
    parent = p3 + [-1, 7]
    seg_len = l3 + [40, 300]
    run_case(parent, seg_len, 2, 64, "f32", 51, "two trees K3+K1 f32 d64")
