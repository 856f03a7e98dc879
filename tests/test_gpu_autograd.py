"""The PyTorch-facing entry ``tree_la`` through ``torch.autograd``, and the
in-library recompute-forward (``harts_la_bwd`` with saved = NULL).

``tree_la`` wraps the rounds of a plan in one ``torch.autograd.Function``;
with ``recompute=True`` the forward keeps no block states and each round's
backward re-runs its state pass from the plan ("Full-layer activation
recomputation", Sec. 3.4).  Gradients reached through
``torch.autograd.backward`` are compared with the fp64 oracle on a
three-call forest, and the recompute path is checked bitwise against the
saved-state path.
"""
import numpy as np
import pytest
import torch

from oracle.compact import compact_fwd_bwd
from tests.harness import TOL, max_rel, phys_index, record
from tests.test_gpu_parity import run_gpu
from workloads import draw_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2608_28158_amd import _lib
    _lib.lib()


PARENT = [-1, 0, 0, 1, 1, 2, 2]
SEG_LEN = [150, 100, 90, 130, 70, 80, 60]     # a three-call plan


@pytest.mark.parametrize("dtype,d,recompute", [("f32", 64, False), ("f32", 64, True),
                                               ("bf16", 128, False), ("bf16", 128, True)])
def test_tree_la_autograd_matches_oracle(dtype, d, recompute):
    from paper_2608_28158_amd.plan import HartsPlan
    from paper_2608_28158_amd.tree_la import tree_la
    H = 2
    label = f"tree_la autograd {dtype} d{d} recompute={recompute}"
    print(f"[gpu] {label}", flush=True)
    r = np.random.default_rng(7 + d + recompute)
    x = draw_inputs(sum(SEG_LEN), 4, H, d, d, r, dtype, n_trees=1, s0_scale=0.3)
    plan = HartsPlan(PARENT, SEG_LEN, 64, heads=H)
    assert plan["n_rounds"] == 3
    phys = phys_index(SEG_LEN, plan["seg_row"])
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16

    def leaf(a, dt):
        out = np.empty_like(a)
        out[phys] = a
        return torch.from_numpy(out).to("cuda", dt).requires_grad_(True)

    q, k, v = (leaf(x[n], tdt) for n in ("q", "k", "v"))
    g = leaf(x["g"], torch.float32)
    S0 = torch.from_numpy(x["S0"]).cuda().requires_grad_(True)
    dO = np.empty_like(x["dO"])
    dO[phys] = x["dO"]
    dO = torch.from_numpy(dO).to("cuda", tdt)
    dSf = torch.from_numpy(x["dS_final"]).cuda()
    o, S_final = tree_la(q, k, v, g, plan, S0_tree=S0, recompute=recompute)
    torch.autograd.backward([o, S_final], [dO, dSf])
    torch.cuda.synchronize()
    ref = compact_fwd_bwd(PARENT, SEG_LEN, 64, x["q"], x["k"], x["v"], x["g"], d ** -0.5,
                          x["dO"], x["dS_final"], x["S0"])
    canon = lambda t: t.detach().float().cpu().numpy()[phys]
    errs = {"o": max_rel(canon(o), ref["o"]),
            "S_final": max_rel(S_final.detach().cpu().numpy(), ref["S_final"]),
            "dq": max_rel(canon(q.grad), ref["dq"]), "dk": max_rel(canon(k.grad), ref["dk"]),
            "dv": max_rel(canon(v.grad), ref["dv"]), "dg": max_rel(canon(g.grad), ref["dg"]),
            "dS0_tree": max_rel(S0.grad.cpu().numpy(), ref["dS0_tree"])}
    print(f"[gpu] {label}: " + ", ".join(f"{n}={e:.2e}" for n, e in errs.items()), flush=True)
    record(label, dtype, errs)
    bad = {n: e for n, e in errs.items() if not e <= TOL[dtype]}
    assert not bad, f"{label}: above {TOL[dtype]}: {bad}"


@pytest.mark.parametrize("dtype,H", [("f32", 2), ("bf16", 3)])
def test_recompute_in_library_matches_saved_multiblock(dtype, H):
    """Sequences of several blocks at d = 64 (8-chunk blocks), on a
    three-call forest: the backward that recomputes every round's block
    states inside harts_la_bwd gives the same bits as the backward reading
    the states its forward saved, and reruns are identical."""
    parent = [-1, 0, 0, 1, 1, 2, 2]
    seg_len = [1300, 700, 900, 610, 575, 333, 820]
    r = np.random.default_rng(300 + H)
    x = draw_inputs(sum(seg_len), 4, H, 64, 64, r, dtype, n_trees=1, s0_scale=0.3)
    print(f"[gpu] recompute vs saved, multi-block {dtype}", flush=True)
    a, plan = run_gpu(parent, seg_len, x, H, 64, dtype, 0.125, recompute=False, min_blocks=100000)
    assert plan["n_rounds"] == 3
    assert any(rd["n_blk"] > rd["n_seq"] for rd in plan.rounds)
    b, _ = run_gpu(parent, seg_len, x, H, 64, dtype, 0.125, recompute=True, min_blocks=100000)
    c, _ = run_gpu(parent, seg_len, x, H, 64, dtype, 0.125, recompute=True, min_blocks=100000)
    for name in a:
        assert np.array_equal(a[name], b[name]), name
        assert np.array_equal(b[name], c[name]), name
