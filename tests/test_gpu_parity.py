"""GPU parity of the HIP path against the fp64 CPU oracle, through the C ABI.

Every case prints what it runs before touching the GPU.  Tolerances are the
max relative error per tensor (max |x - ref| / max |ref|): 1e-4 for float32
inputs, 2e-2 for bfloat16 inputs.  Large workloads compare sampled heads
(heads are independent in the recurrence) at the full shape on the GPU.
"""
import numpy as np
import pytest
import torch

from oracle.compact import compact_fwd, compact_fwd_bwd
from tests.harness import TOL, config_inputs, max_rel, phys_index, record
from workloads import draw_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2608_28158_amd import _lib
    _lib.lib()  # the HIP library must be built; no fallback exists


def _dev(a, phys, dtype):
    out = np.empty_like(a)
    out[phys] = a
    return torch.from_numpy(out).to("cuda").to(dtype).contiguous()


def _canon(t, phys):
    return t.float().cpu().numpy()[phys]


def run_gpu(parent, seg_len, x, H, d, dtype, scale, recompute=False, gather_init=False,
            min_blocks=0):
    from paper_2608_28158_amd.plan import HartsPlan
    from paper_2608_28158_amd.tree_la import TreeLARunner
    plan = HartsPlan(parent, seg_len, 64, heads=H, min_blocks=min_blocks)
    phys = phys_index(seg_len, plan["seg_row"])
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    q, k, v = (_dev(x[n], phys, tdt) for n in ("q", "k", "v"))
    g = _dev(x["g"], phys, torch.float32)
    dO = _dev(x["dO"], phys, tdt)
    dSf = torch.from_numpy(x["dS_final"]).cuda()
    S0 = torch.from_numpy(x["S0"]).cuda()
    runner = TreeLARunner(plan, H, d, tdt, "cuda", scale, gather_init=gather_init)
    fwd = runner.forward(q, k, v, g, S0, keep_states=not recompute)
    bwd = runner.backward(q, k, v, g, dO, dSf, fwd=fwd, S0_tree=S0, recompute=recompute)
    torch.cuda.synchronize()
    out = dict(o=_canon(fwd["o"], phys), S_final=fwd["S_final"].cpu().numpy(),
               dq=_canon(bwd["dq"], phys), dk=_canon(bwd["dk"], phys),
               dv=_canon(bwd["dv"], phys), dg=_canon(bwd["dg"], phys),
               dS0_tree=bwd["dS0_tree"].cpu().numpy(), dS0_seq=bwd["dS0_seq"].cpu().numpy())
    return out, plan


def compare(parent, seg_len, x, H, d, dtype, heads=None, recompute=False, label="", min_blocks=0):
    scale = d ** -0.5
    print(f"[gpu] {label} n_seg={len(parent)} C={int(np.sum(seg_len))} H={H} d={d} "
          f"{dtype} recompute={recompute}", flush=True)
    got, plan = run_gpu(parent, seg_len, x, H, d, dtype, scale, recompute, min_blocks=min_blocks)
    hs = list(range(H)) if heads is None else list(heads)
    sl = lambda a: a[:, hs]
    ref = compact_fwd_bwd(parent, seg_len, 64, sl(x["q"]), sl(x["k"]), sl(x["v"]), sl(x["g"]),
                          scale, sl(x["dO"]), sl(x["dS_final"]), sl(x["S0"]))
    tol = TOL[dtype]
    errs = {}
    for name in ("o", "S_final", "dq", "dk", "dv", "dg", "dS0_tree", "dS0_seq"):
        errs[name] = max_rel(sl(got[name]), ref[name])
    print(f"[gpu] {label} max-rel errors: " +
          ", ".join(f"{k}={v:.2e}" for k, v in errs.items()), flush=True)
    record(label, dtype, errs)
    bad = {k: v for k, v in errs.items() if not v <= tol}
    assert not bad, f"{label}: above {tol}: {bad}"
    # the plan the GPU ran is the oracle's plan
    assert plan["n_rounds"] == ref["plan"]["K"]
    assert np.array_equal(plan["seq_init_bank"], ref["plan"]["seq_init_bank"])
    return got


def test_config0_figure1_fp32():
    f, cfg, x = config_inputs(0, s0_scale=0.5)
    compare(f.parent, f.seg_len, x, cfg["H"], cfg["d"], "f32", label="config0")


def test_config0_recompute_matches_saved_bitwise():
    f, cfg, x = config_inputs(0, s0_scale=0.5)
    print("[gpu] config0 recompute vs saved", flush=True)
    a, _ = run_gpu(f.parent, f.seg_len, x, cfg["H"], cfg["d"], "f32", cfg["d"] ** -0.5, False)
    b, _ = run_gpu(f.parent, f.seg_len, x, cfg["H"], cfg["d"], "f32", cfg["d"] ** -0.5, True)
    c, _ = run_gpu(f.parent, f.seg_len, x, cfg["H"], cfg["d"], "f32", cfg["d"] ** -0.5, False)
    for name in a:
        assert np.array_equal(a[name], b[name]), name   # recompute-forward
        assert np.array_equal(a[name], c[name]), name   # run-to-run determinism


def test_gathered_and_indexed_initial_states_agree_bitwise():
    """Initial states read in place from the bank (S0 = NULL) and gathered
    into a dense buffer first (harts_state_gather) give the same bits, on
    the Figure 1 tree and on a multi-round config-1 forest."""
    for cfg_i, dtype in ((0, "f32"), (1, "bf16")):
        f, cfg, x = config_inputs(cfg_i, s0_scale=0.5)
        print(f"[gpu] config{cfg_i} gathered vs indexed initial states", flush=True)
        sc = cfg["d"] ** -0.5
        a, _ = run_gpu(f.parent, f.seg_len, x, cfg["H"], cfg["d"], dtype, sc, True, False)
        b, _ = run_gpu(f.parent, f.seg_len, x, cfg["H"], cfg["d"], dtype, sc, True, True)
        for name in a:
            assert np.array_equal(a[name], b[name]), name


def test_final_states_with_and_without_outputs():
    """Final states from a forward with outputs (the block kernel ends the
    sequences of one block) and from a state-only forward that requests them
    (summaries and chains for every sequence) agree with the oracle, on the
    Figure 1 tree and on a config-1 forest (sequences of one block and of
    several in both)."""
    from paper_2608_28158_amd.plan import HartsPlan
    from paper_2608_28158_amd.tree_la import TreeLARunner
    for cfg_i, dtype in ((0, "f32"), (1, "bf16")):
        f, cfg, x = config_inputs(cfg_i, s0_scale=0.5)
        H, d = cfg["H"], cfg["d"]
        print(f"[gpu] config{cfg_i} final states with and without outputs", flush=True)
        plan = HartsPlan(f.parent, f.seg_len, 64, heads=H)
        phys = phys_index(f.seg_len, plan["seg_row"])
        tdt = torch.float32 if dtype == "f32" else torch.bfloat16
        q, k, v = (_dev(x[n], phys, tdt) for n in ("q", "k", "v"))
        g = _dev(x["g"], phys, torch.float32)
        S0 = torch.from_numpy(x["S0"]).cuda()
        runner = TreeLARunner(plan, H, d, tdt, "cuda", d ** -0.5)
        a = runner.forward(q, k, v, g, S0, outputs=True)["S_final"]
        b = runner.forward(q, k, v, g, S0, outputs=False, final_states=True)["S_final"]
        torch.cuda.synchronize()
        f64 = lambda a: torch.from_numpy(np.asarray(a, np.float64))
        ref = compact_fwd(f.parent, f.seg_len, 64, f64(x["q"]), f64(x["k"]), f64(x["v"]), f64(x["g"]),
                          d ** -0.5, f64(x["S0"]))["S_final"].numpy()
        for got in (a, b):
            err = max_rel(got.cpu().numpy(), ref)
            print(f"[gpu] config{cfg_i} S_final max-rel {err:.2e}", flush=True)
            record(f"config{cfg_i} final states", dtype, {"S_final": err})
            assert err <= TOL[dtype]


def _random_forest(r, n, max_len, p_root=0.1):
    parent = [-1]
    for v in range(1, n):
        parent.append(-1 if r.random() < p_root else int(r.integers(0, v)))
    seg_len = [int(x) for x in r.integers(1, max_len, size=n)]
    return parent, seg_len


EDGE_FORESTS = [
    ("single segment", [-1], [300]),
    ("single short segment", [-1], [5]),
    ("fork on a chunk boundary", [-1, 0, 0], [128, 40, 70]),
    ("fork one before a boundary", [-1, 0, 0], [127, 40, 70]),
    ("fork one after a boundary", [-1, 0, 0], [129, 40, 70]),
    ("replay spans several ancestors", [-1, 0, 1, 2, 2, 1, 0], [70, 9, 3, 30, 44, 20, 15]),
    ("chain of tiny segments", [-1, 0, 1, 2, 3, 4, 4, 3], [1, 1, 1, 1, 1, 1, 90, 2]),
    ("star", [-1] + [0] * 9, [100] + [7 * i + 3 for i in range(9)]),
    ("two trees", [-1, 0, 0, -1, 3, 3], [65, 10, 80, 200, 1, 64]),
    ("exact multiples of the chunk", [-1, 0, 0, 1, 1], [64, 64, 128, 64, 192]),
]


@pytest.mark.parametrize("label,parent,seg_len", EDGE_FORESTS, ids=[e[0] for e in EDGE_FORESTS])
def test_edge_forests_fp32(label, parent, seg_len):
    r = np.random.default_rng(len(parent) * 1000 + sum(seg_len))
    n_leaves = len([v for v in range(len(parent)) if v not in parent])
    n_trees = parent.count(-1)
    x = draw_inputs(sum(seg_len), n_leaves, 2, 64, 64, r, "f32", n_trees=n_trees, s0_scale=0.3)
    compare(parent, seg_len, x, 2, 64, "f32", label=label)


def test_random_forests_fp32():
    r = np.random.default_rng(1234)
    for trial in range(6):
        parent, seg_len = _random_forest(r, int(r.integers(2, 14)), 160)
        n_leaves = len([v for v in range(len(parent)) if v not in parent])
        x = draw_inputs(sum(seg_len), n_leaves, 2, 64, 64, r, "f32",
                        n_trees=parent.count(-1), s0_scale=0.3)
        compare(parent, seg_len, x, 2, 64, "f32", label=f"random{trial}")


def test_random_forests_bf16_d64():
    r = np.random.default_rng(99)
    for trial in range(3):
        parent, seg_len = _random_forest(r, int(r.integers(2, 12)), 300)
        n_leaves = len([v for v in range(len(parent)) if v not in parent])
        x = draw_inputs(sum(seg_len), n_leaves, 3, 64, 64, r, "bf16",
                        n_trees=parent.count(-1), s0_scale=0.3)
        compare(parent, seg_len, x, 3, 64, "bf16", label=f"bf16-d64-{trial}")


@pytest.mark.parametrize("dtype,H", [("f32", 2), ("bf16", 3)])
def test_multiblock_sequences_d64(dtype, H):
    """Sequences of several blocks at d = 64 in both dtypes: block
    summaries, the local adjoints formed by the forward-order kernel, and
    both chains over blocks.  A 1,900-token root (30 chunks) with forks at
    unaligned offsets, cut into 8-chunk blocks (the planner's smallest, for
    a block target it cannot reach)."""
    parent = [-1, 0, 0, 1, 1]
    seg_len = [1900, 700, 333, 75, 610]
    r = np.random.default_rng(2024 + H)
    x = draw_inputs(sum(seg_len), 3, H, 64, 64, r, dtype, n_trees=1, s0_scale=0.3)
    from paper_2608_28158_amd.plan import HartsPlan
    plan = HartsPlan(parent, seg_len, 64, heads=H, min_blocks=100000)
    assert plan.rounds[0]["block_chunks"] == 8 and plan.rounds[0]["n_blk"] > plan.rounds[0]["n_seq"]
    compare(parent, seg_len, x, H, 64, dtype, label=f"multi-block {dtype}", min_blocks=100000)


def test_config1_spine_bf16_all_heads():
    f, cfg, x = config_inputs(1)
    compare(f.parent, f.seg_len, x, cfg["H"], cfg["d"], "bf16", label="config1 all heads")


@pytest.mark.parametrize("min_blocks,sizes", [("1", "64"), ("12", "16 and 24"), ("16", "12")])
def test_config1_block_sizes(min_blocks, sizes):
    """The same workload cut into blocks of other sizes (the block target of
    harts_plan_set_blocks) stays within tolerance."""
    f, cfg, x = config_inputs(1)
    compare(f.parent, f.seg_len, x, cfg["H"], cfg["d"], "bf16", heads=[0, 9],
            label=f"config1 blocks of {sizes} chunks", min_blocks=int(min_blocks))


def test_config2_agentic_bf16_sampled_heads():
    f, cfg, x = config_inputs(2)
    compare(f.parent, f.seg_len, x, cfg["H"], cfg["d"], "bf16", heads=[3], label="config2")


def test_config2_recompute_bf16_sampled_heads():
    f, cfg, x = config_inputs(2)
    compare(f.parent, f.seg_len, x, cfg["H"], cfg["d"], "bf16", heads=[11], recompute=True,
            label="config2-recompute")


def test_config3_large_bf16_sampled_head():
    f, cfg, x = config_inputs(3)
    compare(f.parent, f.seg_len, x, cfg["H"], cfg["d"], "bf16", heads=[17], label="config3")
