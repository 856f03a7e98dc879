"""harts_la_fwd_noalloc against harts_la_fwd, through the C ABI.

The allocation-free forward keeps its scratch in the library's fixed device
array instead of a caller workspace; on the same inputs it must give the same
bits as harts_la_fwd with a workspace and no saved buffer: outputs, final
states and every requested boundary state of every round.  Two plans run
back to back, the second smaller than the first, so the second reads the
array as the first left it.
"""
import ctypes as C

import numpy as np
import pytest
import torch

from workloads import draw_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2608_28158_amd import _lib
    return _lib.lib()


def _p(t):
    return C.c_void_p(t.data_ptr() if t is not None else 0)


def forward_all_rounds(L, plan, blob, code, H, d, x, noalloc):
    from paper_2608_28158_amd import _lib
    dt = torch.float32 if code == _lib.HARTS_F32 else torch.bfloat16
    # rows are taken in physical order as drawn: both paths read the same
    # tensors, so no canonical reordering is needed for a bitwise comparison
    q, k, v = (torch.from_numpy(x[n]).to("cuda", dt).contiguous() for n in ("q", "k", "v"))
    g = torch.from_numpy(x["g"]).cuda().contiguous()
    o = torch.full_like(q, float("nan"))
    S_final = torch.full((plan["n_leaves"], H, d, d), float("nan"), device="cuda")
    bank = torch.full((plan["n_bank"], H, d, d), float("nan"), device="cuda")
    bank[: plan["n_trees"]] = torch.from_numpy(x["S0"]).cuda()
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    sz = C.c_size_t()
    for r in range(plan["n_rounds"]):
        if noalloc:
            rc = L.harts_la_fwd_noalloc(plan.handle, r, _p(blob), code, H, d, d, C.c_float(d ** -0.5),
                                        _p(q), _p(k), _p(v), _p(g), _p(None), _p(o), _p(S_final),
                                        _p(bank), stream)
        else:
            _lib.check(L.harts_la_workspace_size(plan.handle, r, 0, code, H, d, d, 0, C.byref(sz)),
                       "harts_la_workspace_size")
            ws = torch.empty(max(sz.value, 16), dtype=torch.uint8, device="cuda")
            rc = L.harts_la_fwd(plan.handle, r, _p(blob), code, H, d, d, C.c_float(d ** -0.5),
                                _p(q), _p(k), _p(v), _p(g), _p(None), _p(o), _p(S_final), _p(bank),
                                _p(None), _p(ws), C.c_size_t(ws.numel()), stream)
        _lib.check(rc, "forward")
    torch.cuda.synchronize()
    return {n: t.float().cpu().numpy() for n, t in (("o", o), ("S_final", S_final), ("bank", bank))}


CASES = [
    # (label, parent, seg_len, H, d, dtype): the second of each pair is smaller
    ("three-call tree, bf16 d128", [-1, 0, 0, 1, 1, 2, 2], [1300, 700, 900, 610, 575, 333, 820],
     4, 128, "bf16"),
    ("Figure-1 tree, bf16 d128", [-1, 0, 0, 1, 1], [200, 77, 90, 64, 50], 2, 128, "bf16"),
    ("three-call tree, f32 d64", [-1, 0, 0, 1, 1, 2, 2], [900, 400, 700, 310, 275, 133, 620],
     3, 64, "f32"),
    ("two trees, f32 d64", [-1, 0, 0, -1, 3], [65, 10, 80, 130, 9], 2, 64, "f32"),
]


def test_noalloc_forward_matches_workspace_forward(L):
    from paper_2608_28158_amd import _lib
    from paper_2608_28158_amd.plan import HartsPlan
    for i, (label, parent, seg_len, H, d, dtype) in enumerate(CASES):
        print(f"[gpu] noalloc call {i}: {label}", flush=True)
        # short blocks: several blocks per sequence, so the scratch holds
        # summaries and chained block-end states
        plan = HartsPlan(parent, seg_len, 64, heads=H, min_blocks=100000)
        blob = plan.blob("cuda")
        code = _lib.HARTS_F32 if dtype == "f32" else _lib.HARTS_BF16
        n_leaves = plan["n_leaves"]
        x = draw_inputs(plan["C"], n_leaves, H, d, d, np.random.default_rng(500 + i), dtype,
                        n_trees=plan["n_trees"], s0_scale=0.3)
        a = forward_all_rounds(L, plan, blob, code, H, d, x, noalloc=False)
        b = forward_all_rounds(L, plan, blob, code, H, d, x, noalloc=True)
        for name in a:
            assert np.isfinite(a[name]).all(), name
            assert np.array_equal(a[name], b[name]), f"{label}: {name} differs"
        plan.close()


def test_noalloc_rejects_rounds_beyond_its_scratch(L):
    """A round whose scratch exceeds the fixed array is refused with
    HARTS_ENOMEM before anything is enqueued."""
    from paper_2608_28158_amd import _lib
    from paper_2608_28158_amd.plan import HartsPlan
    plan = HartsPlan([-1], [64 * 64 * 40], 64)      # 40 blocks of 64 chunks
    null = C.c_void_p()
    rc = L.harts_la_fwd_noalloc(plan.handle, 0, null, _lib.HARTS_BF16, 64, 128, 128,
                                C.c_float(0.1), null, null, null, null, null, null, null, null,
                                null)
    assert rc == _lib.HARTS_ENOMEM
    assert "scratch" in _lib.last_error()
    plan.close()
