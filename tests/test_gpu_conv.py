"""GPU parity of the causal depthwise convolution with true-ancestor context
(Sec. 4.2) against the fp64 oracle, through the C ABI: y, dx and dW on small
forests (every element), and on the 64k-token agentic microbatch with the
paper's width 4 over 6,144 channels (q, k, v of 16 heads of 128), the launch
configuration the benchmark times, compared on 48 sampled channels (channels
are independent).  Tolerances: max relative error per tensor, 1e-4 for
float32, 2e-2 for bf16."""
import ctypes as C

import numpy as np
import pytest
import torch

from oracle.conv import conv_bwd, conv_fwd
from tests.harness import TOL, max_rel, phys_index, record
from workloads.tensors import to_bf16_roundtrip
from workloads.trees import figure1_forest, forest_for_config

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def L():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2608_28158_amd import _lib
    return _lib.lib()


def _p(t):
    return C.c_void_p(t.data_ptr())


def context(L, plan, w):
    from paper_2608_28158_amd import _lib
    Cn, k = plan["C"], w - 1
    pred = np.zeros(Cn * k, np.int32)
    off = np.zeros(Cn + 1, np.int64)
    succ = np.zeros(max(Cn * k, 1), np.int32)
    _lib.check(L.harts_conv_context(plan.handle, w, pred.ctypes.data, off.ctypes.data,
                                    succ.ctypes.data), "harts_conv_context")
    return pred, off, succ


def run_conv(L, plan, x_phys, W, dy_phys, w, tdt):
    """x_phys, dy_phys: device tensors [C, Cch] in physical rows."""
    from paper_2608_28158_amd import _lib
    code = _lib.HARTS_BF16 if tdt == torch.bfloat16 else _lib.HARTS_F32
    Cn, Cch = x_phys.shape
    pred, off, succ = context(L, plan, w)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    pd, od, sd = dev(pred), dev(off), dev(succ)
    Wd = torch.from_numpy(np.ascontiguousarray(W, np.float32)).cuda()
    y = torch.empty_like(x_phys)
    dx = torch.empty_like(x_phys)
    dW = torch.empty((Cch, w), dtype=torch.float32, device="cuda")
    sz = C.c_size_t()
    _lib.check(L.harts_conv_workspace_size(Cn, Cch, w, C.byref(sz)), "harts_conv_workspace_size")
    ws = torch.empty(sz.value, dtype=torch.uint8, device="cuda")
    st = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    _lib.check(L.harts_conv_fwd(code, Cn, Cch, w, _p(x_phys), _p(Wd), _p(pd), _p(y), st),
               "harts_conv_fwd")
    _lib.check(L.harts_conv_bwd(code, Cn, Cch, w, _p(x_phys), _p(Wd), _p(pd), _p(od), _p(sd),
                                int(off[-1]), _p(dy_phys), _p(dx), _p(dW), _p(ws), ws.numel(), st),
               "harts_conv_bwd")
    torch.cuda.synchronize()
    return y, dx, dW


SMALL = [
    ("figure 1", figure1_forest().parent, figure1_forest().seg_len),
    ("one-token segments", [-1, 0, 1, 2, 3, 3, 5, -1, 7], [1, 1, 1, 1, 1, 4, 2, 70, 600]),
    ("star", [-1] + [0] * 30, [5] + [2] * 30),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("w", [2, 4, 8])
@pytest.mark.parametrize("label,parent,seg_len", SMALL, ids=[c[0] for c in SMALL])
def test_conv_matches_oracle_small(L, label, parent, seg_len, w, dtype):
    from paper_2608_28158_amd.plan import HartsPlan
    print(f"[gpu] conv {label} w={w} {dtype}", flush=True)
    plan = HartsPlan(parent, seg_len, 64)
    Cn, Cch = int(np.sum(seg_len)), 64
    r = np.random.default_rng(Cn + w)
    x = r.standard_normal((Cn, Cch)).astype(np.float32)
    dy = r.standard_normal((Cn, Cch)).astype(np.float32)
    W = r.standard_normal((Cch, w)).astype(np.float32)
    if dtype == "bf16":
        x, dy = to_bf16_roundtrip(x), to_bf16_roundtrip(dy)
    phys = phys_index(seg_len, plan["seg_row"])
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16

    def dev(a):
        out = np.empty_like(a)
        out[phys] = a
        return torch.from_numpy(out).to("cuda", tdt).contiguous()

    y, dx, dW = run_conv(L, plan, dev(x), W, dev(dy), w, tdt)
    y_ref = conv_fwd(parent, seg_len, x, W)
    dx_ref, dW_ref = conv_bwd(parent, seg_len, x, W, dy)
    errs = {"y": max_rel(y.float().cpu().numpy()[phys], y_ref),
            "dx": max_rel(dx.float().cpu().numpy()[phys], dx_ref),
            "dW": max_rel(dW.cpu().numpy(), dW_ref)}
    print(f"[gpu] conv {label} w={w} {dtype}: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()),
          flush=True)
    record(f"conv {label} w={w}", dtype, errs)
    assert all(e <= TOL[dtype] for e in errs.values()), errs


def test_conv_64k_workload_6144_channels_sampled(L):
    from paper_2608_28158_amd.plan import HartsPlan
    f, _, cfg = forest_for_config(2)
    plan = HartsPlan(f.parent, f.seg_len, 64, heads=cfg["H"])
    Cn, Cch, w = f.n_rows, 6144, 4
    print(f"[gpu] conv 64k workload C={Cn} channels={Cch} w={w} bf16", flush=True)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7)
    x = torch.randn((Cn, Cch), device="cuda", generator=gen).to(torch.bfloat16)
    dy = torch.randn((Cn, Cch), device="cuda", generator=gen).to(torch.bfloat16)
    r = np.random.default_rng(7)
    W = r.standard_normal((Cch, w)).astype(np.float32) * 0.5
    y, dx, dW = run_conv(L, plan, x, W, dy, w, torch.bfloat16)
    ch = np.sort(r.choice(Cch, 48, replace=False))
    phys = phys_index(f.seg_len, plan["seg_row"])
    chd = torch.from_numpy(ch).cuda().long()
    take = lambda t: t[:, chd].float().cpu().numpy()[phys]
    xs, dys = take(x), take(dy)
    y_ref = conv_fwd(f.parent, f.seg_len, xs, W[ch])
    dx_ref, dW_ref = conv_bwd(f.parent, f.seg_len, xs, W[ch], dys)
    errs = {"y": max_rel(take(y), y_ref), "dx": max_rel(take(dx), dx_ref),
            "dW": max_rel(dW.cpu().numpy()[ch], dW_ref)}
    print("[gpu] conv 64k workload: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()),
          flush=True)
    record("conv 68k x 6144, w=4 (48 ch)", "bf16", errs)
    assert all(e <= TOL["bf16"] for e in errs.values()), errs
