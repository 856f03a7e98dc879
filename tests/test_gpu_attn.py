"""Full attention through asymmetric Q/KV views (Sec. 4.2) on the GPU,
against the fp64 trajectory-wise oracle, through the C ABI: o, dq, dk, dv on
small forests (every element) and, on the 64k-token agentic microbatch at
16 heads of 128, o and dq of sampled query rows and dk, dv of sampled key
rows, each from its own oracle computation.  bf16 inputs; tolerance: max
relative error per tensor, 2e-2."""
import ctypes as C

import numpy as np
import pytest
import torch

from oracle.attn import forest_attention, view_attention
from oracle.forest import SegTree
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


def views_of(L, plan):
    from paper_2608_28158_amd import _lib
    lay = _lib.AttnLayout()
    _lib.check(L.harts_attn_layout(plan.handle, C.byref(lay)), "harts_attn_layout")
    views = np.zeros(4 * lay.n_views, np.int32)
    kv_rows = np.zeros(max(lay.n_kv, 1), np.int32)
    qt = np.zeros(2 * max(lay.n_qtiles, 1), np.int32)
    kt = np.zeros(2 * max(lay.n_kvtiles, 1), np.int32)
    off = np.zeros(plan["C"] + 1, np.int64)
    ent = np.zeros(max(lay.n_kv, 1), np.int32)
    _lib.check(L.harts_attn_views(plan.handle, views.ctypes.data, kv_rows.ctypes.data, qt.ctypes.data,
                                  kt.ctypes.data, off.ctypes.data, ent.ctypes.data), "harts_attn_views")
    return lay, views, kv_rows, qt, kt, off, ent


def run_attn(L, plan, q, k, v, dO, H, d, scale):
    """q, k, v, dO: device bf16 [C, H, d] in physical rows."""
    from paper_2608_28158_amd import _lib
    lay, views, kv_rows, qt, kt, off, ent = views_of(L, plan)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    vd, kr, qd, kd, od, ed = (dev(a) for a in (views, kv_rows, qt, kt, off, ent))
    Cn = q.shape[0]
    st = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    kvk = torch.empty((lay.n_kv, H, d), dtype=torch.bfloat16, device="cuda")
    kvv = torch.empty_like(kvk)
    _lib.check(L.harts_attn_gather(_p(k), _p(kr), lay.n_kv, Cn, H, d, _p(kvk), st), "gather k")
    _lib.check(L.harts_attn_gather(_p(v), _p(kr), lay.n_kv, Cn, H, d, _p(kvv), st), "gather v")
    o = torch.full_like(q, float("nan"))
    lse = torch.empty((Cn, H), dtype=torch.float32, device="cuda")
    _lib.check(L.harts_attn_fwd(_p(vd), _p(qd), lay.n_qtiles, H, d, C.c_float(scale), _p(q), _p(kvk),
                                _p(kvv), _p(o), _p(lse), st), "harts_attn_fwd")
    delta = torch.empty((Cn, H), dtype=torch.float32, device="cuda")
    dq = torch.full_like(q, float("nan"))
    dkv = torch.full((lay.n_kv, H, d), float("nan"), dtype=torch.float32, device="cuda")
    dvv = torch.full_like(dkv, float("nan"))
    _lib.check(L.harts_attn_bwd(_p(vd), _p(qd), lay.n_qtiles, _p(kd), lay.n_kvtiles, Cn, H, d,
                                C.c_float(scale), _p(q), _p(kvk), _p(kvv), _p(o), _p(lse), _p(dO),
                                _p(delta), _p(dq), _p(dkv), _p(dvv), st), "harts_attn_bwd")
    dk = torch.full_like(q, float("nan"))
    dv = torch.full_like(q, float("nan"))
    _lib.check(L.harts_attn_scatter(_p(dkv), _p(od), _p(ed), Cn, lay.n_kv, H, d, _p(dk), st), "scatter dk")
    _lib.check(L.harts_attn_scatter(_p(dvv), _p(od), _p(ed), Cn, lay.n_kv, H, d, _p(dv), st), "scatter dv")
    torch.cuda.synchronize()
    return dict(o=o, dq=dq, dk=dk, dv=dv, lse=lse)


SMALL = [
    ("figure 1", figure1_forest().parent, figure1_forest().seg_len),
    ("two trees, long ancestors", [-1, 0, 0, 1, 1, -1, 5, 5], [300, 17, 150, 64, 90, 40, 200, 1]),
    ("star", [-1] + [0] * 12, [130] + [5 * i + 1 for i in range(12)]),
]


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("label,parent,seg_len", SMALL, ids=[c[0] for c in SMALL])
def test_attn_matches_oracle_small(L, label, parent, seg_len, d):
    from paper_2608_28158_amd.plan import HartsPlan
    H = 3 if d == 64 else 2
    print(f"[gpu] attn {label} d={d} H={H}", flush=True)
    plan = HartsPlan(parent, seg_len, 64)
    Cn = int(np.sum(seg_len))
    r = np.random.default_rng(Cn + d)
    q, k, v, dO = (to_bf16_roundtrip(r.standard_normal((Cn, H, d)).astype(np.float32)) for _ in range(4))
    phys = phys_index(seg_len, plan["seg_row"])

    def dev(a):
        out = np.empty_like(a)
        out[phys] = a
        return torch.from_numpy(out).to("cuda", torch.bfloat16).contiguous()

    scale = d ** -0.5
    got = run_attn(L, plan, dev(q), dev(k), dev(v), dev(dO), H, d, scale)
    ref = forest_attention(parent, seg_len, q, k, v, scale, dO=dO)
    errs = {n: max_rel(got[n].float().cpu().numpy()[phys], ref[n]) for n in ("o", "dq", "dk", "dv")}
    print(f"[gpu] attn {label} d={d}: " + ", ".join(f"{k_}={v_:.2e}" for k_, v_ in errs.items()),
          flush=True)
    record(f"attn {label} d={d}", "bf16", errs)
    assert all(e <= TOL["bf16"] for e in errs.values()), errs


def prefix_rows(t, v, pos):
    """Canonical rows of trajectory positions 0 .. pos - 1 on the path to v."""
    out = []
    for u in t.path(v):
        n = min(t.len[u], pos - t.s[u])
        if n <= 0:
            break
        out.extend(range(t.row0[u], t.row0[u] + n))
    return out


def test_attn_64k_workload_sampled(L):
    """16 heads of 128 on the 64k-token agentic microbatch, the launch
    configuration the benchmark times.  Two heads are checked: o and dq of
    40 sampled query rows, each one view of a single query over its whole
    trajectory prefix; dk and dv of 24 key rows near the end of sampled leaf
    segments (only the later rows of the same leaf see them), one view of
    those queries."""
    from paper_2608_28158_amd.plan import HartsPlan
    f, _, cfg = forest_for_config(2)
    H, d = cfg["H"], cfg["d"]
    plan = HartsPlan(f.parent, f.seg_len, 64, heads=H)
    Cn = f.n_rows
    print(f"[gpu] attn 64k workload C={Cn} H={H} d={d}", flush=True)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(11)
    q, k, v, dO = (torch.randn((Cn, H, d), device="cuda", generator=gen).to(torch.bfloat16) for _ in range(4))
    scale = d ** -0.5
    got = run_attn(L, plan, q, k, v, dO, H, d, scale)
    r = np.random.default_rng(11)
    heads = torch.tensor(np.sort(r.choice(H, 2, replace=False))).cuda()
    phys = phys_index(f.seg_len, plan["seg_row"])
    host = lambda x: torch.from_numpy(x.index_select(1, heads).float().cpu().numpy()[phys]).double()
    Q, K, V, G = host(q), host(k), host(v), host(dO)
    out = {n: host(got[n]) for n in ("o", "dq", "dk", "dv")}
    t = SegTree(f.parent, f.seg_len)
    seg_of = np.repeat(np.arange(t.n), t.len)
    errs = {}
    ref, val = {n: [] for n in out}, {n: [] for n in out}
    for c in r.choice(Cn, 40, replace=False):
        u = int(seg_of[c])
        pos = t.s[u] + int(c) - t.row0[u]
        idx = prefix_rows(t, u, pos) + [int(c)]
        qo = Q[[int(c)]].clone().requires_grad_(True)
        o = view_attention(qo, K[idx], V[idx], len(idx) - 1, scale)
        (o * G[[int(c)]]).sum().backward()
        ref["o"].append(o.detach()[0])
        ref["dq"].append(qo.grad[0])
        val["o"].append(out["o"][c])
        val["dq"].append(out["dq"][c])
    leaves = [u for u in t.leaves if t.len[u] >= 2]
    for u in r.choice(leaves, 24, replace=False):
        u = int(u)
        c = t.row0[u] + t.len[u] - 1 - int(r.integers(0, min(64, t.len[u])))
        pos = t.s[u] + c - t.row0[u]
        own = list(range(c, t.row0[u] + t.len[u]))
        idx = prefix_rows(t, u, pos) + own
        kv = K[idx].clone().requires_grad_(True)
        vv = V[idx].clone().requires_grad_(True)
        o = view_attention(Q[own], kv, vv, len(idx) - len(own), scale)
        (o * G[own]).sum().backward()
        h = len(idx) - len(own)
        ref["dk"].append(kv.grad[h])
        ref["dv"].append(vv.grad[h])
        val["dk"].append(out["dk"][c])
        val["dv"].append(out["dv"][c])
    for n in out:
        errs[n] = max_rel(torch.stack(val[n]).numpy(), torch.stack(ref[n]).numpy())
    print("[gpu] attn 64k workload: " + ", ".join(f"{k_}={v_:.2e}" for k_, v_ in errs.items()), flush=True)
    record("attn 68k x 16 heads of 128 (sampled)", "bf16", errs)
    assert all(e <= TOL["bf16"] for e in errs.values()), errs
