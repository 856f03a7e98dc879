"""GPU parity of the compact-to-semantic log-probabilities (Sec. 3.5, eqs.
mapped-logp and mapped-logp-grad) against the fp64 oracle, through the C ABI.

Small forests are compared on every position and every gradient element;
the 64k-token agentic microbatch at the paper's vocabulary (157,184, bf16
logits, the launch configuration the benchmark times) is compared on
sampled positions and on whole gradient rows of sampled compact rows, the
rows serving the most positions among them.  Tolerances: max relative error
per tensor, 1e-4 for float32 logits, 2e-2 for bf16 logits.
"""
import ctypes as C

import numpy as np
import pytest
import torch

from oracle.logprob import log_softmax_row, logp_bwd, logp_fwd, semantic_positions
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


def semantic_map(L, plan, tok_phys):
    from paper_2608_28158_amd import _lib
    n_pos = plan["S"] - plan["n_leaves"]
    m = np.zeros(n_pos, np.int32)
    y = np.zeros(n_pos, np.int32)
    off = np.zeros(plan["C"] + 1, np.int64)
    pos = np.zeros(n_pos, np.int32)
    tok = np.ascontiguousarray(tok_phys, np.int32)
    _lib.check(L.harts_semantic_map(plan.handle, tok.ctypes.data, n_pos, m.ctypes.data,
                                    y.ctypes.data, off.ctypes.data, pos.ctypes.data),
               "harts_semantic_map")
    return m, y, off, pos


def run_logp(L, z, m, y, off, pos, g):
    """Forward and backward on the device; z is a [C, V] device tensor."""
    from paper_2608_28158_amd import _lib
    code = _lib.HARTS_BF16 if z.dtype == torch.bfloat16 else _lib.HARTS_F32
    Cn, V = z.shape
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    md, yd, offd, posd, gd = dev(m), dev(y), dev(off), dev(pos), dev(g.astype(np.float32))
    lse = torch.empty(Cn, dtype=torch.float32, device="cuda")
    logp = torch.empty(len(m), dtype=torch.float32, device="cuda")
    row_g = torch.empty(Cn, dtype=torch.float32, device="cuda")
    dz = torch.full_like(z, float("nan"))
    st = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    _lib.check(L.harts_logp_fwd(code, Cn, V, _p(z), len(m), _p(md), _p(yd), _p(lse), _p(logp), st),
               "harts_logp_fwd")
    _lib.check(L.harts_logp_bwd(code, Cn, V, _p(z), _p(lse), len(m), _p(offd), _p(posd), _p(yd),
                                _p(gd), _p(row_g), _p(dz), st), "harts_logp_bwd")
    torch.cuda.synchronize()
    return logp.cpu().numpy(), dz, row_g.cpu().numpy()


SMALL = [
    ("figure 1, V=1024", figure1_forest().parent, figure1_forest().seg_len, 1024),
    ("star of 40 leaves, V=16 (repeated targets at the fork)", [-1] + [0] * 40, [100] + [3] * 40, 16),
    ("two trees, V=8 (smallest vocabulary)", [-1, 0, 0, -1, 3, 3, 5], [65, 10, 80, 200, 1, 64, 3], 8),
]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("label,parent,seg_len,V", SMALL, ids=[c[0] for c in SMALL])
def test_logp_matches_oracle_small(L, label, parent, seg_len, V, dtype):
    from paper_2608_28158_amd.plan import HartsPlan
    print(f"[gpu] logp {label} {dtype}", flush=True)
    plan = HartsPlan(parent, seg_len, 64)
    Cn = int(np.sum(seg_len))
    r = np.random.default_rng(V + Cn)
    tokens = r.integers(0, V, size=Cn)
    z = (r.standard_normal((Cn, V)) * 2.0).astype(np.float32)
    if dtype == "bf16":
        z = to_bf16_roundtrip(z)
    phys = phys_index(seg_len, plan["seg_row"])
    tok_phys = np.empty(Cn, np.int64)
    tok_phys[phys] = tokens
    z_phys = np.empty_like(z)
    z_phys[phys] = z
    m, y, off, pos = semantic_map(L, plan, tok_phys)
    m_ref, y_ref = semantic_positions(parent, seg_len, tokens)
    assert np.array_equal(m, phys[m_ref]) and np.array_equal(y, y_ref)
    g = r.standard_normal(len(m)) * (r.random(len(m)) < 0.7)      # an action mask
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    logp, dz, row_g = run_logp(L, torch.from_numpy(z_phys).to("cuda", tdt), m, y, off, pos, g)
    lam_ref = logp_fwd(z, m_ref, y_ref)
    dz_ref = logp_bwd(z, m_ref, y_ref, g)
    dz_got = dz.float().cpu().numpy()[phys]
    G_ref = np.zeros(Cn)
    np.add.at(G_ref, m_ref, g)
    errs = {"logp": max_rel(logp, lam_ref), "dlogits": max_rel(dz_got, dz_ref),
            "row_g": max_rel(row_g[phys], G_ref)}
    print(f"[gpu] logp {label} {dtype}: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()),
          flush=True)
    record(f"logp {label[:28]}", dtype, errs)
    assert all(e <= TOL[dtype] for e in errs.values()), errs


def test_logp_full_vocabulary_64k_workload_sampled(L):
    """68,161 compact rows x 157,184 bf16 logits, every semantic position of
    the 64k-token agentic microbatch (389,279), in the benchmark's launch
    configuration; compared on 4,096 sampled positions and on the whole
    gradient rows of 12 rows: the 6 serving the most positions and 6 drawn
    at random."""
    from paper_2608_28158_amd.plan import HartsPlan
    V = 157184
    f, _, cfg = forest_for_config(2)
    plan = HartsPlan(f.parent, f.seg_len, 64, heads=cfg["H"])
    Cn = f.n_rows
    print(f"[gpu] logp full vocabulary C={Cn} V={V} bf16", flush=True)
    r = np.random.default_rng(42)
    tokens = r.integers(0, V, size=Cn)
    phys = phys_index(f.seg_len, plan["seg_row"])
    tok_phys = np.empty(Cn, np.int64)
    tok_phys[phys] = tokens
    m, y, off, pos = semantic_map(L, plan, tok_phys)
    g = r.standard_normal(len(m)) * (r.random(len(m)) < 0.7)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(42)
    z = torch.randn((Cn, V), device="cuda", dtype=torch.float32, generator=gen)
    z = z.mul_(2.0).to(torch.bfloat16)
    logp, dz, row_g = run_logp(L, z, m, y, off, pos, g)
    # sampled positions, each against one oracle log-softmax of its row
    sel = r.choice(len(m), 4096, replace=False)
    rows = np.unique(m[sel])
    zr = z[torch.from_numpy(rows).cuda().long()].float().cpu().numpy()
    local = {int(c): i for i, c in enumerate(rows)}
    lam_ref = logp_fwd(zr, np.array([local[int(c)] for c in m[sel]]), y[sel])
    errs = {"logp": max_rel(logp[sel], lam_ref)}
    # whole gradient rows: every position the row serves
    counts = np.diff(off)
    chk = np.concatenate([np.argsort(-counts, kind="stable")[:6], r.choice(Cn, 6, replace=False)])
    worst = 0.0
    for c in chk:
        ps = pos[off[c]:off[c + 1]]
        zc = z[int(c)].float().cpu().numpy()[None, :]
        ref = logp_bwd(zc, np.zeros(len(ps), np.int64), y[ps], g[ps])[0]
        if len(ps) == 0:
            assert np.all(dz[int(c)].float().cpu().numpy() == 0)
            continue
        worst = max(worst, max_rel(dz[int(c)].float().cpu().numpy(), ref))
        assert abs(row_g[c] - g[ps].sum()) <= 1e-5 * max(1.0, np.abs(g[ps]).sum())
    errs["dlogits_rows"] = worst
    print(f"[gpu] logp full vocabulary: max positions per row {counts.max()}, " +
          ", ".join(f"{k}={v:.2e}" for k, v in errs.items()), flush=True)
    record("logp 68k x 157,184 sampled", "bf16", errs)
    assert all(e <= TOL["bf16"] for e in errs.values()), errs
    assert np.all(np.isfinite(logp)) and np.all(logp <= 0)
    del z, dz
    torch.cuda.empty_cache()


def test_logp_invalid_indices_give_nan_not_a_fault(L):
    """A position whose row or target lies outside the logits reads nothing
    out of bounds: its log-probability is NaN, the others are unaffected."""
    from paper_2608_28158_amd import _lib
    Cn, V = 4, 16
    z = torch.randn((Cn, V), device="cuda")
    m = torch.tensor([0, 5, -1, 2, 3], dtype=torch.int32, device="cuda")
    y = torch.tensor([1, 2, 3, 99, 15], dtype=torch.int32, device="cuda")
    lse = torch.empty(Cn, device="cuda")
    logp = torch.empty(5, device="cuda")
    st = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    _lib.check(L.harts_logp_fwd(_lib.HARTS_F32, Cn, V, _p(z), 5, _p(m), _p(y), _p(lse), _p(logp),
                                st), "harts_logp_fwd")
    got = logp.cpu().numpy()
    assert np.isnan(got[1]) and np.isnan(got[2]) and np.isnan(got[3])
    zz = z.cpu().double().numpy()
    assert abs(got[0] - log_softmax_row(zz[0])[1]) < 1e-5
    assert abs(got[4] - log_softmax_row(zz[3])[15]) < 1e-5
    null = C.c_void_p()
    assert L.harts_logp_fwd(_lib.HARTS_BF16, Cn, 12, null, 0, null, null, null, null,
                            null) == _lib.HARTS_EUNSUPPORTED
