#!/usr/bin/env python
"""Benchmark of tree-packed chunkwise linear attention on one MI355X.

One step = one pass of the whole hot path over one synthetic microbatch with
inputs resident in HBM: for every execution round the state gather, the
packed forward (outputs, requested and final states); then, with full-layer
activation recomputation as in every performance run of the paper, the
backward re-runs the state pass of every round from the fixed plan and walks
the rounds in reverse (gradients, handoff scatter-add), ending with the
replay-gradient reduction.  The host planner runs once per microbatch and is
timed separately (the paper's F/B/Grad vs Core split).

Workload (default): 8 agentic rollout trees, ~64k compact tokens, 16 heads,
d = 128, chunk 64, bf16 q/k/v, float32 decay and states.

Prints one JSON line.  ``--gpus`` above 1 is not supported: this build runs
one GPU.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0      # dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3

WORKLOADS = {
    2: "8 agentic rollout trees, ~64k compact tokens, H=16, d=128, chunk 64, bf16; "
       "forward + backward with full-layer recompute",
    3: "32 agentic rollout trees (depth <= 6), ~128k compact tokens, H=32, d=128, chunk 64, "
       "bf16; forward + backward with full-layer recompute",
    1: "4 spine trees, ~16k compact tokens, H=16, d=128, chunk 64, bf16; "
       "forward + backward with full-layer recompute",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# short workload names used by the committed profile summaries
WORKLOAD_KEY = {1: "spine16k", 2: "agentic64k", 3: "agentic128k"}


def la_source_sha(kernel=None):
    if kernel and kernel.startswith("k_logp"):
        names = ("logp.hip",)
    elif kernel and kernel.startswith("k_conv"):
        names = ("conv.hip",)
    elif kernel and kernel.startswith("k_attn"):
        names = ("attn.hip", "la_common.hpp")
    else:
        names = ("la.hip", "la_common.hpp")
    h = hashlib.sha256()
    for name in names:
        with open(os.path.join(ROOT, "paper_2608_28158_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def to_device(x, phys, dt):
    import torch
    out = np.empty_like(x)
    out[phys] = x
    return torch.from_numpy(out).to("cuda").to(dt).contiguous()


def phys_index(seg_len, seg_row):
    seg_len = np.asarray(seg_len, np.int64)
    row0 = np.concatenate([[0], np.cumsum(seg_len)[:-1]])
    phys = np.empty(int(seg_len.sum()), np.int64)
    for v in range(len(seg_len)):
        phys[row0[v]:row0[v] + seg_len[v]] = seg_row[v] + np.arange(seg_len[v])
    return phys


def seq_blocks(plan, i, B, block_chunks):
    """Blocks of sequence i as the planner cuts them (at every requested
    boundary and after at most block_chunks chunks), as (packed rows, own
    rows) per block."""
    n_rep = int(plan["seq_n_replay"][i])
    tok = n_rep + int(plan["seq_n_own"][i])
    nc = (tok + B - 1) // B
    reqs = [int(c) for c in plan["req_chunk"][plan["seq_req_off"][i]:plan["seq_req_off"][i + 1]]]
    out, c0, j = [], 0, 0
    while c0 < nc:
        c1 = min(nc, c0 + block_chunks)
        while j < len(reqs) and reqs[j] <= c0:
            j += 1
        if j < len(reqs) and reqs[j] <= c1:
            c1 = reqs[j]
        p0, p1 = c0 * B, min(c1 * B, tok)
        out.append((p1 - p0, max(0, p1 - max(p0, n_rep))))
        c0 = c1
    return out


def alg_bytes(plan, H, d, el):
    """Algorithmic bytes of one step: what the method must move, the
    per-token figures of the measurement plan (q, k, v, dO read once; o, dq,
    dk, dv, g and dg once) plus the plan's replay rows and states.

    Per compact (own) row, with E = d * el bytes per head vector:
      forward          q, k, v, g read; o written           H (4E + 4)
      backward         q, k, v, dO, g read; dq, dk, dv, dg   H (7E + 8)
      recompute        q, k, v, g read (state pass)          H (3E + 4)
    Per replay row: k, v, g read in every pass (H (2E + 4) each), and in the
    backward its dk, dv, dg contributions written once, float32
    (H (2d + 1) 4).  Per state (H d d 4 bytes): forward reads every
    sequence's initial state and writes every requested state and every
    final state; the backward reads initial states, dS_final and the
    requested states' gradients and writes dS0 of every sequence; the
    recompute reads initial states again.

    Returns {"fwd", "bwd", "state"} bytes and the share of the two backward
    kernels and of the forward block kernel (the bytes of their own outputs:
    the inputs those outputs need, once, and the outputs).  At H = 16,
    d = 128, bf16 the per-row figures are 16,448 / 28,800 / 12,352 bytes."""
    E = d * el
    st = H * d * d * 4
    C, R = plan.info["C"], plan.info["R"]
    n_seq, n_slots, n_leaves = plan.info["n_seq"], plan.info["n_slots"], plan.info["n_leaves"]
    rep = H * (2 * E + 4)
    out = {
        "fwd": C * H * (4 * E + 4) + R * rep + (n_seq + n_slots + n_leaves) * st,
        "bwd": C * H * (7 * E + 8) + R * (rep + H * (2 * d + 1) * 4)
               + (2 * n_seq + n_leaves + n_slots) * st,
        "state": C * H * (3 * E + 4) + R * rep + n_seq * st,
    }
    # per-kernel shares, per step (each kernel runs once per round)
    share = {
        "k_fwd_block": C * H * (4 * E + 4) + R * rep + (n_seq + n_leaves) * st,
        "k_bwd_fwdorder": C * H * (5 * E + 4) + R * rep + n_seq * st,
        "k_bwd_revorder": C * H * (6 * E + 8) + R * (rep + H * (2 * d + 1) * 4)
                          + 2 * n_seq * st,
    }
    return out, share


def design_bytes(plan, H, d, el):
    """Design traffic: the bytes each kernel of this implementation moves
    over one step (forward, then the backward with the recompute-forward),
    by kernel, for the launches the runner makes -- a diagnostic of the
    decomposition, not the method's minimum (``alg_bytes``).  The local adjoint of a block is formed by the
    forward-order backward kernel, which reads the block's q and dO anyway.

    Rows are packed rows (own + replay); q, o, dO and dq exist on own rows
    only.  Block-level states (summaries, chained block-end states, local
    adjoints) are float32 H*d*d each and are counted for the kernels whose
    job is to produce or consume them; per-chunk states are never
    materialised.  Initial states are read in place from the bank (no
    gather).  The block kernels end every sequence's forward chain and start
    its adjoint chain: no forward summary of a last block (its g only, for
    the total decay), no adjoint summary of a first block, no chain step for
    either; the forward block kernel writes the final states, the
    forward-order backward kernel reads dS_final for the boundary term, the
    reverse-order one starts last blocks from dS_final and writes dS0.
    Returns (bytes per step, launches per step) per kernel, and the bytes of
    the separate passes: "fwd" (outputs and final states), "state" (the
    state pass that the recompute-forward repeats) and "bwd" (the backward
    from saved block states)."""
    st = H * d * d * 4
    B = 64
    names = ["k_blocksum", "k_fwd_blockscan", "k_fwd_block", "k_bwd_fwdorder", "k_bwd_blockscan",
             "k_bwd_revorder", "k_dg_carry", "k_scatter_add", "k_replay_reduce"]
    b = dict.fromkeys(names, 0)
    n = dict.fromkeys(names, 0)
    passes = {"fwd": 0, "state": 0, "bwd": 0}
    init_bank = np.asarray(plan["seq_init_bank"])
    for r in plan.rounds:
        rows, own, rep, nseq, nblk = (r["n_rows"], r["n_own"], r["n_replay"], r["n_seq"],
                                      r["n_blk"])
        s0, s1 = r["seq_begin"], r["seq_begin"] + nseq
        blks = [seq_blocks(plan, i, B, r["block_chunks"]) for i in range(s0, s1)]
        assert sum(len(x) for x in blks) == nblk, "block count differs from the planner's"
        multi = [i for i, x in zip(range(s0, s1), blks) if len(x) > 1]
        nblk_m = sum(len(x) for x in blks if len(x) > 1)
        nseq_m = len(multi)
        rows_nl = sum(rw for x in blks for rw, _ in x[:-1])      # rows of blocks not last
        rows_l = sum(x[-1][0] for x in blks)                      # rows of last blocks
        nreq = int(sum(plan["seq_req_off"][i + 1] - plan["seq_req_off"][i] for i in range(s0, s1)))
        ninit = int(np.sum(init_bank[s0:s1] >= 0))             # sequences with a non-zero start
        ninit_m = int(sum(1 for i in multi if init_bank[i] >= 0))
        kv = rows * H * (2 * d * el + 4)                        # k, v, g of every packed row
        chained = nblk_m - nseq_m                               # blocks with a chain step
        starts = (nblk - nseq + ninit) * st                     # start state of every block
        # forward chain (start states of blocks after the first): summaries
        # in, states out, the initial states in, requested states out; in the
        # forward and in the recompute pass
        scan = 2 * chained * st + ninit_m * st + nreq * st
        # the recompute inside the backward writes no bank slots
        b["k_fwd_blockscan"] += 2 * scan - nreq * st
        n["k_fwd_blockscan"] += 2
        # forward summaries, in the forward and the recompute pass (k, v, g
        # of blocks not last, g of last blocks)
        side0 = rows_nl * H * (2 * d * el + 4) + rows_l * H * 4 + (nblk - nseq) * st
        b["k_blocksum"] += 2 * side0
        n["k_blocksum"] += 2
        fblock = kv + own * H * 2 * d * el + starts + nseq * st
        b["k_fwd_block"] += fblock
        # dq and q.dq, and the local adjoints of blocks not first (written)
        fwdorder = kv + own * H * 3 * d * el + rows * H * 4 + starts + nseq * st + (nblk - nseq) * st
        b["k_bwd_fwdorder"] += fwdorder
        # adjoint chain: dS_final in, local adjoints of blocks not first in,
        # end adjoints of blocks not last out, requested injections and states in
        bscan = (nseq_m + 2 * chained + 2 * nreq) * st
        b["k_bwd_blockscan"] += bscan
        revorder = (kv + own * H * (2 * d * el + 2 * d * el + 4) + rep * H * (2 * d + 1) * 4
                    + rows * H * 4 + nblk * st + nseq * st)
        b["k_bwd_revorder"] += revorder
        b["k_dg_carry"] += rows * H * 8
        b["k_scatter_add"] += 3 * nseq * st
        for name in ("k_fwd_block", "k_bwd_fwdorder", "k_bwd_blockscan", "k_bwd_revorder",
                     "k_dg_carry", "k_scatter_add"):
            n[name] += 1
        passes["fwd"] += side0 + scan + fblock
        passes["state"] += side0 + scan - nreq * st
        passes["bwd"] += bscan + fwdorder + revorder + rows * H * 8 + 3 * nseq * st
    R = plan.info["R"]
    b["k_replay_reduce"] = R * H * (2 * d + 1) * 4 + R * H * (2 * d * el * 2 + 8)
    n["k_replay_reduce"] = 1 if R else 0
    passes["bwd"] += b["k_replay_reduce"]
    assert abs(passes["fwd"] + passes["state"] + passes["bwd"] - sum(b.values())) < 1, \
        "pass bytes add up to the step"
    return b, n, passes


def read_traffic(kernel, workload_key):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if
    it was taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload_key}.txt")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("source_sha") != la_source_sha(kernel):
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _cpu_item(args):
    """One (trajectory, head) work item of the fp64 trajectory-wise
    recurrence: the forward, or the backward (which runs the forward states
    itself).  Runs in a worker process; returns (tokens, seconds)."""
    from oracle.recurrent import la_bwd, la_fwd
    q, k, v, g, dO, dSf, scale, mode = args
    t0 = time.perf_counter()
    S0 = np.zeros((1, q.shape[2], v.shape[2]))
    if mode == "fwd":
        la_fwd(q, k, v, g, S0, scale)
    else:
        la_bwd(q, k, v, g, S0, scale, dO, dSf)
    return q.shape[0], time.perf_counter() - t0


def _trajectory_rows(forest):
    parent = forest.parent
    row0 = np.concatenate([[0], np.cumsum(forest.seg_len)[:-1]])
    out = []
    for leaf in forest.leaves():
        path, v = [], leaf
        while v >= 0:
            path.append(v)
            v = parent[v]
        out.append(np.concatenate([row0[w] + np.arange(forest.seg_len[w]) for w in reversed(path)]))
    return out


def cpu_baseline(forest, x, cfg, budget_s=8.0, seed=0):
    """The fp64 oracle's trajectory-wise recurrence (every root-to-leaf path
    run token by token, forward and backward) on the host's cores: a
    process pool over (trajectory, head) items on every core of
    os.sched_getaffinity (at most 16, the box's share), and one core.  Each
    run takes a seeded random sample of the workload's items until its work
    reaches about budget_s seconds of pool time; the measured token-head
    rate is scaled to the whole job (S trajectory tokens times H heads) and
    reported as compact tokens per second, C / time."""
    import multiprocessing as mp
    trajs = _trajectory_rows(forest)
    H, d = cfg["H"], cfg["d"]
    S = sum(len(r) for r in trajs)
    rng = np.random.default_rng(seed)
    items = [(t, h) for t in range(len(trajs)) for h in range(H)]
    order = rng.permutation(len(items))

    def item_args(i, mode):
        t, h = items[i]
        r = trajs[t]
        sl = lambda a: np.ascontiguousarray(a[r][:, h:h + 1])
        return (sl(x["q"]), sl(x["k"]), sl(x["v"]), sl(x["g"]), sl(x["dO"]),
                x["dS_final"][t, h:h + 1].astype(np.float64), d ** -0.5, mode)

    ncore = min(len(os.sched_getaffinity(0)), 16)
    os.environ.setdefault("OMP_NUM_THREADS", "1")
    ctx = mp.get_context("spawn")
    res = {}
    for label, procs in (("all_cores", ncore), ("one_core", 1)):
        res[label] = {"cores": procs}
        with ctx.Pool(procs) as pool:
            for mode in ("fwd", "fwd_bwd"):
                # probe: one short item gives the per-token cost; then a sample
                # sized to the budget
                n_tok, sec = pool.apply(_cpu_item, (item_args(order[0], mode),))
                per_tok = sec / max(n_tok, 1)
                want = budget_s * procs / per_tok / (2 if label == "one_core" else 1)
                pick, tok = [], 0
                for i in order:
                    if tok >= want:
                        break
                    pick.append(i)
                    tok += len(trajs[items[i][0]])
                t0 = time.perf_counter()
                done = pool.map(_cpu_item, [item_args(i, mode) for i in pick], chunksize=1)
                wall = time.perf_counter() - t0
                tok_heads = sum(n for n, _ in done)
                full_s = S * H / (tok_heads / wall)
                res[label][mode] = {"compact_tok_s": forest.n_rows / full_s,
                                    "items": len(pick), "token_heads": tok_heads,
                                    "wall_s": wall, "job_s_est": full_s}
    a = res["all_cores"]
    return {"value": a["fwd_bwd"]["compact_tok_s"], "unit": "compact tokens/s",
            "cores": a["cores"], "kind": "oracle",
            "sample": (f"fp64 trajectory-wise recurrence (oracle), forward + backward, "
                       f"{a['fwd_bwd']['items']} random (trajectory, head) items of the same "
                       f"microbatch ({a['fwd_bwd']['token_heads']} token-heads of "
                       f"{S * H}) in {a['fwd_bwd']['wall_s']:.1f} s on a pool of {a['cores']} "
                       f"processes, scaled to the whole job (S = {S} trajectory tokens x "
                       f"{H} heads), reported as C / time"),
            "forward_compact_tok_s": a["fwd"]["compact_tok_s"],
            "one_core": {"cores": 1,
                         "fwd_bwd_compact_tok_s": res["one_core"]["fwd_bwd"]["compact_tok_s"],
                         "fwd_compact_tok_s": res["one_core"]["fwd"]["compact_tok_s"]},
            "detail": res}


def run_step(runner, t):
    fwd = runner.forward(t["q"], t["k"], t["v"], t["g"], t["S0"], outputs=True,
                         keep_states=False)
    runner.backward(t["q"], t["k"], t["v"], t["g"], t["dO"], t["dS_final"], fwd=fwd,
                    S0_tree=t["S0"], recompute=True)
    return fwd


def time_steps(runner, t, steps, warmup, profile, fn=None):
    """Times `steps` calls of fn (default: one full step) after `warmup`
    untimed ones, bracketed by synchronisations.  Returns (mean ms, kernel
    profile, per-step ms) -- per-step times from events between the steps."""
    import torch
    from paper_2608_28158_amd import _lib
    fn = fn or (lambda: run_step(runner, t))
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    if profile:
        _lib.profile_begin()
    ev[0].record(stream)
    for i in range(steps):
        fn()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    ms = ev[0].elapsed_time(ev[steps]) / steps
    kern = _lib.profile_end() if profile else {}
    return ms, kern, per


def pass_times(runner, t, steps, warmup):
    """Median ms of the separate passes: forward, backward from saved states,
    forward + backward (states saved), forward + backward with
    recompute-forward."""
    q, k, v, g, dO, dSf, S0 = (t[n] for n in ("q", "k", "v", "g", "dO", "dS_final", "S0"))
    saved = runner.forward(q, k, v, g, S0, outputs=True, keep_states=True)
    fns = {
        "fwd": lambda: runner.forward(q, k, v, g, S0, outputs=True, keep_states=False),
        "bwd": lambda: runner.backward(q, k, v, g, dO, dSf, fwd=saved, S0_tree=S0,
                                       recompute=False),
        "fwd_bwd": lambda: runner.backward(q, k, v, g, dO, dSf,
                                           fwd=runner.forward(q, k, v, g, S0, outputs=True,
                                                              keep_states=True),
                                           S0_tree=S0, recompute=False),
        "recompute_fwd_bwd": lambda: run_step(runner, t),
    }
    out = {}
    for name, fn in fns.items():
        _, _, per = time_steps(runner, t, steps, warmup, False, fn)
        out[name] = float(np.median(per))
    return out


def setup(idx):
    import torch
    from paper_2608_28158_amd.plan import HartsPlan
    from paper_2608_28158_amd.tree_la import TreeLARunner
    from workloads import config_inputs
    forest, cfg, x = config_inputs(idx)
    plan_times = []
    for _ in range(5):
        t0 = time.perf_counter()
        plan = HartsPlan(forest.parent, forest.seg_len, 64, heads=cfg["H"])
        plan_times.append(time.perf_counter() - t0)
    phys = phys_index(forest.seg_len, plan["seg_row"])
    dt = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
    t = dict(q=to_device(x["q"], phys, dt), k=to_device(x["k"], phys, dt),
             v=to_device(x["v"], phys, dt), g=to_device(x["g"], phys, torch.float32),
             dO=to_device(x["dO"], phys, dt),
             dS_final=torch.from_numpy(x["dS_final"]).cuda(),
             S0=torch.from_numpy(x["S0"]).cuda())
    runner = TreeLARunner(plan, cfg["H"], cfg["d"], dt, "cuda")
    return forest, cfg, x, plan, t, runner, float(np.median(plan_times))


def expanded_comparison(steps, warmup):
    """Config 4: the same inputs run tree-packed and trajectory-wise (every
    root-to-leaf path its own zero-initialised sequence, inputs expanded on
    the device beforehand, one packed call)."""
    import torch
    from paper_2608_28158_amd.plan import HartsPlan
    from paper_2608_28158_amd.tree_la import TreeLARunner
    forest, cfg, x, plan, t, runner, _ = setup(4)
    ms_tree, _, _ = time_steps(runner, t, steps, warmup, profile=False)
    # expanded forest: one single-segment tree per trajectory, canonical rows
    parent = forest.parent
    row0 = np.concatenate([[0], np.cumsum(forest.seg_len)[:-1]])
    trajs = []
    for leaf in forest.leaves():
        path = []
        v = leaf
        while v >= 0:
            path.append(v)
            v = parent[v]
        rows = np.concatenate([row0[w] + np.arange(forest.seg_len[w]) for w in reversed(path)])
        trajs.append(rows)
    lens = np.array([len(r) for r in trajs], np.int64)
    eplan = HartsPlan(np.full(len(trajs), -1, np.int32), lens, 64, heads=cfg["H"])
    assert eplan.info["n_rounds"] == 1
    erows = np.concatenate(trajs)                       # canonical row of each expanded row
    ephys = phys_index(lens, eplan["seg_row"])          # expanded canonical -> physical
    dt = t["q"].dtype
    te = {}
    for name in ("q", "k", "v", "g", "dO"):
        src = x[name][erows]
        te[name] = to_device(src, ephys, torch.float32 if name == "g" else dt)
    te["dS_final"] = torch.from_numpy(x["dS_final"]).cuda()
    te["S0"] = torch.zeros((len(trajs), cfg["H"], cfg["d"], cfg["d"]), dtype=torch.float32,
                           device="cuda")
    erunner = TreeLARunner(eplan, cfg["H"], cfg["d"], dt, "cuda")
    ms_exp, _, _ = time_steps(erunner, te, steps, warmup, profile=False)
    # metamorphic check (Sec. 2.2: the same chunk grid from every
    # trajectory's start): outputs agree on every trajectory row and final
    # states per leaf; with row c's upstream gradient given to one
    # trajectory through c, the compact gradients of c equal the sums over
    # the trajectories through c
    first = np.full(forest.n_rows, -1, np.int64)
    for i, r in enumerate(trajs):
        new = first[r] < 0
        first[r[new]] = i
    owner = np.repeat(np.arange(len(trajs)), lens)
    dO_e = np.where((first[erows] == owner)[:, None, None], x["dO"][erows], 0).astype(np.float32)
    te_chk = dict(te, dO=to_device(dO_e, ephys, dt))

    def full(rn, tt):
        fwd = rn.forward(tt["q"], tt["k"], tt["v"], tt["g"], tt["S0"], outputs=True,
                         keep_states=False)
        grads = rn.backward(tt["q"], tt["k"], tt["v"], tt["g"], tt["dO"], tt["dS_final"],
                            fwd=fwd, S0_tree=tt["S0"], recompute=True)
        out = {"o": fwd["o"], "S_final": fwd["S_final"]}
        out.update({n: grads[n] for n in ("dq", "dk", "dv", "dg")})
        return {n: v.float().cpu().numpy().astype(np.float64) for n, v in out.items()}

    a = full(runner, t)
    b = full(erunner, te_chk)
    phys = phys_index(forest.seg_len, plan["seg_row"])
    rel = lambda u, w: float(np.max(np.abs(u - w)) / max(np.max(np.abs(w)), 1e-30))
    agree = {"o": rel(a["o"][phys][erows], b["o"][ephys]),
             "S_final": rel(a["S_final"], b["S_final"])}
    for n in ("dq", "dk", "dv", "dg"):
        acc = np.zeros_like(a[n])
        np.add.at(acc, erows, b[n][ephys])
        agree[n] = rel(a[n][phys], acc)
    tol = 2e-2 if cfg["dtype"] == "bf16" else 1e-4
    bad = {n: e for n, e in agree.items() if not e <= tol}
    assert not bad, f"tree-packed and expanded runs disagree: {bad}"
    C = forest.n_rows
    S = int(lens.sum())
    return {"workload": "4 agentic trees, ~32k compact tokens, H=16, d=128, bf16, fwd+bwd "
                        "with recompute",
            "C": C, "S": S, "expansion_S_over_C": S / C,
            "tree_packed_ms": ms_tree, "expanded_ms": ms_exp,
            "tree_packed_compact_tok_s": C / (ms_tree * 1e-3),
            "expanded_compact_tok_s": C / (ms_exp * 1e-3),
            "speedup": ms_exp / ms_tree,
            "agreement_max_rel": agree, "agreement_tol": tol,
            "paper_context": "4.81-4.87x F/B/Grad end-to-end speedup, 8x H20-3e, BF16, "
                             "Ling-3.0-tiny (whole model, not this operator)"}


LOGP_V = 157184        # the paper's vocabulary (bf16 logits)


def logp_measurement(steps, warmup, profile_only=False):
    """Compact-to-semantic log-probabilities on the same 64k-token
    microbatch: 68,161 compact logit rows x 157,184 bf16 logits (seeded
    N(0, 4) on the device), every nonterminal semantic position; forward
    (row log-sum-exp, target gather) and backward (row sums, softmax
    gradient rows, target columns) timed separately with events on the
    launch stream.  Algorithmic bytes: the forward reads the logits once,
    the backward reads them once and writes dlogits once; per row and per
    position only scalars move (counted)."""
    import ctypes as C
    import torch
    from paper_2608_28158_amd import _lib
    from paper_2608_28158_amd.plan import HartsPlan
    from workloads import forest_for_config
    L = _lib.lib()
    f, _, cfg = forest_for_config(2)
    t0 = time.perf_counter()
    plan = HartsPlan(f.parent, f.seg_len, 64, heads=cfg["H"])
    Cn, V = f.n_rows, LOGP_V
    rng = np.random.default_rng(42)
    tok = rng.integers(0, V, size=Cn).astype(np.int32)          # physical row order
    n_pos = plan["S"] - plan["n_leaves"]
    m = np.zeros(n_pos, np.int32)
    y = np.zeros(n_pos, np.int32)
    off = np.zeros(Cn + 1, np.int64)
    pos = np.zeros(n_pos, np.int32)
    t1 = time.perf_counter()
    _lib.check(L.harts_semantic_map(plan.handle, tok.ctypes.data, n_pos, m.ctypes.data,
                                    y.ctypes.data, off.ctypes.data, pos.ctypes.data),
               "harts_semantic_map")
    map_ms = (time.perf_counter() - t1) * 1e3
    g = (rng.standard_normal(n_pos) * (rng.random(n_pos) < 0.7)).astype(np.float32)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    md, yd, offd, posd, gd = dev(m), dev(y), dev(off), dev(pos), dev(g)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(42)
    z = torch.empty((Cn, V), dtype=torch.bfloat16, device="cuda")
    for i in range(0, Cn, 4096):
        n = min(4096, Cn - i)
        z[i:i + n] = torch.randn((n, V), device="cuda", generator=gen).mul_(2.0)
    dz = torch.empty_like(z)
    lse = torch.empty(Cn, dtype=torch.float32, device="cuda")
    logp = torch.empty(n_pos, dtype=torch.float32, device="cuda")
    row_g = torch.empty(Cn, dtype=torch.float32, device="cuda")
    P = lambda t: C.c_void_p(t.data_ptr())
    stream = torch.cuda.current_stream()
    st = C.c_void_p(stream.cuda_stream)
    code = _lib.HARTS_BF16

    def fwd():
        _lib.check(L.harts_logp_fwd(code, Cn, V, P(z), n_pos, P(md), P(yd), P(lse), P(logp), st),
                   "harts_logp_fwd")

    def bwd():
        _lib.check(L.harts_logp_bwd(code, Cn, V, P(z), P(lse), n_pos, P(offd), P(posd), P(yd),
                                    P(gd), P(row_g), P(dz), st), "harts_logp_bwd")

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record(stream)
        for _ in range(steps):
            fn()
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / steps

    ms_f = timed(fwd)
    ms_b = timed(bwd)
    if profile_only:
        return None
    el = 2
    by_f = Cn * V * el + Cn * 4 + n_pos * (4 + 4 + el + 4 + 4)
    by_b = 2 * Cn * V * el + Cn * (8 + 4 + 4 + 4) + n_pos * (4 + 4 + 4) + n_pos * (el * 2 + 4)
    out = {"workload": f"64k-token agentic microbatch: {Cn} compact logit rows x {V} bf16 "
                       f"logits, {n_pos} semantic positions",
           "C": Cn, "V": V, "positions": n_pos,
           "fwd_ms": ms_f, "bwd_ms": ms_b,
           "fwd": {"alg_GB": by_f / 1e9, "achieved_GBs": by_f / (ms_f * 1e-3) / 1e9,
                   "hbm_frac": by_f / (ms_f * 1e-3) / 1e9 / PEAK_HBM_GBS},
           "bwd": {"alg_GB": by_b / 1e9, "achieved_GBs": by_b / (ms_b * 1e-3) / 1e9,
                   "hbm_frac": by_b / (ms_b * 1e-3) / 1e9 / PEAK_HBM_GBS},
           "semantic_positions_per_s_fwd_bwd": n_pos / ((ms_f + ms_b) * 1e-3),
           "traffic_k_logp_lse": read_traffic("k_logp_lse", "agentic64k_v157184"),
           "traffic_k_logp_grad": read_traffic("k_logp_grad", "agentic64k_v157184"),
           "map_ms": map_ms, "plan_ms": (t1 - t0) * 1e3}
    # the oracle's one log-softmax per semantic position (fp64), timed on a
    # sample of positions and scaled to all of them
    from oracle.logprob import logp_bwd, logp_fwd
    k = 1024
    sel = rng.choice(n_pos, k, replace=False)
    rows = z[torch.from_numpy(m[sel]).cuda().long()].float().cpu().numpy()
    loc = np.arange(k)
    t2 = time.perf_counter()
    logp_fwd(rows, loc, y[sel])
    logp_bwd(rows, loc, y[sel], g[sel].astype(np.float64))
    cpu_s = time.perf_counter() - t2
    out["cpu_baseline"] = {"value": k / cpu_s, "unit": "semantic positions/s", "cores": 1,
                           "kind": "oracle",
                           "sample": f"{k} random positions of the same microbatch, forward + "
                                     f"backward, one fp64 log-softmax over {V} logits per "
                                     f"position ({cpu_s:.1f} s)"}
    del z, dz
    torch.cuda.empty_cache()
    return out


CONV_CH, CONV_W = 6144, 4   # q, k, v of 16 heads x 128; the paper's KDA width


def conv_measurement(steps, warmup, profile_only=False):
    """Causal depthwise convolution with true-ancestor context on the
    64k-token microbatch: 68,161 compact rows x 6,144 bf16 channels, width
    4.  Algorithmic bytes: the forward reads x once and writes y once; the
    backward reads dy and writes dx once, and reads x and dy once more for
    the weight gradient (the taps of a row's window hit rows already read);
    the row tables (12 bytes a row) are counted."""
    import ctypes as C
    import torch
    from paper_2608_28158_amd import _lib
    from paper_2608_28158_amd.plan import HartsPlan
    from workloads import forest_for_config
    L = _lib.lib()
    f, _, cfg = forest_for_config(2)
    plan = HartsPlan(f.parent, f.seg_len, 64, heads=cfg["H"])
    Cn, Cch, w = f.n_rows, CONV_CH, CONV_W
    k = w - 1
    pred = np.zeros(Cn * k, np.int32)
    off = np.zeros(Cn + 1, np.int64)
    succ = np.zeros(Cn * k, np.int32)
    t0 = time.perf_counter()
    _lib.check(L.harts_conv_context(plan.handle, w, pred.ctypes.data, off.ctypes.data,
                                    succ.ctypes.data), "harts_conv_context")
    ctx_ms = (time.perf_counter() - t0) * 1e3
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    pd, od, sd = dev(pred), dev(off), dev(succ)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7)
    x = torch.randn((Cn, Cch), device="cuda", generator=gen).to(torch.bfloat16)
    dy = torch.randn((Cn, Cch), device="cuda", generator=gen).to(torch.bfloat16)
    Wd = (torch.randn((Cch, w), device="cuda", generator=gen) * 0.5).contiguous()
    y, dx = torch.empty_like(x), torch.empty_like(x)
    dW = torch.empty((Cch, w), dtype=torch.float32, device="cuda")
    sz = C.c_size_t()
    _lib.check(L.harts_conv_workspace_size(Cn, Cch, w, C.byref(sz)), "harts_conv_workspace_size")
    ws = torch.empty(sz.value, dtype=torch.uint8, device="cuda")
    P = lambda t: C.c_void_p(t.data_ptr())
    stream = torch.cuda.current_stream()
    st = C.c_void_p(stream.cuda_stream)
    code = _lib.HARTS_BF16

    def fwd():
        _lib.check(L.harts_conv_fwd(code, Cn, Cch, w, P(x), P(Wd), P(pd), P(y), st), "harts_conv_fwd")

    def bwd():
        _lib.check(L.harts_conv_bwd(code, Cn, Cch, w, P(x), P(Wd), P(pd), P(od), P(sd), int(off[-1]),
                                    P(dy), P(dx), P(dW), P(ws), ws.numel(), st), "harts_conv_bwd")

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record(stream)
        for _ in range(steps):
            fn()
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / steps

    ms_f, ms_b = timed(fwd), timed(bwd)
    if profile_only:
        return None
    row = Cch * 2
    by_f = 2 * Cn * row + Cn * 12 + Cch * w * 4
    by_b = 3 * Cn * row + Cn * 12 + int(off[-1]) * 4 + Cn * 8 + 2 * Cch * w * 4
    out = {"workload": f"64k-token agentic microbatch: {Cn} compact rows x {Cch} bf16 channels, "
                       f"width {w}",
           "fwd_ms": ms_f, "bwd_ms": ms_b,
           "fwd": {"alg_GB": by_f / 1e9, "achieved_GBs": by_f / (ms_f * 1e-3) / 1e9,
                   "hbm_frac": by_f / (ms_f * 1e-3) / 1e9 / PEAK_HBM_GBS},
           "bwd": {"alg_GB": by_b / 1e9, "achieved_GBs": by_b / (ms_b * 1e-3) / 1e9,
                   "hbm_frac": by_b / (ms_b * 1e-3) / 1e9 / PEAK_HBM_GBS},
           "context_ms": ctx_ms,
           "traffic_k_conv_fwd": read_traffic("k_conv_fwd", "agentic64k_c6144"),
           "traffic_k_conv_bwd": read_traffic("k_conv_bwd", "agentic64k_c6144")}
    # the oracle (fp64, trajectory by trajectory) on a sample of channels
    from oracle.conv import conv_bwd, conv_fwd
    chs = 8
    phys = phys_index(f.seg_len, plan["seg_row"])
    take = lambda t: t[:, :chs].float().cpu().numpy()[phys]
    xs, dys, Ws = take(x), take(dy), Wd[:chs].cpu().numpy()
    t1 = time.perf_counter()
    conv_fwd(f.parent, f.seg_len, xs, Ws)
    conv_bwd(f.parent, f.seg_len, xs, Ws, dys)
    cpu_s = time.perf_counter() - t1
    out["cpu_baseline"] = {"value": Cn * chs / Cch / cpu_s, "unit": "compact rows/s (all channels)",
                           "cores": 1, "kind": "oracle",
                           "sample": f"{chs} of {Cch} channels, forward + backward over every "
                                     f"trajectory ({cpu_s:.1f} s), scaled by {Cch // chs}"}
    del x, dy, y, dx
    torch.cuda.empty_cache()
    return out


ATTN_H, ATTN_D = 16, 128


def attn_measurement(steps, warmup, profile_only=False):
    """Full attention through asymmetric Q/KV views on the 64k-token
    microbatch: 68,161 compact query rows, 16 heads of 128, bf16.  One step
    gathers the key and value views, runs the forward, the backward and the
    two gradient scatters; the view tables are built once per plan (host).
    Algorithmic FLOPs count visible (query, key) pairs only: 4 d per pair
    and head forward (scores, P V), 10 d backward (scores, dP, dV, dK, dQ);
    the kernels also recompute the scores and dP once more in the dq pass
    and spend the masked halves of diagonal tiles."""
    import ctypes as C
    import torch
    from paper_2608_28158_amd import _lib
    from paper_2608_28158_amd.plan import HartsPlan
    from workloads import forest_for_config
    L = _lib.lib()
    f, _, cfg = forest_for_config(2)
    H, d = ATTN_H, ATTN_D
    plan = HartsPlan(f.parent, f.seg_len, 64, heads=H)
    Cn = f.n_rows
    t0 = time.perf_counter()
    lay = _lib.AttnLayout()
    _lib.check(L.harts_attn_layout(plan.handle, C.byref(lay)), "harts_attn_layout")
    views = np.zeros((lay.n_views, 4), np.int32)
    kv_rows = np.zeros(lay.n_kv, np.int32)
    qt = np.zeros((lay.n_qtiles, 2), np.int32)
    kt = np.zeros((lay.n_kvtiles, 2), np.int32)
    off = np.zeros(Cn + 1, np.int64)
    ent = np.zeros(lay.n_kv, np.int32)
    _lib.check(L.harts_attn_views(plan.handle, views.ctypes.data, kv_rows.ctypes.data, qt.ctypes.data,
                                  kt.ctypes.data, off.ctypes.data, ent.ctypes.data), "harts_attn_views")
    views_ms = (time.perf_counter() - t0) * 1e3
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    vd, kr, qd, kd, od, ed = (dev(a) for a in (views, kv_rows, qt, kt, off, ent))
    gen = torch.Generator(device="cuda")
    gen.manual_seed(11)
    q, k, v, dO = (torch.randn((Cn, H, d), device="cuda", generator=gen).to(torch.bfloat16) for _ in range(4))
    nkv = lay.n_kv
    kvk = torch.empty((nkv, H, d), dtype=torch.bfloat16, device="cuda")
    kvv = torch.empty_like(kvk)
    o, dq, dk, dv = (torch.empty_like(q) for _ in range(4))
    lse = torch.empty((Cn, H), dtype=torch.float32, device="cuda")
    delta = torch.empty_like(lse)
    dkv = torch.empty((nkv, H, d), dtype=torch.float32, device="cuda")
    dvv = torch.empty_like(dkv)
    P = lambda x: C.c_void_p(x.data_ptr())
    stream = torch.cuda.current_stream()
    st = C.c_void_p(stream.cuda_stream)
    scale = C.c_float(d ** -0.5)

    def gather():
        _lib.check(L.harts_attn_gather(P(k), P(kr), nkv, Cn, H, d, P(kvk), st), "harts_attn_gather")
        _lib.check(L.harts_attn_gather(P(v), P(kr), nkv, Cn, H, d, P(kvv), st), "harts_attn_gather")

    def fwd():
        _lib.check(L.harts_attn_fwd(P(vd), P(qd), lay.n_qtiles, H, d, scale, P(q), P(kvk), P(kvv), P(o),
                                    P(lse), st), "harts_attn_fwd")

    def bwd():
        _lib.check(L.harts_attn_bwd(P(vd), P(qd), lay.n_qtiles, P(kd), lay.n_kvtiles, Cn, H, d, scale, P(q),
                                    P(kvk), P(kvv), P(o), P(lse), P(dO), P(delta), P(dq), P(dkv), P(dvv), st),
                   "harts_attn_bwd")

    def scatter():
        _lib.check(L.harts_attn_scatter(P(dkv), P(od), P(ed), Cn, nkv, H, d, P(dk), st), "harts_attn_scatter")
        _lib.check(L.harts_attn_scatter(P(dvv), P(od), P(ed), Cn, nkv, H, d, P(dv), st), "harts_attn_scatter")

    def step():
        gather()
        fwd()
        bwd()
        scatter()

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record(stream)
        for _ in range(steps):
            fn()
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / steps

    step()
    ms = {"step": timed(step), "gather": timed(gather), "fwd": timed(fwd), "bwd": timed(bwd),
          "scatter": timed(scatter)}
    if profile_only:
        return None
    hv = views[:, 3].astype(np.int64)
    lv = views[:, 1].astype(np.int64)
    pairs = int(np.sum(lv * hv + lv * (lv + 1) // 2))          # visible (query, key) pairs
    # pairs of a plain causal pass over every expanded trajectory
    from oracle.forest import SegTree
    t = SegTree(f.parent, f.seg_len)
    traj = np.array([t.s[u] + t.len[u] for u in t.leaves], np.int64)
    pairs_expanded = int(np.sum(traj * (traj + 1) // 2))
    fl_f, fl_b = 4 * d * pairs * H, 10 * d * pairs * H
    tf = lambda fl, m: fl / (m * 1e-3) / 1e12
    out = {"workload": f"64k-token agentic microbatch: {Cn} compact query rows, {lay.n_views} views, "
                       f"{nkv} view key rows, {H} heads of {d}, bf16",
           "ms_per_step": ms["step"], "compact_tok_s": Cn / (ms["step"] * 1e-3), "views_host_ms": views_ms,
           "visible_pairs": pairs, "expanded_pairs": pairs_expanded,
           "fwd": {"ms": ms["fwd"], "alg_TFLOP": fl_f / 1e12, "TFLOPs": tf(fl_f, ms["fwd"]),
                   "mfma_frac": tf(fl_f, ms["fwd"]) / PEAK_BF16_TFLOPS},
           "bwd": {"ms": ms["bwd"], "alg_TFLOP": fl_b / 1e12, "TFLOPs": tf(fl_b, ms["bwd"]),
                   "mfma_frac": tf(fl_b, ms["bwd"]) / PEAK_BF16_TFLOPS},
           "gather_ms": ms["gather"], "scatter_ms": ms["scatter"],
           "step_TFLOPs": tf(fl_f + fl_b, ms["step"])}
    # the oracle (fp64, every trajectory) on one tree and one head
    from oracle.attn import forest_attention
    tree0 = [u for u in range(t.n) if t.tree[u] == 0]
    ix = {u: i for i, u in enumerate(tree0)}
    par = [ix[f.parent[u]] if f.parent[u] >= 0 else -1 for u in tree0]
    sl = [int(f.seg_len[u]) for u in tree0]
    rows = np.concatenate([np.arange(t.row0[u], t.row0[u] + t.len[u]) for u in tree0])
    sub = lambda x: x[:, :1].float().cpu().numpy()[phys_index(f.seg_len, plan["seg_row"])][rows]
    t1 = time.perf_counter()
    forest_attention(par, sl, sub(q), sub(k), sub(v), d ** -0.5, dO=sub(dO))
    cpu_s = time.perf_counter() - t1
    out["cpu_baseline"] = {"value": len(rows) / H / cpu_s, "unit": "compact rows/s (all heads)",
                           "cores": torch.get_num_threads(), "kind": "oracle",
                           "sample": f"tree 0 ({len(rows)} compact rows, {len(par)} segments), 1 of {H} "
                                     f"heads, forward + backward over every trajectory ({cpu_s:.1f} s), "
                                     f"scaled by {H}"}
    del q, k, v, dO, kvk, kvv, dkv, dvv, o, dq, dk, dv
    torch.cuda.empty_cache()
    return out


def kda_measurement(steps, warmup, profile_only=False):
    """KDA (per-channel decay with the delta rule) over the plan of the
    64k-token microbatch: 68,161 compact rows, 16 heads of 128, bf16 q, k,
    v, float32 g and beta.  One step is the forward of every round and the
    backward of every round in reverse order, with the handoffs and the
    gradient reductions.  Algorithmic FLOPs per (64-row chunk, head) of the
    chunk form (eq. chunk-state): forward 5 B^2 d (At, M, W, U', M X) +
    6 B d^2 (W S, Q S, K^T X), backward twice that."""
    import torch
    from paper_2608_28158_amd.kda import KdaRunner
    from paper_2608_28158_amd.plan import HartsPlan
    from workloads import forest_for_config
    f, _, cfg = forest_for_config(2)
    H, d = cfg["H"], cfg["d"]
    plan = HartsPlan(f.parent, f.seg_len, 64, heads=H)
    Cn = f.n_rows
    t0 = time.perf_counter()
    run = KdaRunner(plan, H, d, torch.bfloat16)
    setup_ms = (time.perf_counter() - t0) * 1e3   # tables, their device copies and the workspace
    gen = torch.Generator(device="cuda")
    gen.manual_seed(13)
    rnd = lambda *sh: torch.randn(sh, device="cuda", generator=gen)
    q = rnd(Cn, H, d).to(torch.bfloat16)
    k = rnd(Cn, H, d)
    k = (k / k.norm(dim=-1, keepdim=True)).to(torch.bfloat16)
    v = rnd(Cn, H, d).to(torch.bfloat16)
    g = -0.3 * torch.rand((Cn, H, d), device="cuda", generator=gen)
    beta = 0.05 + 0.95 * torch.rand((Cn, H), device="cuda", generator=gen)
    dO = rnd(Cn, H, d).to(torch.bfloat16)
    S0 = 0.5 * rnd(plan["n_trees"], H, d, d)
    dSf = 0.1 * rnd(plan["n_leaves"], H, d, d)
    scale = d ** -0.5
    stream = torch.cuda.current_stream()

    def fwd():
        run.forward(q, k, v, g, beta, S0, scale)

    def step():
        run.forward(q, k, v, g, beta, S0, scale)
        run.backward(dO, dSf)

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record(stream)
        for _ in range(steps):
            fn()
        ev[1].record(stream)
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / steps

    ms_f, ms = timed(fwd), timed(step)
    if profile_only:
        return None
    nch = run.sizes.n_chunks
    B = 64
    fl_f = nch * H * (5 * B * B * d + 6 * B * d * d)
    fl = 3 * fl_f
    tf = lambda x, m: x / (m * 1e-3) / 1e12
    out = {"workload": f"64k-token agentic microbatch: {Cn} compact rows, {plan['R']} replay rows, "
                       f"{nch} packed 64-row chunks, K={plan['n_rounds']}, {H} heads of {d}, bf16 q/k/v, "
                       f"float32 g/beta/states",
           "ms_per_step": ms, "compact_tok_s": Cn / (ms * 1e-3), "fwd_ms": ms_f, "tables_host_ms": run.tables_ms,
           "runner_setup_ms": setup_ms,
           "alg_TFLOP_step": fl / 1e12, "TFLOPs": tf(fl, ms), "fwd_TFLOPs": tf(fl_f, ms_f),
           "fp32_peak_frac": tf(fl, ms) / PEAK_F32_TFLOPS}
    # the oracle: the trajectory-wise fp64 recurrence, forward and backward by
    # reverse mode, on the first 512 tokens of one trajectory and one head
    from oracle.kda import kda_recurrent
    from oracle.forest import SegTree
    t = SegTree(f.parent, f.seg_len)
    rows = t.trajectory_rows(t.leaves[0])[:512]
    phys = phys_index(f.seg_len, plan["seg_row"])
    pick = torch.from_numpy(phys[rows]).cuda()
    h1 = lambda x: x[pick][:, :1].double().cpu()
    xs = [h1(x).requires_grad_(True) for x in (q, k, v, g)] + [h1(beta).requires_grad_(True)]
    S0h = S0[0, :1].double().cpu().requires_grad_(True)
    dOh = h1(dO)
    t1 = time.perf_counter()
    o_, S_ = kda_recurrent(*xs, scale, S0h)
    (o_ * dOh).sum().backward()
    cpu_s = time.perf_counter() - t1
    rate = len(rows) / cpu_s                              # token-heads per second
    job_s = plan["S"] * H / rate
    out["cpu_baseline"] = {"value": Cn / job_s, "unit": "compact tokens/s", "cores": torch.get_num_threads(),
                           "kind": "oracle",
                           "sample": f"fp64 trajectory-wise recurrence, forward + backward by reverse mode, "
                                     f"{len(rows)} tokens of one trajectory and one head ({cpu_s:.1f} s), scaled "
                                     f"to S = {plan['S']} trajectory tokens x {H} heads"}
    del run
    torch.cuda.empty_cache()
    return out


def mbplan_measurement(D=4, T=65536):
    """Prefix-aware microbatch/DP planning at the paper's scale: a seeded
    batch of 215 agentic rollout trees at full length (about 1,600
    trajectories, 45 M trajectory tokens, 8.5 M compact), capacity 65,536
    and DP degree 4; trajectories longer than the capacity cannot be
    scheduled and are dropped.  The oracle (plain Python) is timed on the
    first 48 trajectories, next to the library on the same sample."""
    import ctypes as C
    from oracle.mbplan import plan_microbatches
    from paper_2608_28158_amd import _lib
    from workloads import agentic_forest, trajectory_tokens
    L = _lib.lib()
    f, rng = agentic_forest(11, 215, 1.0, 8_000_000, tol=0.1)
    all_t = trajectory_tokens(f, rng)
    trajs = [t for t in all_t if len(t) <= T]

    def run(ts):
        N = len(ts)
        off = np.zeros(N + 1, np.int64)
        off[1:] = np.cumsum([len(t) for t in ts])
        tok = np.concatenate(ts).astype(np.int32)
        outs = [np.zeros(N, np.int32) for _ in range(3)] + [np.zeros(N, np.int64)]
        res = _lib.MbResult()
        t0 = time.perf_counter()
        _lib.check(L.harts_mb_plan(N, off.ctypes.data, tok.ctypes.data, D, T, 0,
                                   *[o.ctypes.data for o in outs], C.byref(res)), "harts_mb_plan")
        return time.perf_counter() - t0, res

    times = []
    for _ in range(3):
        dt, res = run(trajs)
        times.append(dt)
    raw = sum(len(t) for t in trajs)
    sample = [list(map(int, t)) for t in trajs[:48]]
    dt_lib_s, res_s = run([np.asarray(t, np.int32) for t in sample])
    t0 = time.perf_counter()
    ref = plan_microbatches(sample, D, T)
    dt_orc = time.perf_counter() - t0
    assert ref["J"] == (res_s.work_total, res_s.slot_critical, res_s.replica_max)
    return {"workload": f"{len(trajs)} trajectories of 215 agentic rollout trees "
                        f"({len(all_t) - len(trajs)} above the capacity dropped), "
                        f"{raw} trajectory tokens, T={T}, D={D}",
            "plan_ms": float(np.median(times)) * 1e3, "K": res.K, "natural_K": res.natural_K,
            "J": [res.work_total, res.slot_critical, res.replica_max],
            "trie_work_one_microbatch": res.trie_work,
            "raw_over_compact": raw / res.work_total,
            "cpu_baseline": {"value": 48 / dt_orc, "unit": "trajectories planned/s", "cores": 1,
                             "kind": "oracle",
                             "sample": f"first 48 trajectories, {dt_orc:.2f} s; the library plans "
                                       f"the same sample in {dt_lib_s * 1e3:.2f} ms with the "
                                       f"same J"}}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", type=int, default=2, choices=(1, 2, 3))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-expanded", action="store_true")
    ap.add_argument("--no-logp", action="store_true")
    ap.add_argument("--no-mbplan", action="store_true")
    ap.add_argument("--no-conv", action="store_true")
    ap.add_argument("--no-attn", action="store_true")
    ap.add_argument("--no-kda", action="store_true")
    ap.add_argument("--kda-only", action="store_true",
                    help="run the timed KDA steps only (for profiler runs)")
    ap.add_argument("--attn-only", action="store_true",
                    help="run the timed attention calls only (for profiler runs)")
    ap.add_argument("--conv-only", action="store_true",
                    help="run the timed convolution calls only (for profiler runs)")
    ap.add_argument("--steps-only", action="store_true",
                    help="run the timed steps only (for profiler runs)")
    ap.add_argument("--logp-only", action="store_true",
                    help="run the timed log-probability calls only (for profiler runs)")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="run a plain device copy of this many MiB (counter scale)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1"}))
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    if args.copy_probe_mib:
        n = args.copy_probe_mib * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        log(f"copy probe: {args.copy_probe_mib} MiB read + written, 5 launches")
        return
    if args.logp_only:
        logp_measurement(args.steps, args.warmup, profile_only=True)
        log("[bench] logp calls done")
        return
    if args.kda_only:
        kda_measurement(args.steps, args.warmup, profile_only=True)
        log("[bench] kda steps done")
        return
    if args.attn_only:
        attn_measurement(args.steps, args.warmup, profile_only=True)
        log("[bench] attention calls done")
        return
    if args.conv_only:
        conv_measurement(args.steps, args.warmup, profile_only=True)
        log("[bench] conv calls done")
        return
    log(f"[bench] config {args.config}: building workload")
    forest, cfg, x, plan, t, runner, plan_s = setup(args.config)
    log(f"[bench] C={plan.info['C']} S={plan.info['S']} R={plan.info['R']} "
        f"K={plan.info['n_rounds']} seqs={plan.info['n_seq']}")
    ms, _, step_ms = time_steps(runner, t, args.steps, args.warmup, profile=False)
    log(f"[bench] {ms:.3f} ms/step")
    if args.steps_only:
        return
    # per-kernel times come from a separate run: the events recorded around
    # every launch add host and queue work to the step
    _, kern, _ = time_steps(runner, t, args.steps, 1, profile=True)
    H, d = cfg["H"], cfg["d"]
    el = 2 if cfg["dtype"] == "bf16" else 4
    C = plan.info["C"]
    K = plan.info["n_rounds"]
    value = C / (ms * 1e-3)
    pass_bytes, share = alg_bytes(plan, H, d, el)
    step_bytes = pass_bytes["fwd"] + pass_bytes["state"] + pass_bytes["bwd"]
    dbytes, per_step, dpass = design_bytes(plan, H, d, el)
    kstats = {}
    ktot = sum(v[1] for v in kern.values())
    for name, (n, tot) in kern.items():
        avg_ms = tot / n
        st = {"launches": n, "avg_ms": avg_ms, "share_of_time": tot / ktot}
        if name in share:        # its own outputs' bytes, per launch (one launch per round)
            b = share[name] / K
            st.update(alg_bytes_per_launch=b, alg_GBs=b / (avg_ms * 1e-3) / 1e9,
                      alg_frac=b / (avg_ms * 1e-3) / 1e9 / PEAK_HBM_GBS)
        if name in dbytes and per_step.get(name):
            b = dbytes[name] / per_step[name]
            st.update(design_bytes_per_launch=b, design_GBs=b / (avg_ms * 1e-3) / 1e9)
        kstats[name] = st
    dom = max(kstats, key=lambda k: kstats[k]["avg_ms"] * kstats[k]["launches"])
    if dom not in share:
        raise RuntimeError(f"dominant kernel {dom} has no algorithmic share")
    ds = kstats[dom]
    traffic = read_traffic(dom, WORKLOAD_KEY[args.config])
    flop_tok = H * (98304 + 245760 + 32768) * (d / 128) ** 2  # fwd + bwd + recompute state pass
    achieved_tflops = C * flop_tok / (ms * 1e-3) / 1e12
    peak_tf = PEAK_BF16_TFLOPS if el == 2 else PEAK_F32_TFLOPS
    step_gbs = step_bytes / (ms * 1e-3) / 1e9
    out = {
        "metric": "compact tokens/s, tree-packed linear-attn fwd+bwd; MFMA util % of peak",
        "value": value,
        "unit": "compact tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg["dtype"],
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.config], "C": C, "S": plan.info["S"],
                   "R": plan.info["R"], "rounds": K,
                   "sequences": plan.info["n_seq"], "H": H, "d": d, "chunk": 64},
        "roofline": {"bound": "hbm", "kernel": dom,
                     "achieved": ds["alg_GBs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                     "frac": ds["alg_frac"], "traffic": traffic,
                     "alg_bytes_per_launch": ds["alg_bytes_per_launch"],
                     "avg_launch_ms": ds["avg_ms"]},
        "step_roofline": {"alg_GB": step_bytes / 1e9, "achieved_GBs": step_gbs,
                          "hbm_frac": step_gbs / PEAK_HBM_GBS,
                          "design_GB": sum(dbytes.values()) / 1e9,
                          "design_over_alg": sum(dbytes.values()) / step_bytes},
        "mfma_util_pct": 100.0 * achieved_tflops / peak_tf,
        "ms_median": float(np.median(step_ms)),
        "ms_p10": float(np.percentile(step_ms, 10)),
        "ms_p90": float(np.percentile(step_ms, 90)),
        "plan_ms": plan_s * 1e3,
        "value_with_plan": C / ((ms + plan_s * 1e3) * 1e-3),
        "kernels": kstats,
        "kernel_source_sha": la_source_sha(),
    }
    log("[bench] separate passes")
    passes = pass_times(runner, t, args.steps, args.warmup)
    # per pass: algorithmic bytes and FLOPs (per compact token and head at
    # d = 128: forward 98,304, backward 245,760, state pass 32,768)
    fscale = H * (d / 128) ** 2
    work = {"fwd": (pass_bytes["fwd"], 98304 * fscale),
            "bwd": (pass_bytes["bwd"], 245760 * fscale),
            "fwd_bwd": (pass_bytes["fwd"] + pass_bytes["bwd"], (98304 + 245760) * fscale),
            "recompute_fwd_bwd": (pass_bytes["fwd"] + pass_bytes["state"] + pass_bytes["bwd"],
                                  (98304 + 245760 + 32768) * fscale)}
    out["passes"] = {}
    for k, v in passes.items():
        by, fl = work[k]
        gbs = by / (v * 1e-3) / 1e9
        tfs = C * fl / (v * 1e-3) / 1e12
        out["passes"][k] = {"ms": v, "compact_tok_s": C / (v * 1e-3),
                            "alg_GB": by / 1e9, "alg_GBs": gbs, "hbm_frac": gbs / PEAK_HBM_GBS,
                            "TFLOPs": tfs, "mfma_frac": tfs / peak_tf}
    if not args.no_expanded:
        log("[bench] compact vs expanded (4 trees, ~32k compact tokens)")
        out["compact_vs_expanded"] = expanded_comparison(max(3, args.steps // 2), 2)
    if not args.no_logp:
        log("[bench] compact-to-semantic log-probabilities (157,184-token vocabulary)")
        out["logp"] = logp_measurement(args.steps, args.warmup)
    if not args.no_conv:
        log("[bench] causal convolution with ancestor context (6,144 channels)")
        out["conv"] = conv_measurement(args.steps, args.warmup)
    if not args.no_attn:
        log("[bench] full attention through asymmetric Q/KV views (16 heads of 128)")
        out["attn"] = attn_measurement(args.steps, args.warmup)
    if not args.no_kda:
        log("[bench] KDA over the same plan (16 heads of 128)")
        out["kda"] = kda_measurement(max(2, args.steps // 4), 1)
    if not args.no_mbplan:
        log("[bench] prefix-aware microbatch planning (host)")
        out["mb_plan"] = mbplan_measurement()
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle, trajectory-wise recurrence)")
        out["cpu_baseline"] = cpu_baseline(forest, x, cfg, budget_s=6.0)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
