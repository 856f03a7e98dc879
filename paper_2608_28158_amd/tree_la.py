"""Round driver and autograd wrapper for tree-packed linear attention.

Each execution round is one packed call (Sec. 3.4, "Round-wise execution"):
``harts_la_fwd`` runs the round, reading each sequence's initial state from
the state bank (tree initial states, then the boundary states written by
earlier rounds) through the round's init index; with ``gather_init=True``
the round's initial states are first gathered into a dense buffer by
``harts_state_gather`` instead.  The backward walks the rounds in reverse
(Sec. 3.4, "Differentiable boundary states"): ``harts_la_bwd`` per round,
then the scatter-add adjoint of the gather into the bank gradient, and
finally ``harts_replay_reduce``.  With ``recompute=True`` the forward keeps
only its inputs, the plan and the bank of boundary states the rounds hand
over; each round's backward re-runs that round's state pass from the same
plan inside ``harts_la_bwd`` (saved = NULL), "Full-layer activation
recomputation" of Sec. 3.4.

Python here only marshals arguments and owns torch buffers; every step runs
in libharts.
"""
from __future__ import annotations

import ctypes as C

import torch

from . import _lib
from .plan import HartsPlan


def _ptr(t):
    return C.c_void_p(t.data_ptr()) if t is not None else C.c_void_p(0)


def _dtype_code(dt):
    if dt == torch.float32:
        return _lib.HARTS_F32
    if dt == torch.bfloat16:
        return _lib.HARTS_BF16
    raise TypeError(f"unsupported dtype {dt}")


class TreeLARunner:
    """Forward / backward of one linear-attention layer over a plan."""

    def __init__(self, plan: HartsPlan, H: int, d: int, dtype, device, scale=None,
                 gather_init=False):
        self.plan = plan
        self.gather_init = gather_init
        self.H, self.d = H, d
        self.dtype = dtype
        self.code = _dtype_code(dtype)
        self.device = torch.device(device)
        if self.device.type != "cuda":
            raise RuntimeError("tree-packed linear attention runs on the GPU only")
        if self.device.index is None:
            self.device = torch.device("cuda", torch.cuda.current_device())
        self.scale = float(d ** -0.5 if scale is None else scale)
        self.L = _lib.lib()
        self.blob = plan.blob(self.device)
        self.elems = H * d * d
        sz = C.c_size_t()
        self.saved_bytes, self.ws_fwd, self.ws_fwd_nosave = [], [], []
        self.ws_bwd_saved, self.ws_bwd_rec = [], []
        for r in range(plan.info["n_rounds"]):
            _lib.check(self.L.harts_la_saved_size(plan.handle, r, self.code, H, d, d,
                                                  C.byref(sz)), "harts_la_saved_size")
            self.saved_bytes.append(sz.value)
            _lib.check(self.L.harts_la_workspace_size(plan.handle, r, 0, self.code, H, d, d, 1,
                                                      C.byref(sz)), "harts_la_workspace_size")
            self.ws_fwd.append(sz.value)
            _lib.check(self.L.harts_la_workspace_size(plan.handle, r, 0, self.code, H, d, d, 0,
                                                      C.byref(sz)), "harts_la_workspace_size")
            self.ws_fwd_nosave.append(sz.value)
            _lib.check(self.L.harts_la_workspace_size(plan.handle, r, 1, self.code, H, d, d, 1,
                                                      C.byref(sz)), "harts_la_workspace_size")
            self.ws_bwd_saved.append(sz.value)
            _lib.check(self.L.harts_la_workspace_size(plan.handle, r, 1, self.code, H, d, d, 0,
                                                      C.byref(sz)), "harts_la_workspace_size")
            self.ws_bwd_rec.append(sz.value)

    # -- helpers -------------------------------------------------------------
    def _stream(self):
        return C.c_void_p(torch.cuda.current_stream(self.device).cuda_stream)

    def _bytes(self, n):
        return torch.empty(max(int(n), 16), dtype=torch.uint8, device=self.device)

    def _init_idx(self, r):
        off = self.plan.rounds[r]["init_idx_off"]
        return C.c_void_p(self.blob.data_ptr() + off)

    def gather(self, bank, r):
        n = self.plan.rounds[r]["n_seq"]
        S0 = torch.empty((n, self.H, self.d, self.d), dtype=torch.float32, device=self.device)
        _lib.check(self.L.harts_state_gather(_ptr(bank), self._init_idx(r), n, self.elems,
                                             _ptr(S0), 0, self._stream()), "harts_state_gather")
        return S0

    def scatter_add(self, dS0, dbank, r):
        n = self.plan.rounds[r]["n_seq"]
        _lib.check(self.L.harts_state_gather(_ptr(dS0), self._init_idx(r), n, self.elems,
                                             _ptr(dbank), 1, self._stream()),
                   "harts_state_gather")

    def _check_inputs(self, q, k, v, g):
        Cn = self.plan.info["C"]
        for name, t, last in (("q", q, self.d), ("k", k, self.d), ("v", v, self.d)):
            if t.shape != (Cn, self.H, last) or t.dtype != self.dtype or not t.is_contiguous():
                raise ValueError(f"{name} must be contiguous {self.dtype} [{Cn},{self.H},{last}]")
            if t.device != self.device:
                raise ValueError(f"{name} is on {t.device}, expected {self.device}")
        if g.shape != (Cn, self.H) or g.dtype != torch.float32 or not g.is_contiguous():
            raise ValueError(f"g must be contiguous float32 [{Cn},{self.H}]")

    # -- forward -------------------------------------------------------------
    def forward(self, q, k, v, g, S0_tree=None, outputs=True, keep_states=True, final_states=None):
        """Run all rounds.  Returns dict(o, S_final, bank, saved[r]).  The
        final states are written when final_states is true (default: with
        the outputs)."""
        self._check_inputs(q, k, v, g)
        P = self.plan
        H, d = self.H, self.d
        # the tree-initial states lead the bank; every other slot is written by
        # its producing round before a later round gathers it
        bank = torch.empty((P.info["n_bank"], H, d, d), dtype=torch.float32, device=self.device)
        if S0_tree is not None:
            bank[: P.info["n_trees"]].copy_(S0_tree)
        else:
            bank[: P.info["n_trees"]].zero_()
        o = torch.empty_like(q) if outputs else None
        # the state-only pass (recompute-forward) writes no final states
        if final_states is None:
            final_states = outputs
        S_final = torch.empty((P.info["n_leaves"], H, d, d), dtype=torch.float32,
                              device=self.device) if final_states else None
        saved = []
        for r in range(P.info["n_rounds"]):
            S0 = self.gather(bank, r) if self.gather_init else None
            sv = self._bytes(self.saved_bytes[r]) if keep_states else None
            ws = self._bytes(self.ws_fwd[r] if keep_states else self.ws_fwd_nosave[r])
            _lib.check(self.L.harts_la_fwd(
                P.handle, r, _ptr(self.blob), self.code, H, d, d, self.scale,
                _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(S0), _ptr(o), _ptr(S_final),
                _ptr(bank), _ptr(sv), _ptr(ws), ws.numel(), self._stream()), "harts_la_fwd")
            saved.append(sv)
        return dict(o=o, S_final=S_final, bank=bank, saved=saved)

    # -- backward ------------------------------------------------------------
    def backward(self, q, k, v, g, dO, dS_final, fwd=None, S0_tree=None, recompute=False):
        """Gradients of <dO, o> + <dS_final, S_final>.  ``fwd`` is the dict
        from forward(); its bank holds the boundary states every round starts
        from.  With recompute=True, or when the forward kept no block states
        (keep_states=False), each round's ``harts_la_bwd`` re-runs that
        round's state pass itself (saved = NULL); with fwd None a state-only
        forward first rebuilds the bank."""
        P = self.plan
        H, d = self.H, self.d
        if fwd is None:
            fwd = self.forward(q, k, v, g, S0_tree, outputs=False, keep_states=False)
            recompute = True
        if dO.dtype != self.dtype or not dO.is_contiguous() or dO.shape != q.shape:
            raise ValueError("dO must match o")
        if dS_final is None:
            dS_final = torch.zeros((P.info["n_leaves"], H, d, d), dtype=torch.float32,
                                   device=self.device)
        dS_final = dS_final.contiguous().float()
        dbank = torch.zeros((P.info["n_bank"], H, d, d), dtype=torch.float32, device=self.device)
        dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
        dg = torch.empty_like(g)
        R = P.info["R"]
        rep = torch.empty((max(R, 1), H, 2 * d + 1), dtype=torch.float32, device=self.device)
        # dS0 of every sequence, in sequence (round) order; each round writes its slice
        dS0_seq = torch.empty((P.info["n_seq"], H, d, d), dtype=torch.float32, device=self.device)
        for r in reversed(range(P.info["n_rounds"])):
            n = P.rounds[r]["n_seq"]
            s0 = P.rounds[r]["seq_begin"]
            dS0 = dS0_seq[s0:s0 + n]
            S0 = self.gather(fwd["bank"], r) if self.gather_init else None
            sv = None if recompute else fwd["saved"][r]
            ws = self._bytes(self.ws_bwd_rec[r] if sv is None else self.ws_bwd_saved[r])
            _lib.check(self.L.harts_la_bwd(
                P.handle, r, _ptr(self.blob), self.code, H, d, d, self.scale,
                _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(S0), _ptr(fwd["bank"]), _ptr(dO),
                _ptr(dS_final),
                _ptr(dbank), _ptr(sv), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dg),
                _ptr(rep), _ptr(dS0), _ptr(ws), ws.numel(), self._stream()), "harts_la_bwd")
            self.scatter_add(dS0, dbank, r)
        _lib.check(self.L.harts_replay_reduce(
            P.handle, _ptr(self.blob), self.code, H, d, d, _ptr(rep), _ptr(dk), _ptr(dv),
            _ptr(dg), self._stream()), "harts_replay_reduce")
        return dict(dq=dq, dk=dk, dv=dv, dg=dg, dS0_tree=dbank[: P.info["n_trees"]],
                    dS0_seq=dS0_seq, dbank=dbank)


class _TreeLAFn(torch.autograd.Function):
    @staticmethod
    def forward(ctx, q, k, v, g, S0_tree, runner, recompute):
        res = runner.forward(q, k, v, g, S0_tree, outputs=True, keep_states=not recompute)
        ctx.runner = runner
        ctx.recompute = recompute
        # with recompute the block states are not kept: the backward re-runs
        # each round's state pass from the bank of boundary states
        ctx.fwd = res
        ctx.save_for_backward(q, k, v, g, S0_tree)
        return res["o"], res["S_final"]

    @staticmethod
    def backward(ctx, dO, dS_final):
        q, k, v, g, S0_tree = ctx.saved_tensors
        runner = ctx.runner
        if dO is None:
            dO = torch.zeros_like(q)
        grads = runner.backward(q, k, v, g, dO.contiguous().to(q.dtype), dS_final, fwd=ctx.fwd,
                                S0_tree=S0_tree, recompute=ctx.recompute)
        ctx.fwd = None
        return grads["dq"], grads["dk"], grads["dv"], grads["dg"], grads["dS0_tree"], None, None


def tree_la(q, k, v, g, plan: HartsPlan, S0_tree=None, scale=None, recompute=False):
    """Tree-packed chunkwise linear attention over the plan's physical rows.

    q, k: [C,H,d]; v: [C,H,d] (float32 or bfloat16); g: float32 [C,H];
    S0_tree: optional float32 [n_trees,H,d,d].  Returns (o [C,H,d],
    S_final [n_leaves,H,d,d] float32), differentiable in all inputs."""
    H, d = q.shape[1], q.shape[2]
    runner = TreeLARunner(plan, H, d, q.dtype, q.device, scale)
    if S0_tree is None:
        S0_tree = torch.zeros((plan.info["n_trees"], H, d, d), dtype=torch.float32,
                              device=q.device)
    return _TreeLAFn.apply(q, k, v, g, S0_tree, runner, recompute)
