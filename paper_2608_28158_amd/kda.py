"""KDA over a plan (Sec. 2.2, eq. chunk-state; handoffs of Sec. 3.4): argument
marshalling around the harts_kda_* entry points of libharts.so.  Every step
of the forward and backward runs in the library's kernels; this module only
builds the host tables once per plan, orders the rounds and hands device
pointers over.

    run = KdaRunner(plan, H, d, dtype)
    o, S_final = run.forward(q, k, v, g, beta, S0_tree, scale)
    grads = run.backward(dO, dS_final)          # uses the forward's workspace

q, k, v, o: [C, H, d] in the plan's physical row order (bf16 or float32);
g: [C, H, d] float32 log-decays; beta: [C, H] float32; S0_tree:
[n_trees, H, d, d] float32.
"""
from __future__ import annotations

import ctypes as C
import time

import numpy as np
import torch

from . import _lib


def _p(t):
    return C.c_void_p(t.data_ptr()) if t is not None else None


class KdaRunner:
    def __init__(self, plan, H: int, d: int, dtype=torch.bfloat16, device="cuda"):
        L = _lib.lib()
        self.L, self.plan, self.H, self.d, self.dtype, self.device = L, plan, H, d, dtype, device
        self.code = _lib.HARTS_BF16 if dtype == torch.bfloat16 else _lib.HARTS_F32
        sz = _lib.KdaSizes()
        _lib.check(L.harts_kda_layout(plan.handle, C.byref(sz)), "harts_kda_layout")
        self.sizes = sz
        self.chunk_rows = np.zeros(max(sz.n_chunks, 1) * 64, np.int32)
        self.seq_tab = np.zeros((sz.n_seq, 8), np.int32)
        self.req_tab = np.zeros((max(sz.n_req, 1), 2), np.int32)
        self.group_tab = np.zeros((max(sz.n_groups, 1), 4), np.int32)
        self.group_seq = np.zeros(max(sz.n_seq, 1), np.int32)
        self.pos_slot = np.zeros(max(sz.n_chunks, 1) * 64, np.int32)
        self.multi_row = np.zeros(max(sz.n_multi, 1), np.int32)
        self.multi_off = np.zeros(sz.n_multi + 1, np.int64)
        t0 = time.perf_counter()
        _lib.check(L.harts_kda_tables(plan.handle, self.chunk_rows.ctypes.data, self.seq_tab.ctypes.data,
                                      self.req_tab.ctypes.data, self.group_tab.ctypes.data,
                                      self.group_seq.ctypes.data, self.pos_slot.ctypes.data,
                                      self.multi_row.ctypes.data, self.multi_off.ctypes.data), "harts_kda_tables")
        self.tables_ms = (time.perf_counter() - t0) * 1e3   # host tables alone
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
        self.d_rows, self.d_seq, self.d_req = dev(self.chunk_rows), dev(self.seq_tab), dev(self.req_tab)
        self.d_group, self.d_gseq = dev(self.group_tab), dev(self.group_seq)
        self.d_slot, self.d_mrow, self.d_moff = dev(self.pos_slot), dev(self.multi_row), dev(self.multi_off)
        # per round: sequences [s0, s1), chunks [c0, c1), groups [g0, g1)
        self.rounds = []
        for r in range(sz.n_rounds):
            seqs = np.nonzero(self.seq_tab[:, 0] == r)[0]
            grp = np.nonzero(self.group_tab[:sz.n_groups, 0] == r)[0]
            s0, s1 = int(seqs[0]), int(seqs[-1]) + 1
            c0 = int(self.seq_tab[s0, 1])
            c1 = int(self.seq_tab[s1 - 1, 1] + self.seq_tab[s1 - 1, 2])
            self.rounds.append((s0, s1, c0, c1, int(grp[0]), int(grp[-1]) + 1))
        nb = C.c_size_t()
        _lib.check(L.harts_kda_workspace_size(sz.n_chunks, H, d, C.byref(nb)), "harts_kda_workspace_size")
        self.ws = torch.empty(max(nb.value // 4, 1), dtype=torch.float32, device=device)
        self.n_bank = plan["n_bank"]
        self.n_trees = plan["n_trees"]
        self.n_leaves = plan["n_leaves"]
        self._saved = None

    def _stream(self):
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)

    def forward(self, q, k, v, g, beta, S0_tree, scale, outputs=True):
        H, d = self.H, self.d
        bank = torch.zeros((self.n_bank, H, d, d), dtype=torch.float32, device=self.device)
        bank[:self.n_trees] = S0_tree
        S_final = torch.empty((self.n_leaves, H, d, d), dtype=torch.float32, device=self.device)
        o = torch.empty_like(q) if outputs else None
        st = self._stream()
        for s0, s1, c0, c1, _, _ in self.rounds:
            _lib.check(self.L.harts_kda_fwd(_p(self.d_rows), _p(self.d_seq), _p(self.d_req), c0, c1 - c0, s0,
                                            s1 - s0, self.code, H, d, C.c_float(scale), _p(q), _p(k), _p(v),
                                            _p(g), _p(beta), _p(bank), _p(S_final), _p(o), _p(self.ws), st),
                       "harts_kda_fwd")
        self._saved = (q, k, v, g, beta, scale)
        return o, S_final

    def backward(self, dO, dS_final=None):
        if self._saved is None:
            raise RuntimeError("KdaRunner.backward needs the forward of the same inputs first")
        q, k, v, g, beta, scale = self._saved
        H, d, sz = self.H, self.d, self.sizes
        dbank = torch.zeros((self.n_bank, H, d, d), dtype=torch.float32, device=self.device)
        dS0_seq = torch.empty((sz.n_seq, H, d, d), dtype=torch.float32, device=self.device)
        Cn = self.plan["C"]
        out = {n: torch.empty((Cn, H, d), dtype=self.dtype, device=self.device) for n in ("dq", "dk", "dv")}
        out["dg"] = torch.empty((Cn, H, d), dtype=torch.float32, device=self.device)
        out["dbeta"] = torch.empty((Cn, H), dtype=torch.float32, device=self.device)
        # float32 partials of the compact rows that are also replayed: one slot per packed row
        ns = max(sz.n_slots, 1)
        slots = {n: torch.empty((ns, H, d), dtype=torch.float32, device=self.device) for n in ("dq", "dk", "dv", "dg")}
        slots["dbeta"] = torch.empty((ns, H), dtype=torch.float32, device=self.device)
        names = ("dq", "dk", "dv", "dg", "dbeta")
        st = self._stream()
        for s0, s1, c0, c1, g0, g1 in reversed(self.rounds):
            _lib.check(self.L.harts_kda_bwd(_p(self.d_rows), _p(self.d_seq), _p(self.d_req), _p(self.d_slot), c0,
                                            c1 - c0, s0, s1 - s0, self.code, H, d, C.c_float(scale), _p(q), _p(k),
                                            _p(v), _p(g), _p(beta), _p(dO), _p(dS_final), _p(dbank), _p(dS0_seq),
                                            _p(self.ws), *(_p(out[n]) for n in names),
                                            *(_p(slots[n]) for n in names), st), "harts_kda_bwd")
            _lib.check(self.L.harts_kda_bank_add(_p(self.d_group), g0, g1 - g0, _p(self.d_gseq), H * d * d,
                                                 _p(dS0_seq), _p(dbank), st), "harts_kda_bank_add")
        for n in names:
            width = H if n == "dbeta" else H * d
            code = _lib.HARTS_BF16 if out[n].dtype == torch.bfloat16 else _lib.HARTS_F32
            _lib.check(self.L.harts_kda_reduce(_p(slots[n]), _p(self.d_mrow), _p(self.d_moff), sz.n_multi, width,
                                               code, _p(out[n]), st), "harts_kda_reduce")
        out["dS0_tree"] = dbank[:self.n_trees]
        return out
