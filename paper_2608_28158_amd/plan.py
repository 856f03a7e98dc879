"""Python view of a ``harts_plan`` (Algorithm "minimum-call", Sec. 3.3).

``HartsPlan`` owns the library plan, exposes its arrays as numpy (host) and
uploads the device descriptor image once (step "round descriptors to the
device").  No planning happens in Python.
"""
from __future__ import annotations

import ctypes as C

import numpy as np

from . import _lib


class HartsPlan:
    def __init__(self, parent, seg_len, chunk: int = 64, heads: int = 16, min_blocks: int = 0):
        """Plan a forest (``harts_plan``) and cut its rounds into device
        work blocks for ``heads`` heads (``harts_plan_set_blocks``; a
        non-zero ``min_blocks`` overrides the head-count rule)."""
        L = _lib.lib()
        parent = np.ascontiguousarray(parent, dtype=np.int32)
        seg_len = np.ascontiguousarray(seg_len, dtype=np.int64)
        if parent.shape != seg_len.shape or parent.ndim != 1:
            raise ValueError("parent and seg_len must be 1-D of equal length")
        h = C.c_void_p()
        _lib.check(L.harts_plan(int(parent.shape[0]),
                                parent.ctypes.data_as(_lib._I32),
                                seg_len.ctypes.data_as(_lib._I64),
                                int(chunk), C.byref(h)), "harts_plan")
        self._h = h
        self._L = L
        _lib.check(L.harts_plan_set_blocks(h, int(heads), int(min_blocks)),
                   "harts_plan_set_blocks")
        info = _lib.PlanInfo()
        _lib.check(L.harts_plan_get_info(h, C.byref(info)), "harts_plan_get_info")
        self.info = {n: getattr(info, n) for n, _ in _lib.PlanInfo._fields_}
        self.arrays = self._export()
        self.rounds = []
        for r in range(self.info["n_rounds"]):
            ri = _lib.RoundInfo()
            _lib.check(L.harts_plan_round_info(h, r, C.byref(ri)),
                       "harts_plan_round_info")
            self.rounds.append({n: getattr(ri, n) for n, _ in _lib.RoundInfo._fields_})
        self.blob_host = np.zeros(self.info["blob_bytes"] // 4, np.int32)
        _lib.check(L.harts_plan_blob(h, self.blob_host.ctypes.data,
                                     self.blob_host.nbytes), "harts_plan_blob")
        self._blob_dev = {}

    def _export(self):
        sizes = dict(self.info)
        sizes["n_rounds+1"] = self.info["n_rounds"] + 1
        sizes["n_seq+1"] = self.info["n_seq"] + 1
        out = {}
        st = _lib.PlanArrays()
        for name, ptr_t, dt, key in _lib.PLAN_ARRAY_FIELDS:
            arr = np.zeros(max(int(sizes[key]), 0), dtype=dt)
            out[name] = arr
            setattr(st, name, arr.ctypes.data_as(ptr_t) if arr.size else None)
        _lib.check(self._L.harts_plan_export(self._h, C.byref(st)),
                   "harts_plan_export")
        return out

    @property
    def handle(self):
        return self._h

    def __getitem__(self, key):
        if key in self.arrays:
            return self.arrays[key]
        return self.info[key]

    def blob(self, device):
        """Device copy of the descriptor image (uploaded once per device)."""
        import torch
        key = str(device)
        if key not in self._blob_dev:
            self._blob_dev[key] = torch.from_numpy(self.blob_host).to(device)
        return self._blob_dev[key]

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            self._L.harts_plan_free(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
