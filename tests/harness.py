"""Shared helpers for the parity tests: seeded inputs in the canonical
layout, the canonical <-> physical row map of a plan, the oracle run and the
tolerance metric (max |x - ref| / max |ref| per tensor, ref in float64)."""
from __future__ import annotations

import numpy as np

from workloads import config_inputs  # noqa: F401

TOL = {"f32": 1e-4, "bf16": 2e-2}

# (label, dtype, {tensor: max-rel error}) of every GPU comparison run in this
# session; printed by the terminal summary hook in conftest.py.
MARGINS = []


def record(label, dtype, errs):
    MARGINS.append((label, dtype, dict(errs)))


def max_rel(x, ref):
    x = np.asarray(x, np.float64)
    ref = np.asarray(ref, np.float64)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(x - ref)) / (den if den > 0 else 1.0))


def phys_index(seg_len, seg_row):
    """phys[c] = physical row of canonical row c (segments in id order)."""
    seg_len = np.asarray(seg_len, np.int64)
    row0 = np.concatenate([[0], np.cumsum(seg_len)[:-1]])
    phys = np.empty(int(seg_len.sum()), np.int64)
    for v in range(len(seg_len)):
        phys[row0[v]:row0[v] + seg_len[v]] = seg_row[v] + np.arange(seg_len[v])
    return phys


