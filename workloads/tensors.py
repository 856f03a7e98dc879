"""Seeded input tensors for one linear-attention layer over a forest.

Rows are in the canonical compact layout: segments in id order, tokens in
order within a segment.  Draw order after the forest: q, k, v, g, dO, dS_final
(then the optional per-tree initial state).  q and k are L2-normalised over
the head dimension in float32; bf16 workloads round q, k, v and dO to bf16
(round-to-nearest-even) and every consumer reads the rounded values.
"""
from __future__ import annotations

import numpy as np


def to_bf16_roundtrip(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even), kept as f32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).reshape(x.shape)


def _l2n(x):
    n = np.sqrt(np.sum(x * x, axis=-1, keepdims=True, dtype=np.float32))
    return (x / n).astype(np.float32)


def draw_inputs(n_rows: int, n_leaves: int, H: int, dk: int, dv: int, rng,
                dtype: str = "f32", n_trees: int = 0, s0_scale: float = 0.0,
                g_range=(-0.1, -0.001)):
    """q, k ~ N(0,1) then L2-normalised; v, dO, dS_final ~ N(0,1);
    g ~ U[g_range] per (token, head).  Returns a dict of float32 arrays."""
    f32 = np.float32
    q = _l2n(rng.standard_normal((n_rows, H, dk), dtype=f32))
    k = _l2n(rng.standard_normal((n_rows, H, dk), dtype=f32))
    v = rng.standard_normal((n_rows, H, dv), dtype=f32)
    g = rng.uniform(g_range[0], g_range[1], size=(n_rows, H)).astype(f32)
    dO = rng.standard_normal((n_rows, H, dv), dtype=f32)
    dS_final = rng.standard_normal((n_leaves, H, dk, dv), dtype=f32)
    if n_trees and s0_scale:
        S0 = (rng.standard_normal((n_trees, H, dk, dv), dtype=f32)
              * f32(s0_scale))
    else:
        S0 = np.zeros((max(n_trees, 0), H, dk, dv), f32)
    if dtype == "bf16":
        q, k, v, dO = (to_bf16_roundtrip(t) for t in (q, k, v, dO))
    elif dtype != "f32":
        raise ValueError(dtype)
    return dict(q=q, k=k, v=v, g=g, dO=dO, dS_final=dS_final, S0=S0)


def config_inputs(idx, s0_scale=0.0):
    """Forest, workload table entry and inputs of configuration ``idx``."""
    from .trees import forest_for_config
    forest, rng, cfg = forest_for_config(idx)
    n_leaves = len(forest.leaves())
    n_trees = int(np.sum(forest.parent < 0))
    x = draw_inputs(forest.n_rows, n_leaves, cfg["H"], cfg["d"], cfg["d"], rng,
                    dtype=cfg["dtype"], n_trees=n_trees, s0_scale=s0_scale)
    return forest, cfg, x
