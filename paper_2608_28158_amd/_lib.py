"""ctypes binding of libharts (declarations in include/harts.h).

Argument marshalling only: every step of the path runs in the library.  The
library is built in-tree by ``paper_2608_28158_amd.build`` and loaded from
this package directory; a missing library is an error, never a fallback.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("HARTS_LIB", os.path.join(HERE, "libharts.so"))

HARTS_OK, HARTS_EINVAL, HARTS_EUNSUPPORTED, HARTS_EHIP, HARTS_ENOMEM = 0, -1, -2, -3, -4
HARTS_F32, HARTS_BF16 = 0, 1

# Every symbol include/harts.h declares.
EXPORTS = (
    "harts_last_error", "harts_plan", "harts_plan_free", "harts_plan_get_info",
    "harts_plan_export", "harts_plan_set_blocks", "harts_plan_round_info", "harts_plan_blob",
    "harts_la_fwd", "harts_la_fwd_noalloc", "harts_la_bwd", "harts_la_workspace_size",
    "harts_la_saved_size", "harts_state_gather", "harts_replay_reduce",
    "harts_semantic_map", "harts_logp_fwd", "harts_logp_bwd", "harts_mb_plan",
    "harts_conv_context", "harts_conv_workspace_size", "harts_conv_fwd", "harts_conv_bwd",
    "harts_attn_layout", "harts_attn_views", "harts_attn_gather", "harts_attn_fwd",
    "harts_attn_bwd", "harts_attn_scatter",
    "harts_kda_layout", "harts_kda_tables", "harts_kda_workspace_size", "harts_kda_fwd", "harts_kda_bwd",
    "harts_kda_bank_add", "harts_kda_reduce",
    "harts_profile_begin", "harts_profile_end",
)


class PlanInfo(C.Structure):
    _fields_ = [(n, C.c_int32) for n in (
        "n_seg", "n_trees", "n_leaves", "n_rounds", "n_seq", "n_slots",
        "n_bank", "chunk")] + [(n, C.c_int64) for n in (
        "C", "S", "R", "n_req", "n_chunks", "blob_bytes")]


_I64, _I32 = C.POINTER(C.c_int64), C.POINTER(C.c_int32)
# (name, ctype pointer, numpy dtype, size key) -- order as in the header
PLAN_ARRAY_FIELDS = (
    ("seg_start", _I64, np.int64, "n_seg"),
    ("seg_end", _I64, np.int64, "n_seg"),
    ("seg_row", _I64, np.int64, "n_seg"),
    ("seg_seq", _I32, np.int32, "n_seg"),
    ("seg_mult", _I64, np.int64, "n_seg"),
    ("seg_tpre", _I32, np.int32, "n_seg"),
    ("seg_tin", _I32, np.int32, "n_seg"),
    ("seg_tree", _I32, np.int32, "n_seg"),
    ("leaf_seg", _I32, np.int32, "n_leaves"),
    ("tree_calls", _I32, np.int32, "n_trees"),
    ("round_seq_off", _I32, np.int32, "n_rounds+1"),
    ("seq_round", _I32, np.int32, "n_seq"),
    ("seq_tree", _I32, np.int32, "n_seq"),
    ("seq_first_seg", _I32, np.int32, "n_seq"),
    ("seq_final_leaf", _I32, np.int32, "n_seq"),
    ("seq_init_bank", _I32, np.int32, "n_seq"),
    ("seq_anchor", _I64, np.int64, "n_seq"),
    ("seq_n_replay", _I64, np.int64, "n_seq"),
    ("seq_replay_off", _I64, np.int64, "n_seq+1"),
    ("seq_row", _I64, np.int64, "n_seq"),
    ("seq_n_own", _I64, np.int64, "n_seq"),
    ("seq_chain_off", _I32, np.int32, "n_seq+1"),
    ("chain_seg", _I32, np.int32, "n_seg"),
    ("seq_req_off", _I32, np.int32, "n_seq+1"),
    ("req_chunk", _I32, np.int32, "n_req"),
    ("req_bank", _I32, np.int32, "n_req"),
    ("slot_seq", _I32, np.int32, "n_slots"),
    ("slot_pos", _I64, np.int64, "n_slots"),
    ("replay_row", _I64, np.int64, "R"),
)


class PlanArrays(C.Structure):
    _fields_ = [(n, t) for n, t, _, _ in PLAN_ARRAY_FIELDS]


class RoundInfo(C.Structure):
    _fields_ = [("n_seq", C.c_int32), ("seq_begin", C.c_int32), ("n_blk", C.c_int32),
                ("block_chunks", C.c_int32)] + [
        (n, C.c_int64) for n in ("n_chunks", "n_rows", "n_own", "n_replay",
                                 "own_row_begin", "init_idx_off", "seq_tab_off",
                                 "blk_tab_off", "launch_off")]


class MbResult(C.Structure):
    _fields_ = [("K", C.c_int32), ("natural_K", C.c_int32), ("work_total", C.c_int64),
                ("slot_critical", C.c_int64), ("replica_max", C.c_int64),
                ("trie_work", C.c_int64)]


class AttnLayout(C.Structure):
    _fields_ = [(n, C.c_int64) for n in ("n_views", "n_kv", "n_qtiles", "n_kvtiles")]


class KdaSizes(C.Structure):
    _fields_ = [("n_chunks", C.c_int64), ("n_slots", C.c_int64)] + \
        [(n, C.c_int32) for n in ("n_seq", "n_rounds", "n_groups", "n_req", "n_multi", "pad")]


class KernelTime(C.Structure):
    _fields_ = [("name", C.c_char * 48), ("launches", C.c_int32), ("total_ms", C.c_double)]


class HartsError(RuntimeError):
    def __init__(self, code, where, msg):
        super().__init__(f"{where} failed ({code}): {msg}")
        self.code = code


_lib = None


def lib():
    """Load libharts.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"libharts.so not found at {LIB_PATH}; build it with "
            "`python -c 'import __graft_entry__ as g; g.build()'`")
    L = C.CDLL(LIB_PATH)
    vp, sz, i32, i64, f32 = C.c_void_p, C.c_size_t, C.c_int32, C.c_int64, C.c_float
    fp = C.POINTER(C.c_float)
    L.harts_last_error.restype = C.c_char_p
    L.harts_last_error.argtypes = []
    L.harts_plan.restype = C.c_int
    L.harts_plan.argtypes = [i32, _I32, _I64, i32, C.POINTER(vp)]
    L.harts_plan_free.restype = None
    L.harts_plan_free.argtypes = [vp]
    L.harts_plan_get_info.restype = C.c_int
    L.harts_plan_get_info.argtypes = [vp, C.POINTER(PlanInfo)]
    L.harts_plan_export.restype = C.c_int
    L.harts_plan_export.argtypes = [vp, C.POINTER(PlanArrays)]
    L.harts_plan_set_blocks.restype = C.c_int
    L.harts_plan_set_blocks.argtypes = [vp, i32, i32]
    L.harts_plan_round_info.restype = C.c_int
    L.harts_plan_round_info.argtypes = [vp, i32, C.POINTER(RoundInfo)]
    L.harts_plan_blob.restype = C.c_int
    L.harts_plan_blob.argtypes = [vp, vp, sz]
    L.harts_la_fwd.restype = C.c_int
    L.harts_la_fwd.argtypes = [vp, i32, vp, i32, i32, i32, i32, f32,
                               vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.harts_la_fwd_noalloc.restype = C.c_int
    L.harts_la_fwd_noalloc.argtypes = [vp, i32, vp, i32, i32, i32, i32, f32,
                                       vp, vp, vp, vp, vp, vp, vp, vp, vp]
    L.harts_la_bwd.restype = C.c_int
    L.harts_la_bwd.argtypes = [vp, i32, vp, i32, i32, i32, i32, f32,
                               vp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                               vp, vp, vp, vp, vp, vp, vp, sz, vp]
    L.harts_la_workspace_size.restype = C.c_int
    L.harts_la_workspace_size.argtypes = [vp, i32, i32, i32, i32, i32, i32, i32,
                                          C.POINTER(sz)]
    L.harts_la_saved_size.restype = C.c_int
    L.harts_la_saved_size.argtypes = [vp, i32, i32, i32, i32, i32, C.POINTER(sz)]
    L.harts_state_gather.restype = C.c_int
    L.harts_state_gather.argtypes = [vp, vp, i32, i64, vp, i32, vp]
    L.harts_replay_reduce.restype = C.c_int
    L.harts_replay_reduce.argtypes = [vp, vp, i32, i32, i32, i32, vp, vp, vp,
                                      vp, vp]
    L.harts_semantic_map.restype = C.c_int
    L.harts_semantic_map.argtypes = [vp, vp, i64, vp, vp, vp, vp]
    L.harts_logp_fwd.restype = C.c_int
    L.harts_logp_fwd.argtypes = [i32, i64, i64, vp, i64, vp, vp, vp, vp, vp]
    L.harts_logp_bwd.restype = C.c_int
    L.harts_logp_bwd.argtypes = [i32, i64, i64, vp, vp, i64, vp, vp, vp, vp, vp, vp, vp]
    L.harts_mb_plan.restype = C.c_int
    L.harts_mb_plan.argtypes = [i32, vp, vp, i32, i64, i32, vp, vp, vp, vp, C.POINTER(MbResult)]
    L.harts_conv_context.restype = C.c_int
    L.harts_conv_context.argtypes = [vp, i32, vp, vp, vp]
    L.harts_conv_workspace_size.restype = C.c_int
    L.harts_conv_workspace_size.argtypes = [i64, i32, i32, C.POINTER(sz)]
    L.harts_conv_fwd.restype = C.c_int
    L.harts_conv_fwd.argtypes = [i32, i64, i32, i32, vp, vp, vp, vp, vp]
    L.harts_conv_bwd.restype = C.c_int
    L.harts_conv_bwd.argtypes = [i32, i64, i32, i32, vp, vp, vp, vp, vp, i64, vp, vp, vp, vp, sz, vp]
    L.harts_attn_layout.restype = C.c_int
    L.harts_attn_layout.argtypes = [vp, C.POINTER(AttnLayout)]
    L.harts_attn_views.restype = C.c_int
    L.harts_attn_views.argtypes = [vp, vp, vp, vp, vp, vp, vp]
    L.harts_attn_gather.restype = C.c_int
    L.harts_attn_gather.argtypes = [vp, vp, i64, i64, i32, i32, vp, vp]
    L.harts_attn_fwd.restype = C.c_int
    L.harts_attn_fwd.argtypes = [vp, vp, i64, i32, i32, f32, vp, vp, vp, vp, vp, vp]
    L.harts_attn_bwd.restype = C.c_int
    L.harts_attn_bwd.argtypes = [vp, vp, i64, vp, i64, i64, i32, i32, f32, vp, vp, vp, vp, vp, vp,
                                 vp, vp, vp, vp, vp]
    L.harts_attn_scatter.restype = C.c_int
    L.harts_attn_scatter.argtypes = [vp, vp, vp, i64, i64, i32, i32, vp, vp]
    L.harts_kda_layout.restype = C.c_int
    L.harts_kda_layout.argtypes = [vp, vp]
    L.harts_kda_tables.restype = C.c_int
    L.harts_kda_tables.argtypes = [vp] * 9
    L.harts_kda_workspace_size.restype = C.c_int
    L.harts_kda_workspace_size.argtypes = [i64, i32, i32, vp]
    L.harts_kda_fwd.restype = C.c_int
    L.harts_kda_fwd.argtypes = [vp, vp, vp, i64, i64, i32, i32, i32, i32, i32, C.c_float] + [vp] * 10
    L.harts_kda_bwd.restype = C.c_int
    L.harts_kda_bwd.argtypes = [vp, vp, vp, vp, i64, i64, i32, i32, i32, i32, i32, C.c_float] + [vp] * 21
    L.harts_kda_bank_add.restype = C.c_int
    L.harts_kda_bank_add.argtypes = [vp, i32, i32, vp, i64, vp, vp, vp]
    L.harts_kda_reduce.restype = C.c_int
    L.harts_kda_reduce.argtypes = [vp, vp, vp, i64, i64, i32, vp, vp]
    L.harts_profile_begin.restype = C.c_int
    L.harts_profile_begin.argtypes = []
    L.harts_profile_end.restype = C.c_int
    L.harts_profile_end.argtypes = [C.POINTER(KernelTime), i32, C.POINTER(i32)]
    _lib = L
    return L


def profile_begin():
    check(lib().harts_profile_begin(), "harts_profile_begin")


def profile_end():
    """Per-kernel (launches, total ms) since profile_begin, from HIP events."""
    L = lib()
    n = C.c_int32()
    arr = (KernelTime * 64)()
    check(L.harts_profile_end(arr, 64, C.byref(n)), "harts_profile_end")
    return {arr[i].name.decode(): (arr[i].launches, arr[i].total_ms)
            for i in range(min(n.value, 64))}


def check(code, where):
    if code != HARTS_OK:
        msg = lib().harts_last_error().decode(errors="replace")
        raise HartsError(code, where, msg)


def last_error() -> str:
    return lib().harts_last_error().decode(errors="replace")
