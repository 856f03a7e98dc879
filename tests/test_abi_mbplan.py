"""harts_mb_plan (Sec. 3.2) on the CPU: the library's prefix-aware
microbatch/DP plan equals the oracle's -- the same K, J, microbatch of every
trajectory, replica and slot of every microbatch -- in exact-search mode and
in the heuristic mode (evolution of the natural partition and refinement of
anchors), and its guarantees hold on a larger batch."""
import ctypes as C

import numpy as np
import pytest

from oracle.mbplan import plan_microbatches, trie_nodes
from tests.test_oracle_mbplan import random_trajs


def lib_plan(trajs, D, T, exact_max=0):
    from paper_2608_28158_amd import _lib
    L = _lib.lib()
    N = len(trajs)
    off = np.zeros(N + 1, np.int64)
    off[1:] = np.cumsum([len(t) for t in trajs])
    tok = np.concatenate([np.asarray(t, np.int32) for t in trajs]).astype(np.int32)
    group = np.zeros(N, np.int32)
    rep = np.zeros(N, np.int32)
    slot = np.zeros(N, np.int32)
    work = np.zeros(N, np.int64)
    res = _lib.MbResult()
    rc = L.harts_mb_plan(N, off.ctypes.data, tok.ctypes.data, D, T, exact_max, group.ctypes.data,
                         rep.ctypes.data, slot.ctypes.data, work.ctypes.data, C.byref(res))
    return rc, res, group, rep[:res.K], slot[:res.K], work[:res.K]


def same_plan(trajs, D, T, exact_max=0):
    from paper_2608_28158_amd import _lib
    rc, res, group, rep, slot, work = lib_plan(trajs, D, T, exact_max)
    assert rc == _lib.HARTS_OK, _lib.last_error()
    ref = plan_microbatches(trajs, D, T, n0=exact_max or 512)
    assert res.K == ref["K"]
    assert (res.work_total, res.slot_critical, res.replica_max) == ref["J"]
    assert list(group) == ref["group"]
    assert list(rep) == ref["replica"] and list(slot) == ref["slot"]
    for gi, ms in enumerate(ref["members"]):
        assert work[gi] == trie_nodes([trajs[i] for i in ms])
    return res


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("D", [1, 2, 4])
def test_exact_mode_matches_oracle(seed, D):
    r = np.random.default_rng(300 + seed)
    trajs = random_trajs(r, int(r.integers(D, 18)), max_tail=8)
    T = max(len(t) for t in trajs) + int(r.integers(0, 24))
    same_plan(trajs, D, T)


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("D", [1, 2])
def test_heuristic_mode_matches_oracle(seed, D):
    r = np.random.default_rng(400 + seed)
    trajs = random_trajs(r, int(r.integers(10, 40)), max_tail=10)
    T = max(len(t) for t in trajs) + int(r.integers(0, 16))
    same_plan(trajs, D, T, exact_max=6)


def test_many_samples_of_K_match_oracle():
    """A capacity so small that the K range exceeds the 32 sampled values."""
    r = np.random.default_rng(7)
    trajs = random_trajs(r, 80, vocab=6, max_tail=5)
    T = max(len(t) for t in trajs)
    res = same_plan(trajs, 1, T, exact_max=10)
    assert res.natural_K > 32


def test_rejects_infeasible_inputs():
    from paper_2608_28158_amd import _lib
    assert lib_plan([[1, 2, 3]], 1, 2)[0] == _lib.HARTS_EINVAL      # above capacity
    assert lib_plan([[1], [2]], 4, 10)[0] == _lib.HARTS_EINVAL      # N < D
    assert lib_plan([[1], [2]], 0, 10)[0] == _lib.HARTS_EINVAL
