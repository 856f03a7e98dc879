"""CPU oracle for tree-packed chunkwise linear attention (HARTS, arXiv 2608.28158).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute anything in this package: only ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with
the HIP path (``paper_2608_28158_amd``) and imports nothing from it.

Contents (all float64 unless stated):

* ``forest``      -- positions, anchors a(p) = B*floor(p/B) (eq. resume-anchor),
                     trajectories, multiplicity q_v (eq. multiplicity).
* ``recurrent``   -- the token-by-token scalar-decay recurrence, forward and
                     hand-derived backward, per trajectory and over a forest
                     expanded into all root-to-leaf trajectories.  This is the
                     plain definition the method must reproduce (Sec. 2.2:
                     replay keeps the trajectory-wise chunk partition).
* ``chunkwise``   -- the chunkwise form of the same recurrence (Sec. 2.2,
                     "chunkwise state propagation"), zero-padded chunks.
* ``plan_ref``    -- Algorithm "minimum-call" (Sec. 3.3): the T_pre/T_in
                     dynamic program and Recover, with the ordering
                     conventions the library also follows.
* ``bruteforce``  -- exhaustive search over direct-continuation choices under
                     the execution model of Sec. 3.3, independent of the DP.
* ``compact``     -- execution of plan_ref's rounds with the chunkwise form,
                     boundary-state handoffs (eq. chunkla-interface) and
                     gradients by reverse-mode differentiation of that program.
* ``mbplan``      -- prefix-aware microbatch and data-parallel planning
                     (Sec. 3.2): compact-trie work, natural partition, exact
                     contiguous DP, evolution, trie-aware greedy, refinement,
                     replica/slot assignment and the lexicographic choice.
* ``conv``        -- causal depthwise convolution along every trajectory (the
                     true-ancestor context of Sec. 4.2) and its gradients.
* ``attn``        -- causal softmax attention along every trajectory, and one
                     branch through asymmetric Q/KV views with bottom-right
                     alignment (Sec. 4.2).
* ``logprob``     -- compact-to-semantic log-probabilities and their gradient
                     (eqs. mapped-logp, mapped-logp-grad), one log-softmax
                     per semantic position.
* ``kda``         -- KDA, per-channel decay with the delta rule (Sec. 2.2):
                     the token recurrence, the chunk form of eq. chunk-state,
                     and trajectory-wise execution over a forest with
                     gradients by reverse mode.

Recurrence reading used by every module but ``kda`` (the paper prints only
KDA's chunk update, eq. chunk-state): S_t = exp(g_t) S_{t-1} + k_t v_t^T and o_t = scale S_t^T q_t,
with per-head scalar log-decay g_t and state S of shape [d_k, d_v].
"""
