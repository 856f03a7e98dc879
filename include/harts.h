/*
 * harts.h -- C ABI of libharts: tree-packed chunkwise linear attention with
 * per-head scalar decay over prefix-compressed rollout trees, for one
 * MI355X (gfx950) GPU.
 *
 * Method: HARTS (arXiv 2608.28158).  The planner is the paper's Algorithm
 * "minimum-call" (Sec. 3.3); the device calls implement the selective
 * chunk-state contract of eq. chunkla-interface (Sec. 3.4): one packed call
 * per execution round, each sequence starting from its own initial state,
 * replaying the bounded interval between its resume anchor (eq.
 * resume-anchor) and its fork, writing outputs only for its own rows,
 * returning its final state and the chunk-boundary states later rounds
 * request; the backward carries gradients through those handoffs.
 *
 * Recurrence (per head, state S of shape [dk, dv]):
 *     S_t = exp(g_t) S_{t-1} + k_t v_t^T,      o_t = scale * S_t^T q_t.
 *
 * Conventions shared by every call
 *   - Return value: HARTS_OK (0) or a negative HARTS_E* code; the message of
 *     the last failure on the calling thread is returned by harts_last_error().
 *     Arguments are validated on the host before anything is enqueued: on a
 *     validation error nothing touches the device.
 *   - Device calls are asynchronous on the given stream (a hipStream_t passed
 *     as void*, NULL = the default stream) and never synchronise the host.
 *     Round-to-round dependencies are carried by stream order.
 *   - The library never allocates device memory.  The caller owns every
 *     device buffer; scratch space is passed as (ws, ws_bytes) sized by the
 *     *_workspace_size queries.  Plans are library-owned host objects.  The
 *     one exception is harts_la_fwd_noalloc's fixed scratch array, part of
 *     the library's device image.
 *   - Row layout: token-major [rows, H, d] in the plan's physical row order
 *     (sequences in id order, each sequence's own segments contiguous).
 *     q, k: [C, H, dk]; v, o: [C, H, dv]; g, dg: float32 [C, H].
 *     States: float32 [., H, dk, dv], dv fastest.  Pointers 16-byte aligned.
 *   - dtype: HARTS_F32 (q, k, v, o, dO and gradients float32) or HARTS_BF16
 *     (those tensors bfloat16; g, states and their gradients always float32).
 *   - Supported head shapes: dk = dv in {64, 128} for bf16, 64 for float32;
 *     chunk size 64; fewer than 2^29 packed rows (C + R) per plan.  Anything
 *     else returns HARTS_EUNSUPPORTED.
 */
#ifndef HARTS_H_
#define HARTS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  HARTS_OK = 0,
  HARTS_EINVAL = -1,       /* malformed argument (forest, sizes, pointers) */
  HARTS_EUNSUPPORTED = -2, /* valid but not implemented (dtype, head dims)  */
  HARTS_EHIP = -3,         /* a HIP runtime call or launch failed           */
  HARTS_ENOMEM = -4        /* host allocation failed, or a buffer too small */
};

enum { HARTS_F32 = 0, HARTS_BF16 = 1 };

/* Opaque plan (host memory, owned by the library). */
typedef struct harts_plan_s harts_plan_t;

/* Thread-local message describing the last failure ("" if none). */
const char* harts_last_error(void);

/* ------------------------------------------------------------------------
 * harts_plan -- minimum-call planning and plan recovery (Sec. 3.3,
 * Algorithm "minimum-call"; eqs. leaf-calls, tin, tpre, early-start,
 * mandatory-replay).
 *
 *   n_seg    number of segments (fork-free token runs), >= 1.
 *   parent   [n_seg] parent segment id, -1 for a root.  Several roots make a
 *            forest (one microbatch); trees are ordered by root id and each
 *            tree has its own chunk grid starting at position 0.  Children
 *            are ordered by ascending id (the "fixed child order").
 *   seg_len  [n_seg] tokens per segment, each > 0.
 *   chunk    execution chunk size B >= 1 (the device calls require 64).
 *   out      receives the plan; release it with harts_plan_free.
 *
 * Linear time and space in n_seg + replay length.  Errors: HARTS_EINVAL for
 * a null pointer, n_seg < 1, chunk < 1, a parent id out of range or equal to
 * the segment, a cycle, a length <= 0, or totals beyond int32 row indexing.
 *
 * Ordering conventions (the paper leaves them open): sequences are created
 * in Recover's order -- the direct continuation is recursed into before the
 * side children are launched, side children in child order, trees in root
 * order -- and numbered by a stable sort of that order on the round.  A side
 * branch that starts in the same round reuses its parent sequence's
 * initial-state source; one that starts a round later consumes the state
 * S_{b_v} requested from the parent's sequence.  Requested states are
 * deduplicated and numbered by (producer sequence, boundary position).  The
 * state bank holds the n_trees tree initial states first, then the slots.
 * ---------------------------------------------------------------------- */
int harts_plan(int32_t n_seg, const int32_t* parent, const int64_t* seg_len,
               int32_t chunk, harts_plan_t** out);

void harts_plan_free(harts_plan_t* plan);

typedef struct harts_plan_info {
  int32_t n_seg, n_trees, n_leaves;
  int32_t n_rounds;   /* K: minimum number of sequential packed calls      */
  int32_t n_seq;      /* input sequences over all rounds (= n_leaves)      */
  int32_t n_slots;    /* requested chunk-boundary states                   */
  int32_t n_bank;     /* n_trees + n_slots                                 */
  int32_t chunk;
  int64_t C;          /* compact rows (unique, non-replay)                 */
  int64_t S;          /* semantic positions (sum of trajectory lengths)    */
  int64_t R;          /* replay rows, eq. mandatory-replay                 */
  int64_t n_req;      /* (sequence, boundary) requests, = n_slots          */
  int64_t n_chunks;   /* chunks over all sequences (replay included)       */
  int64_t blob_bytes; /* size of the device descriptor image               */
} harts_plan_info;

int harts_plan_get_info(const harts_plan_t* plan, harts_plan_info* info);

/* Host arrays filled by harts_plan_export; any member may be NULL (skipped).
 * Sizes in brackets come from harts_plan_info. */
typedef struct harts_plan_arrays {
  /* per segment [n_seg] */
  int64_t* seg_start;    /* s_v: trajectory position of the first token     */
  int64_t* seg_end;      /* e_v = s_v + len_v                                */
  int64_t* seg_row;      /* physical row of the first token                 */
  int32_t* seg_seq;      /* sequence that outputs the segment               */
  int64_t* seg_mult;     /* q_v: leaves under v (eq. multiplicity)          */
  int32_t* seg_tpre;     /* T_pre(v), eq. tpre                               */
  int32_t* seg_tin;      /* T_in(v), eq. tin                                 */
  int32_t* seg_tree;     /* tree (root order) of the segment                */
  int32_t* leaf_seg;     /* [n_leaves] leaf segments by ascending id         */
  int32_t* tree_calls;   /* [n_trees] T_pre(root) of every tree              */
  int32_t* round_seq_off;/* [n_rounds+1] sequences of round r (0-based):
                            [off[r], off[r+1])                              */
  /* per sequence [n_seq] */
  int32_t* seq_round;    /* 1-based round                                   */
  int32_t* seq_tree;
  int32_t* seq_first_seg;
  int32_t* seq_final_leaf; /* index into leaf_seg / S_final                 */
  int32_t* seq_init_bank;  /* bank entry holding the initial state          */
  int64_t* seq_anchor;   /* start position A (a multiple of chunk)          */
  int64_t* seq_n_replay; /* replay rows before the first own row (< chunk)  */
  int64_t* seq_replay_off; /* [n_seq+1] offsets into replay_row             */
  int64_t* seq_row;      /* physical row of the first own token             */
  int64_t* seq_n_own;    /* own rows                                        */
  int32_t* seq_chain_off;/* [n_seq+1] offsets into chain_seg                */
  int32_t* chain_seg;    /* [n_seg] segments of every sequence, in order    */
  int32_t* seq_req_off;  /* [n_seq+1] offsets into req_chunk / req_bank     */
  /* requests [n_req] */
  int32_t* req_chunk;    /* boundary c: state at the start of chunk c       */
  int32_t* req_bank;     /* bank entry the boundary state is written to     */
  /* slots [n_slots] */
  int32_t* slot_seq;     /* producer sequence                               */
  int64_t* slot_pos;     /* boundary position b_v                            */
  /* replay [R] */
  int64_t* replay_row;   /* physical row replayed, per sequence in order    */
} harts_plan_arrays;

int harts_plan_export(const harts_plan_t* plan, const harts_plan_arrays* dst);

/* ------------------------------------------------------------------------
 * harts_plan_set_blocks -- the work decomposition of the device tables.
 * Each round's sequences are cut into blocks of consecutive chunks (at every
 * requested boundary, and after at most block_chunks chunks); one workgroup
 * runs one (block, head).  block_chunks is the largest of 64, 48, 32, 24,
 * 16, 12, 8 that still yields min_blocks blocks in the round (8 if none
 * does).  min_blocks = 0 chooses ceil(896 / H), i.e. about 896 (block, head)
 * workgroups per round; a plan fresh from harts_plan is set for H = 16.
 * Only the device descriptor image and the per-round block facts change:
 * fetch harts_plan_get_info / harts_plan_round_info / harts_plan_blob again
 * afterwards.  Results of the device calls do not depend on the blocking
 * beyond floating-point summation order.
 * Errors: HARTS_EINVAL (NULL plan, H < 1, min_blocks outside [0, 2^20]),
 * HARTS_ENOMEM (host memory; the plan's device tables are then unusable).
 * ---------------------------------------------------------------------- */
int harts_plan_set_blocks(harts_plan_t* plan, int32_t H, int32_t min_blocks);

/* Per-round launch facts (round is 0-based, < n_rounds). */
typedef struct harts_round_info {
  int32_t n_seq;         /* sequences in the round                          */
  int32_t seq_begin;     /* first sequence id of the round                  */
  int32_t n_blk;         /* blocks (runs of chunks of one sequence, ending
                            at requested boundaries) -- the device work units */
  int32_t block_chunks;  /* longest block, in chunks                        */
  int64_t n_chunks;      /* chunks over the round's sequences               */
  int64_t n_rows;        /* packed rows: own + replay                       */
  int64_t n_own;         /* own rows (outputs)                              */
  int64_t n_replay;      /* replay rows                                     */
  int64_t own_row_begin; /* own rows of the round are contiguous from here  */
  int64_t init_idx_off;  /* byte offset in the blob of the round's int32
                            [n_seq] initial-state bank indices (the idx
                            argument of harts_state_gather)                 */
  /* Byte offsets in the blob of the round's tables (int32 words), for
   * inspection; the device calls find them themselves.
   *   sequence table [n_seq][16]: chunk offset in the round, packed rows,
   *     replay rows, first replay index, physical row of the first own row,
   *     initial-state bank entry, final leaf, first request, requests,
   *     chunks, first block, blocks, 4 unused;
   *   block table [n_blk][8]: sequence (in the round), first chunk,
   *     chunks, index in the sequence, bank entry requested at its end or
   *     -1, 3 unused;
   *   launch table [n_blk][16]: the blocks in launch order (most chunks
   *     first, ties by block id): block id, sequence, first chunk, chunks,
   *     index in the sequence, blocks of the sequence, final leaf,
   *     initial-state bank entry, packed rows, replay rows, first replay
   *     index, physical row of the first own row, chunk offset, 3 unused. */
  int64_t seq_tab_off;
  int64_t blk_tab_off;
  int64_t launch_off;
} harts_round_info;

int harts_plan_round_info(const harts_plan_t* plan, int32_t round,
                          harts_round_info* info);

/* Device descriptor image (int32, blob_bytes bytes, 256-byte sections).
 * The caller copies it to device memory once per plan (step "round
 * descriptors to the device") and passes that copy as d_blob to the device
 * calls below.  Errors: HARTS_ENOMEM if bytes < blob_bytes. */
int harts_plan_blob(const harts_plan_t* plan, void* host_dst, size_t bytes);

/* ------------------------------------------------------------------------
 * harts_la_fwd -- one execution round of the packed forward (Sec. 3.4,
 * eq. chunkla-interface; chunkwise form of Sec. 2.2).
 *
 * For every sequence i of the round (rows: its replay rows, gathered by
 * index from earlier rows, then its own rows):
 *   reads   q (own rows only), k, v, g; S0[i] = its initial state;
 *   writes  o for its own rows only (o may be NULL: state pass only, the
 *           recompute-forward of the backward -- states, no outputs);
 *           bank[req] = S_c for each requested chunk boundary c;
 *           S_final[final_leaf] = the state after its last token (S_final
 *           may be NULL: not written, e.g. in a recompute-forward);
 *           saved (if non-NULL): what harts_la_bwd needs to skip the
 *           recompute (sized by harts_la_saved_size).
 *   S0       [n_seq_round, H, dk, dv] float32 (harts_state_gather output),
 *            or NULL: every sequence's initial state is then read in place
 *            from bank (its row in the round's init index, a zero state
 *            where that index is -1), which saves the gather's copy; bank
 *            is then required.  Slots this round writes are never its own
 *            initial states, so reading and writing bank in one call is safe.
 *   scale    output scale (1/sqrt(dk) is the usual choice).
 * Errors: HARTS_EINVAL (null required pointer, bad round, ws too small),
 * HARTS_EUNSUPPORTED (dtype / dims / chunk), HARTS_EHIP (launch failed).
 * ---------------------------------------------------------------------- */
int harts_la_fwd(const harts_plan_t* plan, int32_t round, const void* d_blob,
                 int32_t dtype, int32_t H, int32_t dk, int32_t dv, float scale,
                 const void* q, const void* k, const void* v, const float* g,
                 const float* S0, void* o, float* S_final, float* bank,
                 void* saved, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * harts_la_fwd_noalloc -- harts_la_fwd for callers that cannot allocate
 * device memory or pass a workspace: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  Same arguments, results
 * and errors as harts_la_fwd with saved = NULL and no workspace: the
 * round's scratch (block summaries, block-end states and log-decays) lives
 * in a fixed 64 MiB array in device memory that the library holds on every
 * GPU it runs on until the process ends.  The caller still owns and passes
 * inputs and outputs.  Nothing is allocated: no hipMalloc, hipFree or
 * allocating library call.  The scratch needs no clearing between calls
 * (every byte read is written first in the same call).
 *   Limit: rounds whose scratch (2 states of H*dk*dv*4 bytes per block,
 *   plus the block log-decays, 256-byte aligned) exceeds 64 MiB return
 *   HARTS_ENOMEM with the required size in the message, before anything
 *   is enqueued.
 *   Concurrency: all calls on one GPU share its array; two calls that may
 *   overlap on one GPU (different streams, or host threads) race.  Calls
 *   ordered on one stream are safe.
 * ---------------------------------------------------------------------- */
int harts_la_fwd_noalloc(const harts_plan_t* plan, int32_t round, const void* d_blob,
                         int32_t dtype, int32_t H, int32_t dk, int32_t dv, float scale,
                         const void* q, const void* k, const void* v, const float* g,
                         const float* S0, void* o, float* S_final, float* bank,
                         void* stream);

/* ------------------------------------------------------------------------
 * harts_la_bwd -- backward of one round (Sec. 3.4 "Differentiable boundary
 * states"; "Full-layer activation recomputation").  Rounds are run in
 * reverse: a requested state's gradient (dbank[req]) is complete once every
 * later round that consumed it has run and scattered its dS0 (harts_state_gather
 * mode 1).
 *
 *   S0, bank  initial states as for harts_la_fwd: S0 [n_seq_round, H, dk, dv],
 *             or S0 NULL and bank [n_bank, H, dk, dv] read through the round's
 *             init index (bank is unused when S0 is given).
 *   dO        [C, H, dv] upstream gradient of o (own rows of the round read).
 *   dS_final  [n_leaves, H, dk, dv] upstream gradient of the final states.
 *   dbank     [n_bank, H, dk, dv] accumulated gradients of requested states.
 *   saved     from harts_la_fwd, or NULL: the forward states are then
 *             recomputed from S0 inside this call (recompute-forward).
 *   dq, dk_, dv_  [C, H, d] written for the round's own rows (not added).
 *   dg        float32 [C, H] written for own rows.
 *   replay_grad float32 [R, H, dk + dv + 1]: per replay row (global replay
 *             index) its dk, dv and dg contributions; reduced into the
 *             compact rows by harts_replay_reduce after the last round.
 *   dS0       float32 [n_seq_round, H, dk, dv]: gradient at every sequence's
 *             initial state.
 * Deterministic: no floating-point atomics; reruns are bitwise identical.
 * ---------------------------------------------------------------------- */
int harts_la_bwd(const harts_plan_t* plan, int32_t round, const void* d_blob,
                 int32_t dtype, int32_t H, int32_t dk, int32_t dv, float scale,
                 const void* q, const void* k, const void* v, const float* g,
                 const float* S0, const float* bank, const void* dO,
                 const float* dS_final, const float* dbank, const void* saved,
                 void* dq, void* dk_, void* dv_, float* dg, float* replay_grad,
                 float* dS0, void* ws, size_t ws_bytes, void* stream);

/* Bytes of device scratch for a round's forward (pass 0) or backward
 * (pass 1; has_saved = 0 means the recompute path). */
int harts_la_workspace_size(const harts_plan_t* plan, int32_t round,
                            int32_t pass, int32_t dtype, int32_t H, int32_t dk,
                            int32_t dv, int32_t has_saved, size_t* bytes);

/* Bytes of the optional per-round forward save buffer. */
int harts_la_saved_size(const harts_plan_t* plan, int32_t round,
                        int32_t dtype, int32_t H, int32_t dk, int32_t dv,
                        size_t* bytes);

/* ------------------------------------------------------------------------
 * harts_state_gather -- state handoff between rounds (Sec. 3.4: a later
 * sequence starts from a boundary state returned by an earlier round; if
 * several consumers share one boundary tensor, their gradients are summed).
 *
 *   mode 0 (gather):      dst[i] = idx[i] < 0 ? 0 : src[idx[i]],  i < n.
 *   mode 1 (scatter-add): dst[idx[i]] += src[i] for i = 0..n-1 in order
 *                         (idx[i] < 0 skipped).  The adjoint of mode 0;
 *                         deterministic, no atomics.
 *   src, dst  float32 device arrays of states, elems_per_state floats each
 *             (H*dk*dv); idx is an int32 device array.
 * Errors: HARTS_EINVAL (null pointer, n < 0, elems_per_state not a positive
 * multiple of 4, bad mode), HARTS_EHIP.
 * ---------------------------------------------------------------------- */
int harts_state_gather(const float* src, const int32_t* idx, int32_t n,
                       int64_t elems_per_state, float* dst, int32_t mode,
                       void* stream);

/* ------------------------------------------------------------------------
 * harts_replay_reduce -- gradients of replayed rows (Sec. 4.2: replay reads
 * existing compact activations, and the indexed-gather backward accumulates
 * every consumer's gradient at the unique producer).  For every compact row
 * that some sequence replays, adds the replay_grad entries of that row (in
 * ascending replay index) to dk_, dv_ and dg.  Run once, after the backward
 * of the last (first) round.  Deterministic.
 * ---------------------------------------------------------------------- */
int harts_replay_reduce(const harts_plan_t* plan, const void* d_blob,
                        int32_t dtype, int32_t H, int32_t dk, int32_t dv,
                        const float* replay_grad, void* dk_, void* dv_,
                        float* dg, void* stream);

/* ------------------------------------------------------------------------
 * harts_mb_plan -- prefix-aware microbatch and data-parallel planning
 * (Sec. 3.2; eqs. prefix-plan-objective, compact-trie-cost,
 * cut-prefix-loss, k-lower-bound, k-search-range, contiguous-dp,
 * greedy-insertion-delta).  Host only.
 *
 * Groups N trajectories into K microbatches (K a multiple of D, exactly K/D
 * per DP replica, each microbatch's compact-trie work <= T) and orders them
 * into K/D slots, minimising J = (total compact work, sum over slots of the
 * slot's heaviest microbatch, heaviest replica's total) lexicographically
 * over the candidates it generates: the exact minimum-work contiguous
 * partitions (in lexicographic order) for every K of the search range when
 * N <= exact_max, otherwise merge/split evolutions of the natural partition
 * at up to 32 sampled K; and the best trie-aware greedy plan; refined by
 * boundary moves and sparse repair within 8 lexicographic positions.
 *   n_traj     N >= D trajectories; trajectory i is
 *              tokens[tok_off[i] .. tok_off[i+1]), 1 <= length <= T.
 *   D, T       DP degree >= 1; microbatch capacity in compact tokens >= 1.
 *   exact_max  exact-search threshold; 0 means the paper's 512.
 *   group      [N] out: microbatch of every trajectory (0 .. K-1).
 *   mb_replica, mb_slot, mb_work  [N] out (first K entries): replica, slot
 *              and compact work of every microbatch.
 *   result     out: K, the natural partition's size, J and the work of the
 *              whole batch as one trie.
 * Ties are broken by the earlier candidate, the smaller index or the
 * smaller lexicographic rank at every step (deterministic).  Errors:
 * HARTS_EINVAL (NULL, D < 1, T < 1, N < D, an empty trajectory or one above
 * T, no feasible plan), HARTS_ENOMEM.
 * ---------------------------------------------------------------------- */
typedef struct harts_mb_result {
  int32_t K;              /* microbatches in the plan                          */
  int32_t natural_K;      /* microbatches of the natural partition            */
  int64_t work_total;     /* J[0]: summed compact work                        */
  int64_t slot_critical;  /* J[1]: sum over slots of the heaviest microbatch  */
  int64_t replica_max;    /* J[2]: heaviest replica's summed work             */
  int64_t trie_work;      /* G: compact work of all trajectories as one trie  */
} harts_mb_result;

int harts_mb_plan(int32_t n_traj, const int64_t* tok_off, const int32_t* tokens, int32_t D,
                  int64_t T, int32_t exact_max, int32_t* group, int32_t* mb_replica,
                  int32_t* mb_slot, int64_t* mb_work, harts_mb_result* result);

/* ------------------------------------------------------------------------
 * Causal depthwise convolution with true-ancestor context (Sec. 4.2, "KDA
 * state reuse and causal convolution"): along every trajectory,
 *     y_t[c] = sum_{i < w} W[c, i] x_{t-i}[c]   (zero before the start),
 * computed once per compact row.  A row's window reaches its own ancestors
 * only, never an adjacent packed sequence; replay rows of the linear
 * attention read these results and never recompute them.
 *
 * harts_conv_context (host) -- the window of every row, from the plan.
 *   w         width, 2..8 (the paper's KDA uses 4).
 *   pred      [C][w-1] out: physical row of the row's i-th predecessor on
 *             its trajectory (i = 1..w-1), -1 before the trajectory start.
 *   succ_off  [C+1] out, succ [C*(w-1)] out: the consumers of every row,
 *             encoded consumer_row * 8 + i, ordered by (i, consumer_row);
 *             succ_off[C] entries in all (pass it as n_succ).
 *   Linear in C * w.  Errors: HARTS_EINVAL (NULL), HARTS_EUNSUPPORTED
 *   (w, C >= 2^28), HARTS_ENOMEM.
 * harts_conv_fwd (device) -- y [C, Cch] from x [C, Cch] (dtype HARTS_BF16
 *   or HARTS_F32, physical row order) and float32 weights W [Cch][w]; Cch
 *   a positive multiple of 8; x, y, W (and dy, dx) 16-byte aligned.
 * harts_conv_bwd (device) -- for upstream dy [C, Cch]:
 *   dx[r] = W[:, 0] dy[r] + sum over the consumers (s, i) of r of
 *           W[:, i] dy[s]   (written, in x's dtype);
 *   dW[c, i] = sum_r x[pred_i(r)][c] dy[r][c]   (float32, written),
 *   summed in fixed orders (deterministic).  ws: float32 scratch of
 *   harts_conv_workspace_size bytes (per-block partial sums of dW).
 * Table entries outside [0, C) are treated as absent (zero), never read.
 * Errors: HARTS_EINVAL (NULL / misaligned pointer, small workspace),
 * HARTS_EUNSUPPORTED (dtype, w, Cch, C), HARTS_EHIP.  Asynchronous.
 * ---------------------------------------------------------------------- */
int harts_conv_context(const harts_plan_t* plan, int32_t w, int32_t* pred, int64_t* succ_off,
                       int32_t* succ);

int harts_conv_workspace_size(int64_t C, int32_t Cch, int32_t w, size_t* bytes);

int harts_conv_fwd(int32_t dtype, int64_t C, int32_t Cch, int32_t w, const void* x, const float* W,
                   const int32_t* pred, void* y, void* stream);

int harts_conv_bwd(int32_t dtype, int64_t C, int32_t Cch, int32_t w, const void* x, const float* W,
                   const int32_t* pred, const int64_t* succ_off, const int32_t* succ, int64_t n_succ,
                   const void* dy, void* dx, float* dW, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------
 * Full attention through asymmetric packed Q/KV views (Sec. 4.2, eqs.
 * asymmetric-qkv and bottom-right), bf16, d in {64, 128}.
 *
 * One view per input sequence of the plan: its queries are the sequence's
 * l own rows; its key/value row holds the h ancestor positions of its
 * trajectory followed by the same l rows; query i sees keys j <= h + i
 * (bottom-right alignment).  Per head: o = softmax(scale Q K^T) V over the
 * visible keys.  Each compact row is the query of exactly one view, so
 * outputs and dq go straight to compact rows; key/value gradients of the
 * views are summed back into the rows they were gathered from.
 *
 * harts_attn_layout / harts_attn_views (host) -- sizes, then tables:
 *   views    [n_views][4]: first own row, l, offset in the view rows, h.
 *   kv_rows  [n_kv]: compact row of every view row (views in order).
 *   qtiles   [n_qtiles][2], kvtiles [n_kvtiles][2]: (view, first row) of
 *            every 128-row query tile and key tile, heaviest first (query
 *            tiles by the keys they see, key tiles by the queries that see
 *            them; equal work keeps the view order).
 *   row_off  [C+1], row_ent [n_kv]: view rows of every compact row,
 *            ascending (the order of the gradient sums).
 * harts_attn_gather (device) -- dst[e] = src[kv_rows[e]], [rows, H, d] bf16
 *   (the key and value views).
 * harts_attn_fwd (device) -- o [C, H, d] bf16 for every query row and
 *   lse [C, H] float32 (natural log of the softmax denominator, needed by
 *   the backward), from q [C, H, d] and the key/value views [n_kv, H, d].
 * harts_attn_bwd (device) -- from dO [C, H, d]: dq [C, H, d] bf16 (written),
 *   dk_view, dv_view [n_kv, H, d] float32 (written); delta [C, H] float32 is
 *   scratch (dO . o per row).
 * harts_attn_scatter (device) -- dst [C, H, d] bf16 = sum over each row's
 *   view rows of src [n_kv, H, d] float32, in row_ent order (deterministic).
 * Pointers to row tensors 16-byte aligned.  Errors: HARTS_EINVAL (NULL,
 * misaligned, sizes), HARTS_EUNSUPPORTED (H, d; more than 2^31 - 1 view
 * rows), HARTS_EHIP, HARTS_ENOMEM.  Device calls are asynchronous.
 * ---------------------------------------------------------------------- */
typedef struct harts_attn_sizes {
  int64_t n_views, n_kv, n_qtiles, n_kvtiles;
} harts_attn_sizes;

int harts_attn_layout(const harts_plan_t* plan, harts_attn_sizes* out);

int harts_attn_views(const harts_plan_t* plan, int32_t* views, int32_t* kv_rows, int32_t* qtiles,
                     int32_t* kvtiles, int64_t* row_off, int32_t* row_ent);

int harts_attn_gather(const void* src, const int32_t* kv_rows, int64_t n_kv, int64_t C, int32_t H,
                      int32_t d, void* dst, void* stream);

int harts_attn_fwd(const int32_t* views, const int32_t* qtiles, int64_t n_qtiles, int32_t H, int32_t d,
                   float scale, const void* q, const void* kv_k, const void* kv_v, void* o, float* lse,
                   void* stream);

int harts_attn_bwd(const int32_t* views, const int32_t* qtiles, int64_t n_qtiles, const int32_t* kvtiles,
                   int64_t n_kvtiles, int64_t C, int32_t H, int32_t d, float scale, const void* q,
                   const void* kv_k, const void* kv_v, const void* o, const float* lse, const void* dO,
                   float* delta, void* dq, float* dk_view, float* dv_view, void* stream);

int harts_attn_scatter(const float* src, const int64_t* row_off, const int32_t* row_ent, int64_t C,
                       int64_t n_kv, int32_t H, int32_t d, void* dst, void* stream);

/* ------------------------------------------------------------------------
 * KDA: linear attention with per-channel decay and the delta rule (Sec. 2.2,
 * eq. chunk-state), over the same plan: rounds, replay rows, requested
 * boundary states and their differentiable handoffs (Sec. 3.4).  Per head,
 * state S [dk = d][dv = d]:
 *     S_t = Diag(e^{g_t}) S_{t-1}
 *           + beta_t k_t (v_t - (Diag(e^{g_t}) S_{t-1})^T k_t)^T,
 *     o_t = scale S_t^T q_t,
 * run by chunks of 64 packed rows in the form of eq. chunk-state (the plan
 * must have chunk 64).  q, k, v, o [C, H, d] (bf16 or float32), g [C, H, d]
 * float32 log-decays (<= 0), beta [C, H] float32.
 *
 * harts_kda_layout / harts_kda_tables (host) -- sizes, then tables:
 *   chunk_rows [n_chunks][64]: packed rows of every sequence (replay rows,
 *              then own rows, then padding), in sequence order: physical
 *              row * 2 + 1 for an own row, * 2 for a replay row, -1 padding.
 *   seq_tab    [n_seq][8]: round (0-based), first chunk, chunks, initial
 *              bank entry, first request, requests, final leaf, and in the
 *              last column the order in which the state passes take the
 *              round's sequences: row s0 + j holds the sequence taken j-th,
 *              longest first (ties by id).
 *   req_tab    [n_req][2]: (chunk c of the sequence, bank entry): the state
 *              at the start of chunk c (c = chunks: the end state), each
 *              sequence's requests in ascending chunk order.
 *   group_tab  [n_groups][4], group_seq [n_seq]: per round, the sequences
 *              starting from each bank entry (round, entry, first member,
 *              members), in sequence order -- the order of the adjoint sums.
 *   pos_slot   [n_chunks * 64]: per packed row (chunk * 64 + i), -1 when
 *              its compact row has no other packed row (its gradients go
 *              straight to the outputs), else its slot: the n_multi compact
 *              rows with replay copies, ascending, hold slots
 *              [multi_off[m], multi_off[m + 1]) in ascending packed order.
 *   multi_row  [n_multi], multi_off [n_multi + 1] (n_slots in all).
 * harts_kda_workspace_size -- float32 per-(chunk, head) blocks for all
 *   chunks of the plan (the forward's are read by the backward).
 * harts_kda_fwd (device) -- one round: chunks [c0, c0 + n_chunks), sequences
 *   [s0, s0 + n_seq).  bank [n_bank][H][d][d] float32: read at the initial
 *   entries, written at the requested ones; S_final [n_leaves][H][d][d]
 *   (may be NULL); o written for own rows (o NULL: states only).
 * harts_kda_bwd (device) -- one round, after the later rounds' backward:
 *   dO [C, H, d]; dS_final (may be NULL); dbank [n_bank][H][d][d] holds the
 *   later rounds' summed initial-state adjoints; writes dS0_seq
 *   [n_seq][H][d][d] of the round's sequences.  Gradients of the round's
 *   packed rows: for a compact row with one packed row, straight into
 *   dq, dk, dv [C, H, d] (dtype), dg [C, H, d] and dbeta [C, H] (float32);
 *   otherwise float32 partials into its slot of sdq, sdk, sdv, sdg
 *   [n_slots][H][d] and sdb [n_slots][H] (NULL allowed when n_slots = 0).
 *   dq, dk, sdq and sdk must be 16-byte aligned (four-element stores).
 * harts_kda_bank_add (device) -- dbank[entry] += the group's dS0_seq, for
 *   groups [g0, g0 + n_groups) (one round's), in member order.
 * harts_kda_reduce (device) -- after every round's backward: for the
 *   n_multi compact rows with several packed rows, dst [C][width] (bf16 or
 *   float32) row multi_row[m] = the sum of src [n_slots][width] over slots
 *   [multi_off[m], multi_off[m + 1]), in slot order.
 * All arithmetic is float32 and deterministic (no atomics).  Errors:
 * HARTS_EINVAL (NULL, ranges), HARTS_EUNSUPPORTED (dtype, H, d, a plan with
 * chunk != 64, more than 2^31 - 1 packed rows), HARTS_EHIP, HARTS_ENOMEM.
 * ---------------------------------------------------------------------- */
typedef struct harts_kda_sizes {
  int64_t n_chunks, n_slots;
  int32_t n_seq, n_rounds, n_groups, n_req, n_multi, pad;
} harts_kda_sizes;

int harts_kda_layout(const harts_plan_t* plan, harts_kda_sizes* out);

int harts_kda_tables(const harts_plan_t* plan, int32_t* chunk_rows, int32_t* seq_tab, int32_t* req_tab,
                     int32_t* group_tab, int32_t* group_seq, int32_t* pos_slot, int32_t* multi_row,
                     int64_t* multi_off);

int harts_kda_workspace_size(int64_t n_chunks, int32_t H, int32_t d, size_t* bytes);

int harts_kda_fwd(const int32_t* chunk_rows, const int32_t* seq_tab, const int32_t* req_tab, int64_t c0,
                  int64_t n_chunks, int32_t s0, int32_t n_seq, int32_t dtype, int32_t H, int32_t d, float scale,
                  const void* q, const void* k, const void* v, const float* g, const float* beta, float* bank,
                  float* S_final, void* o, float* ws, void* stream);

int harts_kda_bwd(const int32_t* chunk_rows, const int32_t* seq_tab, const int32_t* req_tab, const int32_t* pos_slot,
                  int64_t c0, int64_t n_chunks, int32_t s0, int32_t n_seq, int32_t dtype, int32_t H, int32_t d,
                  float scale, const void* q, const void* k, const void* v, const float* g, const float* beta,
                  const void* dO, const float* dS_final, const float* dbank, float* dS0_seq, float* ws, void* dq,
                  void* dk, void* dv, float* dg, float* dbeta, float* sdq, float* sdk, float* sdv, float* sdg,
                  float* sdb, void* stream);

int harts_kda_bank_add(const int32_t* group_tab, int32_t g0, int32_t n_groups, const int32_t* group_seq,
                       int64_t elems, const float* dS0_seq, float* dbank, void* stream);

int harts_kda_reduce(const float* src, const int32_t* multi_row, const int64_t* multi_off, int64_t n_multi,
                     int64_t width, int32_t dtype, void* dst, void* stream);

/* ------------------------------------------------------------------------
 * Compact-to-semantic log-probabilities (Sec. 3.5, eqs. mapped-logp and
 * mapped-logp-grad).  Vocabulary-wide work runs once per compact logit row;
 * only scalar work runs per semantic position, and no S x V tensor exists.
 *
 * harts_semantic_map (host) -- the positions of the original batch and the
 * rows that serve them.  Trajectories are taken by ascending leaf id (the
 * order of harts_plan_arrays.leaf_seg), positions in trajectory order; the
 * last position of every trajectory has no next token and is left out, so
 * there are n_pos = S - n_leaves positions.
 *   tokens   [C] token id of every compact row, physical row order.
 *   m        [n_pos] out: physical row of position s (its logit row).
 *   y        [n_pos] out: the token at position s + 1 of the same trajectory.
 *   row_off  [C + 1] out, row_pos [n_pos] out: positions served by each
 *            row, row c owning row_pos[row_off[c] .. row_off[c+1]), ordered
 *            by (y, position).
 * Linear in S.  Errors: HARTS_EINVAL (NULL, n_pos != S - n_leaves),
 * HARTS_EUNSUPPORTED (C or n_pos >= 2^31), HARTS_ENOMEM.
 *
 * harts_logp_fwd (device) -- lse[c] = log sum_v exp z[c, v] for every row,
 * then logp[s] = z[m[s], y[s]] - lse[m[s]] for every position.
 *   logits   [C, V] row-major, HARTS_BF16 or HARTS_F32 (dtype), 16-byte
 *            aligned; V a positive multiple of 8.
 *   lse      [C] float32 out; logp [n_pos] float32 out.
 *   An (m, y) pair outside [0, C) x [0, V) yields logp = NaN; nothing is
 *   read out of bounds.
 *
 * harts_logp_bwd (device) -- for upstream gradients dlogp[s] (zero where
 * the action mask drops a position):
 *   row_g[c]        = sum of dlogp over the row's positions (float32 out);
 *   dlogits[c, v]   = -row_g[c] softmax(z[c])_v
 *                     + sum of dlogp[s] over the row's positions with y = v,
 *   written (not added) for every row, in the logits' dtype, rounded once.
 *   lse from harts_logp_fwd; row_off, row_pos, y from harts_semantic_map.
 *   Deterministic: each row's sums run in its (y, position) order.
 * Both: asynchronous on the stream; errors HARTS_EINVAL (NULL required
 * pointer, negative sizes, misaligned logits), HARTS_EUNSUPPORTED (dtype,
 * V), HARTS_EHIP.
 * ---------------------------------------------------------------------- */
int harts_semantic_map(const harts_plan_t* plan, const int32_t* tokens, int64_t n_pos,
                       int32_t* m, int32_t* y, int64_t* row_off, int32_t* row_pos);

int harts_logp_fwd(int32_t dtype, int64_t C, int64_t V, const void* logits, int64_t n_pos,
                   const int32_t* m, const int32_t* y, float* lse, float* logp, void* stream);

int harts_logp_bwd(int32_t dtype, int64_t C, int64_t V, const void* logits, const float* lse,
                   int64_t n_pos, const int64_t* row_off, const int32_t* row_pos,
                   const int32_t* y, const float* dlogp, float* row_g, void* dlogits,
                   void* stream);

/* ------------------------------------------------------------------------
 * Kernel timing (measurement support; not part of the method).  Between
 * harts_profile_begin and harts_profile_end every kernel the library
 * launches is bracketed by a pair of HIP events recorded on its own launch
 * stream.  harts_profile_end waits for those events, sums the elapsed time
 * per kernel name and fills up to cap entries of out (n_out receives the
 * number of distinct kernels).  Host-side only; not thread-safe against
 * concurrent profiling sessions.
 * ---------------------------------------------------------------------- */
typedef struct harts_kernel_time {
  char name[48];
  int32_t launches;
  double total_ms;
} harts_kernel_time;

int harts_profile_begin(void);
int harts_profile_end(harts_kernel_time* out, int32_t cap, int32_t* n_out);

#ifdef __cplusplus
}
#endif
#endif /* HARTS_H_ */
