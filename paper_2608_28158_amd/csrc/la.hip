// Packed chunkwise linear attention with per-head scalar decay, one
// execution round per call (HARTS, Sec. 3.4, eq. chunkla-interface), for
// gfx950.  Recurrence per head (state S: [dk, dv]):
//     S_t = exp(g_t) S_{t-1} + k_t v_t^T,    o_t = scale * S_t^T q_t.
// Chunkwise form (Sec. 2.2): for chunk c with start state S_c and in-chunk
// inclusive prefix sums G (G_i = g_0 + ... + g_i, local to the chunk),
//     O        = scale * ((Q K^T) * exp(G_i - G_j) [j <= i]) V
//              + scale * diag(exp(G)) Q S_c
//     S_{c+1}  = exp(G_last) S_c + (K * exp(G_last - G))^T V.
//
// Work decomposition.  Every sequence of a round is cut into blocks of
// consecutive chunks (the planner ends a block at every requested boundary
// and at most every block_chunks chunks).  One workgroup owns one
// (block, head) and keeps a [d x d] float32 state in MFMA accumulators
// (wave w holds state columns 16w .. 16w+15) while it walks the block's
// chunks; per-chunk states are never written to memory.  The next chunk's
// rows are loaded into registers while the current chunk computes.  Decay
// factors that weight the rows of a state-update operand are applied to its
// fragments in registers, so LDS holds only unscaled chunk tiles.  Blocks of
// one sequence are chained by element-parallel scans over block summaries:
//
//   forward   k_blocksum      state of each block started from zero and
//                             its total log-decay Gamma_b;
//             k_fwd_blockscan S_end[b] = exp(Gamma_b) S_end[b-1] + dS_b,
//                             which also yields every requested boundary
//                             state and every final state;
//             k_fwd_block     outputs of the own rows of each block.
//   backward  (k_blocksum and k_fwd_blockscan first when recomputing)
//             k_bwd_fwdorder  dq and q.dq per row (needs S_c, so it walks
//                             chunks forward), and the block's local adjoint
//                             U_b = sum_t exp(G_t^blk) scale q_t dO_t^T;
//             k_bwd_blockscan dS_end[b] by the reverse recurrence
//                             dS_start[b] = exp(Gamma_b) dS_end[b] + U_b,
//                             bank gradients injected at requested block
//                             ends, dS0 per sequence, boundary terms;
//             k_bwd_revorder  dv (side 0) and dk, k.dk, local suffix sums of
//                             dg (side 1); both need dS_{c+1} and walk
//                             chunks backward;
//             k_dg_carry      adds to dg the contributions of later blocks.
// dg uses dg_t = sum_{u >= t} (q_u.dq_u - k_u.dk_u) + <dS_final, S_final>
//              + sum_{requested P > t} <dbank_P, S_P>   (per sequence),
// which follows from rescaling q and k (adding e to g_t scales q_u by e^e and
// k_u by e^-e for u >= t).
// All products run on MFMA (bf16 16x16x32 / 16x16x16 or f32 16x16x4); states
// and accumulation are float32; no floating-point atomics.
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "la_common.hpp"
#include "plan.hpp"

namespace harts {

// ---------------------------------------------------------------------------
// chunk staging: global rows -> registers (one chunk ahead) -> LDS tiles
// ---------------------------------------------------------------------------
union Vec16 {
  uint4 u;
  float f[4];
  bf16 b[8];
};

template <typename T>
__device__ inline T vget(const Vec16& v, int e);
template <>
__device__ inline float vget<float>(const Vec16& v, int e) { return v.f[e]; }
template <>
__device__ inline bf16 vget<bf16>(const Vec16& v, int e) { return v.b[e]; }
template <typename T>
__device__ inline void vset(Vec16& v, int e, T x);
template <>
__device__ inline void vset<float>(Vec16& v, int e, float x) { v.f[e] = x; }
template <>
__device__ inline void vset<bf16>(Vec16& v, int e, bf16 x) { v.b[e] = x; }

// Rows of one chunk: a contiguous run of 64 own rows (fast: physical rows
// row0 .. row0 + 63, every interior chunk of a sequence) or rows resolved one
// by one (chunks holding replay rows or padding).  Uniform per workgroup.
struct ChunkRows {
  int fast;
  int row0;
};
__device__ inline ChunkRows chunk_rows(const SeqInfo& sq, int c) {
  const int p0 = c * CB;
  ChunkRows cr;
  cr.fast = p0 >= sq.n_rep && p0 + CB <= sq.n_tok;
  cr.row0 = sq.own_row + p0 - sq.n_rep;
  return cr;
}

// How NTH threads split the 16-byte pieces of a [64][D] chunk tile.
template <typename T, int D, int NTH>
struct Stg {
  static constexpr int NTHR = NTH;
  static constexpr int VE = 16 / sizeof(T);   // elements per 16-byte vector
  static constexpr int VPR = D / VE;          // vectors per row
  static constexpr int NV = CB * VPR / NTH;   // vectors per thread per tile
  using TD = Tile<T, D>;
};

// This thread's rows of one chunk (a row's d-range is split over VPR
// threads), each as row * 4 + kind; resolved for chunks that are not fast.
template <typename T, int D, int NTH = Cfg<T, D>::NTHR>
struct ChunkRefs {
  int rk[Stg<T, D, NTH>::NV];
  __device__ inline void resolve(const SeqInfo& seq, int c, const int32_t* replay_row, int t) {
    using C = Stg<T, D, NTH>;
#pragma unroll
    for (int i = 0; i < C::NV; ++i) {
      const RowRef rr = pos_row(seq, c * CB + (t + i * C::NTHR) / C::VPR, replay_row);
      rk[i] = rr.row * 4 + rr.kind;
    }
  }
};

// dst[row][d] = src[row][d] (* scale[row] if scale != nullptr), dst in layout L
template <typename T, int D, int NTH = Cfg<T, D>::NTHR, typename L = Tile<T, D>>
__device__ inline void put(T* dst, const Vec16* src, const float* scale, int t) {
  using C = Stg<T, D, NTH>;
#pragma unroll
  for (int i = 0; i < C::NV; ++i) {
    const int idx = t + i * C::NTHR;
    const int row = idx / C::VPR, d0 = (idx % C::VPR) * C::VE;
    Vec16 v = src[i];
    if (scale) {
      const float s = scale[row];
#pragma unroll
      for (int e = 0; e < C::VE; ++e) vset<T>(v, e, Elem<T>::from_f(Elem<T>::to_f(vget<T>(v, e)) * s));
    }
    *reinterpret_cast<uint4*>(dst + L::at(row, d0)) = v.u;
  }
}

// Per-chunk row table, decay prefix sums and two per-row factors, shared
// through LDS.
struct ChunkMeta {
  alignas(16) float G[CB];  // G_t = g_0 + ... + g_t within the chunk
  alignas(16) float x[CB];  // kernel-specific per-row factors
  alignas(16) float y[CB];
  int rowk[CB];  // physical row * 4 + kind (replay index = replay_off + position)
};

// 1 KiB of zeros: rows that must read as zero (padding, or rows of a kind a
// tensor does not hold) are loaded from here, so that every lane issues the
// same unconditional load and no load sits in a divergent branch (a load in
// one, followed by a write of its register in the other, would have to
// complete before the branches join).
__device__ __align__(16) uint4 kZeroRow[64] = {};  // never written
static_assert(sizeof(kZeroRow) >= 256 * sizeof(float), "one zero row of up to 256 floats");

// Where this thread's rows of one chunk live, resolved one chunk ahead: the
// rows it stages (all threads) and, for the wave that publishes the chunk's
// row table (mrow = its lane, -1 elsewhere), row mrow of the chunk with its g.
template <typename T, int D, int NTH = Cfg<T, D>::NTHR>
struct ChunkSrc {
  ChunkRows cr;
  ChunkRefs<T, D, NTH> refs;
  RowRef mr;
  float gv;
  __device__ inline void resolve(const SeqInfo& seq, int c, const int32_t* replay_row,
                                 const float* g, int H, int h, int t, int mrow) {
    cr = chunk_rows(seq, c);
    // the two cases apart, so that the fast case's g address waits on no load
    if (cr.fast) {
      if (mrow >= 0) {
        mr = RowRef{cr.row0 + mrow, ROW_OWN, -1};
        gv = g[static_cast<int64_t>(mr.row) * H + h];
      }
    } else {
      refs.resolve(seq, c, replay_row, t);
      if (mrow >= 0) {
        mr = pos_row(seq, c * CB + mrow, replay_row);
        gv = *(mr.kind != ROW_PAD ? g + static_cast<int64_t>(mr.row) * H + h
                                  : reinterpret_cast<const float*>(kZeroRow));
      }
    }
  }
};

// This thread's 16-byte pieces of one chunk tile of src (rows of kind below
// min_kind read as zero).
template <typename T, int D, int NTH = Cfg<T, D>::NTHR>
__device__ inline void fetch(Vec16* dst, const T* __restrict__ src, const ChunkSrc<T, D, NTH>& cs,
                             int H, int h, int t, int min_kind) {
  using C = Stg<T, D, NTH>;
  if (cs.cr.fast) {
    const T* base = src + (static_cast<int64_t>(cs.cr.row0) * H + h) * D;
#pragma unroll
    for (int i = 0; i < C::NV; ++i) {
      const int idx = t + i * C::NTHR;
      dst[i].u = *reinterpret_cast<const uint4*>(base + (idx / C::VPR) * H * D + (idx % C::VPR) * C::VE);
    }
    return;
  }
#pragma unroll
  for (int i = 0; i < C::NV; ++i) {
    const int d0 = ((t + i * C::NTHR) % C::VPR) * C::VE;
    const int row = cs.refs.rk[i] >> 2;
    const T* p = (cs.refs.rk[i] & 3) >= min_kind ? src + (static_cast<int64_t>(row) * H + h) * D + d0
                                                 : reinterpret_cast<const T*>(kZeroRow) + d0;
    dst[i].u = *reinterpret_cast<const uint4*>(p);
  }
}

// Resolves chunk c into cs and requests two of its tiles, with the fast and
// the slow case each in one branch.  A load of the slow case's row lookups
// then never reaches the fast case's code, whose address arithmetic would
// otherwise wait for every outstanding memory operation (the output stores
// included) before reusing such a load's destination register.
template <typename T, int D, int NTH = Cfg<T, D>::NTHR>
__device__ inline void resolve_fetch2(ChunkSrc<T, D, NTH>& cs, const SeqInfo& sq, int c,
                                      const int32_t* replay_row, const float* g, int H, int h,
                                      int t, int mrow, Vec16* da, const T* __restrict__ sa,
                                      int ka, Vec16* db, const T* __restrict__ sb, int kb) {
  if (chunk_rows(sq, c).fast) {
    cs.resolve(sq, c, replay_row, g, H, h, t, mrow);
    fetch<T, D, NTH>(da, sa, cs, H, h, t, ka);
    fetch<T, D, NTH>(db, sb, cs, H, h, t, kb);
  } else {
    cs.resolve(sq, c, replay_row, g, H, h, t, mrow);
    fetch<T, D, NTH>(da, sa, cs, H, h, t, ka);
    fetch<T, D, NTH>(db, sb, cs, H, h, t, kb);
  }
}

// The publishing wave (lane t = row t): publishes the row table and G of the
// chunk whose sources are in cs; returns G_t and G_last.
template <typename T, int D, int NTH>
__device__ inline void meta_publish(ChunkMeta& m, const ChunkSrc<T, D, NTH>& cs, int t, float& Gt,
                                    float& GL) {
  m.rowk[t] = cs.mr.row * 4 + cs.mr.kind;
  const float x = wave_prefix_sum(cs.gv, t);
  m.G[t] = x;
  Gt = x;
  GL = lane_value(x, CB - 1);
}

// A wave's part of a [D x D] state is held in the accumulator layout: tile
// j * NT + i covers rows 16 i.., columns 16 (CPW w + j).. of the matrix (or of
// its transpose), lane (g, c) element r at row 16 i + 4g + r, column .. + c.
template <int D, int CPW>
__device__ inline void state_store(float* dst, const f32x4* S, int w, int lane) {
  constexpr int NT = D / 16;
#pragma unroll
  for (int j = 0; j < CPW; ++j)
#pragma unroll
    for (int i = 0; i < NT; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        dst[(i * 16 + acc_row(lane, r)) * D + (CPW * w + j) * 16 + acc_col(lane)] = S[j * NT + i][r];
}

// A [D x D] float state staged through LDS: read once with 16-byte loads by
// all NTH threads (row pitch D + 4 floats), then handed out to the waves in
// their accumulator layout (above).  The pitch makes the reads of the
// plain layout free of bank conflicts; the transposed ones conflict up to
// four ways, once per block.
template <int D>
struct StateStage {
  static constexpr int PITCH = D + 4;
  static constexpr int BYTES = D * PITCH * 4;
};
template <int D, int NTH>
__device__ inline void state_to_lds(float* stg, const float* __restrict__ src, int tid) {
  constexpr int N4 = D * D / 4;
  static_assert(N4 % NTH == 0, "state split");
#pragma unroll
  for (int i = 0; i < N4 / NTH; ++i) {
    const int e4 = tid + i * NTH;
    const int r = e4 / (D / 4), c = (e4 % (D / 4)) * 4;
    *reinterpret_cast<float4*>(stg + r * StateStage<D>::PITCH + c) =
        *reinterpret_cast<const float4*>(src + static_cast<int64_t>(e4) * 4);
  }
}
// The whole staged load, in NPASS passes of D / NPASS stored rows each (for
// LDS that holds only part of a state; src null: a zero state); every thread
// of the workgroup calls it (it synchronises the workgroup), and the waves
// with take set receive their strips.
template <int D, int CPW, int NTH, int NPASS>
__device__ inline void state_via_lds(f32x4* S, float* stg, const float* __restrict__ src,
                                     bool transpose, int w, int lane, int tid, bool take = true) {
  constexpr int NT = D / 16, P = D + 4, RP = D / NPASS, N4 = RP * D / 4;
  static_assert(N4 % NTH == 0, "state split");
#pragma unroll
  for (int pass = 0; pass < NPASS; ++pass) {
#pragma unroll
    for (int i = 0; i < N4 / NTH; ++i) {
      const int e4 = tid + i * NTH;
      const int r = e4 / (D / 4), c = (e4 % (D / 4)) * 4;
      *reinterpret_cast<float4*>(stg + r * P + c) =
          src ? *reinterpret_cast<const float4*>(src + (static_cast<int64_t>(pass) * RP * D + e4 * 4))
              : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    __syncthreads();
    if (take) {
#pragma unroll
      for (int j = 0; j < CPW; ++j)
#pragma unroll
        for (int i = 0; i < NT; ++i)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int a = i * 16 + acc_row(lane, r), b = (CPW * w + j) * 16 + acc_col(lane);
            const int row = transpose ? b : a, col = transpose ? a : b;
            if (row / RP == pass) S[j * NT + i][r] = stg[(row - pass * RP) * P + col];
          }
    }
    __syncthreads();
  }
}

template <int D, int CPW>
__device__ inline void state_from_lds(f32x4* S, const float* stg, bool transpose, int w, int lane) {
  constexpr int NT = D / 16, P = StateStage<D>::PITCH;
#pragma unroll
  for (int j = 0; j < CPW; ++j)
#pragma unroll
    for (int i = 0; i < NT; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int a = i * 16 + acc_row(lane, r), b = (CPW * w + j) * 16 + acc_col(lane);
        S[j * NT + i][r] = transpose ? stg[b * P + a] : stg[a * P + b];
      }
}

// <X, S>_F of a state S held in accumulators (as state_from_lds lays it out,
// transposed or not) with a row-major D x D state X in global memory, summed
// over the waves with take set (of the workgroup of NTH threads) and returned
// to every thread.  X is staged through stg (D x (D + 4) floats); red holds
// NTH / 64 floats.  Every thread calls it (it synchronises the workgroup).
template <int D, int CPW, int NTH>
__device__ inline float state_dot_via_lds(const f32x4* S, float* stg, const float* __restrict__ X,
                                          bool transpose, int w, int lane, int tid, float* red,
                                          bool take = true) {
  constexpr int NT = D / 16, P = StateStage<D>::PITCH, N4 = D * D / 4;
  static_assert(N4 % NTH == 0, "state split");
#pragma unroll
  for (int i = 0; i < N4 / NTH; ++i) {
    const int e4 = tid + i * NTH;
    const int r = e4 / (D / 4), c = (e4 % (D / 4)) * 4;
    *reinterpret_cast<float4*>(stg + r * P + c) = *reinterpret_cast<const float4*>(X + static_cast<int64_t>(e4) * 4);
  }
  __syncthreads();
  float x = 0.f;
  if (take) {
#pragma unroll
    for (int j = 0; j < CPW; ++j)
#pragma unroll
      for (int i = 0; i < NT; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int a = i * 16 + acc_row(lane, r), b = (CPW * w + j) * 16 + acc_col(lane);
          x += S[j * NT + i][r] * (transpose ? stg[b * P + a] : stg[a * P + b]);
        }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  if (lane == 0) red[tid >> 6] = x;
  __syncthreads();
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < NTH / 64; ++i) sum += red[i];
  return sum;
}

// The masked score tile in three 32 x 32 blocks, (row half, column half) =
// (0, 0), (1, 0), (1, 1) for waves 0, 1, 2; the block above the diagonal is
// never read by the consumers and wave 3 does nothing here.  Each block is
// 2 x 2 tiles of 16 and reads 32 rows of each operand (the four row blocks
// of 16 rows each would read all of R four times).  Inside the diagonal blocks the
// tile above the diagonal is skipped and stored as zeros: the consumers'
// 32-deep steps read it.  P[m][n] = f * exp(G_m - G_n) * (L R^T)[m][n] for
// n <= m; with PT the tile is stored transposed.  The weight is one base-2
// exponential per element of the difference of pre-scaled prefix sums (the
// factor f folded in as log2|f| on the row side); above the diagonal of a
// diagonal tile the exponent is -inf, so the weight is exactly zero.
template <bool DIAG, bool NEG, typename T, int D, bool PT, typename TA>
__device__ __forceinline__ void score_epilogue(T* P, const f32x4 (&c)[2][2], const float* G, float lf,
                                               int rb, int cb, int lane) {
  constexpr float L2E = 1.4426950408889634f;
  f32x4 mb;  // exponent bias of a diagonal tile at the lane's rows 4g + r, column lane % 16
#pragma unroll
  for (int r = 0; r < 4; ++r) mb[r] = (lane & 15) <= acc_row(lane, r) ? 0.f : -__builtin_inff();
#pragma unroll
  for (int ti = 0; ti < 2; ++ti) {
    const int m0 = rb + 16 * ti;
    const f32x4 Gm = row_vec(G, m0, lane);
    f32x4 Gm2;
#pragma unroll
    for (int r = 0; r < 4; ++r) Gm2[r] = Gm[r] * L2E + lf;
#pragma unroll
    for (int tj = 0; tj < 2; ++tj) {
      const int n = cb + 16 * tj + acc_col(lane);
      const float Gn2 = G[n] * L2E;
      f32x4 v;
      if (DIAG && ti == 0 && tj == 1) {
        v = f32x4{0.f, 0.f, 0.f, 0.f};
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float a = Gm2[r] - Gn2;
          if (DIAG && ti == tj) a += mb[r];
          v[r] = c[ti][tj][r] * __builtin_amdgcn_exp2f(a);
          if (NEG) v[r] = -v[r];
        }
      }
      if (PT) {
        Vec4<T>::store(P + TA::at(n, m0 + acc_row(lane, 0)), v);
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) P[TA::at(m0 + acc_row(lane, r), n)] = Elem<T>::from_f(v[r]);
      }
    }
  }
}

template <typename T, int D, bool PT = false, typename LL = Tile<T, D>, typename LR = Tile<T, D>,
          typename LP = Tile<T, CB>>
__device__ __forceinline__ void score_block(T* P, const T* Lt, const T* Rt, const float* G, float f,
                                            int w, int lane) {
  using F = Frag<T>;
  const int rb = w == 0 ? 0 : 32, cb = w == 2 ? 32 : 0;
  const bool diag = rb == cb;
  f32x4 c[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) c[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
  for (int k = 0; k < D; k += F::KSTEP) {
    const typename F::V a0 = F::template kc<LL>(Lt, rb, k, lane);
    const typename F::V a1 = F::template kc<LL>(Lt, rb + 16, k, lane);
    const typename F::V b0 = F::template kc<LR>(Rt, cb, k, lane);
    const typename F::V b1 = F::template kc<LR>(Rt, cb + 16, k, lane);
    __builtin_amdgcn_sched_barrier(0);
    F::mma(c[0][0], a0, b0);
    F::mma(c[1][0], a1, b0);
    F::mma(c[1][1], a1, b1);
    if (!diag) F::mma(c[0][1], a0, b1);
  }
  // f = 1 folds away; otherwise log2|f| joins the row exponents
  const float lf = f == 1.f ? 0.f : __builtin_amdgcn_logf(__builtin_fabsf(f));
  if (f < 0.f) {
    if (diag) score_epilogue<true, true, T, D, PT, LP>(P, c, G, lf, rb, cb, lane);
    else score_epilogue<false, true, T, D, PT, LP>(P, c, G, lf, rb, cb, lane);
  } else {
    if (diag) score_epilogue<true, false, T, D, PT, LP>(P, c, G, lf, rb, cb, lane);
    else score_epilogue<false, false, T, D, PT, LP>(P, c, G, lf, rb, cb, lane);
  }
}

// The same as an out-of-line call: the reverse-order kernel keeps its score
// phase in a separate register allocation (its chunk loop holds two states'
// worth of registers).

// ---------------------------------------------------------------------------
// forward block summaries: one pass over a block's chunks, state started from
// zero: dS_b = sum over the block of the chunk recurrence
// S <- exp(G_last) S + K^T diag(exp(G_last - G)) V, and Gamma_b = the total
// log-decay of the block.  (The adjoint summaries U_b are formed by the
// forward-order backward kernel, which holds the chunk's q and dO anyway.)
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ __launch_bounds__((Cfg<T, D>::NTHR), (Cfg<T, D>::WPE)) void k_blocksum(
    const int32_t* __restrict__ seq_tab, const int32_t* __restrict__ blk_tab,
    const int32_t* __restrict__ blk_launch,
    const int32_t* __restrict__ replay_row, int H, const T* __restrict__ k,
    const T* __restrict__ v, const float* __restrict__ g, float* __restrict__ dSb,
    float* __restrict__ gam, int skip1) {
  using C = Cfg<T, D>;
  __shared__ T Xs[Tile<T, D>::SIZE];
  __shared__ T Ys[Tile<T, D>::SIZE];
  __shared__ ChunkMeta meta;
  const BlkInfo bl = blk_info(blk_launch, blockIdx.x / H);
  const int b = bl.b, h = blockIdx.x % H, t = threadIdx.x, lane = t & 63;
  const int w = wave_id(t);
  const SeqInfo sq = bl.sq;
  const int c0 = bl.c0, c_end = c0 + bl.nc;
  const int64_t bi = static_cast<int64_t>(b) * H + h;
  // The block kernels end a sequence's forward chain themselves: of the last
  // block only Gamma_b is needed (for the adjoint chain).
  if (skip1 && bl.idx == bl.n_blk - 1) {
    if (w != 0) return;
    // Gamma_b alone, summed chunk by chunk as below; wave 0, lane = row
    ChunkSrc<T, D> cs;
    float Gs = 0.f;
    for (int c = c0; c < c_end; ++c) {
      cs.resolve(sq, c, replay_row, g, H, h, t, t);
      Gs += lane_value(wave_prefix_sum(cs.gv, t), CB - 1);
    }
    if (t == 0) gam[bi] = Gs;
    return;
  }
  f32x4 S[C::CPW * C::NT];
#pragma unroll
  for (int i = 0; i < C::CPW * C::NT; ++i) S[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float Gs = 0.f;  // log-decay from the block start to the current chunk start
  // One chunk: its row table and decay factors published (wave 0, lane =
  // row, from that row's g), its tiles stored, then (after the next loads
  // are issued by `next`) added to the state.
  const auto sum_chunk = [&](const Vec16* px, const Vec16* py, float gv, auto&& next) {
    if (t < CB) {
      const float x = wave_prefix_sum(gv, t);
      meta.G[t] = x;
      meta.x[t] = __expf(lane_value(x, CB - 1) - x);
    }
    put<T, D>(Xs, px, nullptr, t);
    put<T, D>(Ys, py, nullptr, t);
    __syncthreads();
    next();
    const float GL = meta.G[CB - 1];
    const float dec = __expf(GL);
#pragma unroll
    for (int i = 0; i < C::CPW * C::NT; ++i) S[i] *= dec;
    state_update<T, typename C::TD, typename C::TD, C::NT, C::CPW>(S, Xs, Ys, C::CPW * w * 16, meta.x, lane);
    Gs += GL;
    __syncthreads();
  };
  // A sequence's first chunk holds its replay rows (looked up one by one):
  // it is summed on its own before the others.
  int cf = c0;
  if (c0 == 0 && sq.n_rep > 0) {
    ChunkSrc<T, D> cs;
    Vec16 px[C::NV], py[C::NV];
    cs.resolve(sq, 0, replay_row, g, H, h, t, t < CB ? t : -1);
    fetch<T, D>(px, k, cs, H, h, t, ROW_REPLAY);
    fetch<T, D>(py, v, cs, H, h, t, ROW_REPLAY);
    sum_chunk(px, py, cs.gv, [] {});
    cf = 1;
  }
  // The other chunks hold own rows and padding only, whose addresses need no
  // lookup: every load is issued unconditionally (padding reads the zero
  // row; past the block's end its last chunk is requested again), so the
  // count of outstanding loads is the same on every path and the wait before
  // a chunk's tiles are stored leaves the next chunk's loads in flight.  Two
  // chunks are in flight while one is summed.
  if (cf < c_end) {
    using SG = Stg<T, D, C::NTHR>;
    const auto fetch_own = [&](Vec16* px, Vec16* py, float& gv, int c) {
      c = min(c, c_end - 1);
#pragma unroll
      for (int i = 0; i < C::NV; ++i) {
        const int idx = t + i * C::NTHR;
        const int pos = c * CB + idx / SG::VPR, d0 = (idx % SG::VPR) * SG::VE;
        const int64_t off = (static_cast<int64_t>(sq.own_row + pos - sq.n_rep) * H + h) * D + d0;
        const bool in = pos < sq.n_tok;
        px[i].u = *reinterpret_cast<const uint4*>(in ? k + off : reinterpret_cast<const T*>(kZeroRow) + d0);
        py[i].u = *reinterpret_cast<const uint4*>(in ? v + off : reinterpret_cast<const T*>(kZeroRow) + d0);
      }
      const int pos = c * CB + lane;
      gv = *(pos < sq.n_tok ? g + static_cast<int64_t>(sq.own_row + pos - sq.n_rep) * H + h
                            : reinterpret_cast<const float*>(kZeroRow));
    };
    Vec16 pxa[C::NV], pya[C::NV], pxb[C::NV], pyb[C::NV];
    float ga, gb;
    fetch_own(pxa, pya, ga, cf);
    fetch_own(pxb, pyb, gb, cf + 1);
    // pairs of chunks, both halves unconditional (the same loads outstanding
    // at the loop's back edge as at its entry); an odd last chunk after
    int c = cf;
    for (; c + 1 < c_end; c += 2) {
      sum_chunk(pxa, pya, ga, [&] { fetch_own(pxa, pya, ga, c + 2); });
      sum_chunk(pxb, pyb, gb, [&] { fetch_own(pxb, pyb, gb, c + 3); });
    }
    if (c < c_end) sum_chunk(pxa, pya, ga, [] {});
  }
  state_store<D, C::CPW>(dSb + bi * D * D, S, w, lane);
  if (t == 0) gam[bi] = Gs;
}

// Where the initial states of a round's sequences are: S0 [n_seq, H, d, d],
// or (S0 null) rows of the boundary bank picked by the round's init index,
// -1 meaning a zero state.
struct InitSrc {
  const float* S0;
  const float* bank;
  const int32_t* idx;
};
// Head h of sequence li's initial state, or nullptr for a zero state.
__device__ inline const float* init_state(const InitSrc& is, int li, int H, int h, int64_t DD) {
  if (is.S0) return is.S0 + (static_cast<int64_t>(li) * H + h) * DD;
  const int i = is.idx[li];
  return i >= 0 ? is.bank + (static_cast<int64_t>(i) * H + h) * DD : nullptr;
}
// The same with the bank index already at hand (from the launch table).
__device__ inline const float* init_state(const InitSrc& is, const BlkInfo& bl, int H, int h, int64_t DD) {
  if (is.S0) return is.S0 + (static_cast<int64_t>(bl.li) * H + h) * DD;
  return bl.init_bank >= 0 ? is.bank + (static_cast<int64_t>(bl.init_bank) * H + h) * DD : nullptr;
}

// ---------------------------------------------------------------------------
// element-parallel chains over the blocks of every sequence
// ---------------------------------------------------------------------------
constexpr int SCAN_THR = 256;
// Blocks whose summaries a scan requests together: the chain is serial in
// the blocks, its loads are not.
constexpr int SCAN_PF = 8;
constexpr int DG_HEADS = 16;  // heads per workgroup of k_dg_carry
static_assert(SCAN_THR % DG_HEADS == 0, "head lanes split the workgroup");

template <int D>
__global__ __launch_bounds__(SCAN_THR) void k_fwd_blockscan(
    const int32_t* __restrict__ seq_tab, const int32_t* __restrict__ blk_tab, int H,
    const InitSrc is, const float* __restrict__ dSb, const float* __restrict__ gam,
    float* __restrict__ S_end, float* __restrict__ bank, float* __restrict__ S_final, int skip1) {
  constexpr int64_t SS4 = static_cast<int64_t>(D) * D / 4;
  constexpr int NSW = static_cast<int>(SS4 / SCAN_THR);
  const int li = blockIdx.x / NSW, part = blockIdx.x % NSW, h = blockIdx.y;
  const int64_t e4 = static_cast<int64_t>(part) * SCAN_THR + threadIdx.x;
  const int32_t* seq = seq_tab + li * SEQ_WORDS;
  const int b0 = seq[SEQ_BLK_OFF];
  // skip1: the last block's end state (the final state) comes from the block
  // kernel, and only the start states of the other blocks are chained
  const int nb = seq[SEQ_N_BLK] - (skip1 ? 1 : 0);
  if (nb == 0) return;
  const float* s0 = init_state(is, li, H, h, SS4 * 4);
  float4 s = s0 ? reinterpret_cast<const float4*>(s0)[e4] : make_float4(0.f, 0.f, 0.f, 0.f);
  for (int bg = b0; bg < b0 + nb; bg += SCAN_PF) {
    float4 x[SCAN_PF];
    float gm[SCAN_PF];
#pragma unroll
    for (int i = 0; i < SCAN_PF; ++i) {
      if (bg + i < b0 + nb) {
        const int64_t bi = static_cast<int64_t>(bg + i) * H + h;
        gm[i] = gam[bi];
        x[i] = reinterpret_cast<const float4*>(dSb)[bi * SS4 + e4];
      }
    }
#pragma unroll
    for (int i = 0; i < SCAN_PF; ++i) {
      const int b = bg + i;
      if (b < b0 + nb) {
        const int64_t bi = static_cast<int64_t>(b) * H + h;
        const float dec = __expf(gm[i]);
        s.x = dec * s.x + x[i].x;
        s.y = dec * s.y + x[i].y;
        s.z = dec * s.z + x[i].z;
        s.w = dec * s.w + x[i].w;
        reinterpret_cast<float4*>(S_end)[bi * SS4 + e4] = s;
        const int eb = blk_tab[b * BLK_WORDS + BLK_END_BANK];
        if (eb >= 0 && bank)
          reinterpret_cast<float4*>(bank)[(static_cast<int64_t>(eb) * H + h) * SS4 + e4] = s;
      }
    }
  }
  if (S_final && !skip1)
    reinterpret_cast<float4*>(S_final)[(static_cast<int64_t>(seq[SEQ_FINAL_LEAF]) * H + h) * SS4 + e4] = s;
}

__device__ inline float scan_block_sum(float x, float* red, int t) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
  __syncthreads();
  if ((t & 63) == 0) red[t >> 6] = x;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < SCAN_THR / 64; ++i) s += red[i];
  return s;
}

template <int D>
__global__ __launch_bounds__(SCAN_THR) void k_bwd_blockscan(
    const int32_t* __restrict__ seq_tab, const int32_t* __restrict__ blk_tab, int H,
    const float* __restrict__ dS_final, const float* __restrict__ dbank,
    const float* __restrict__ S_end, const float* __restrict__ U, const float* __restrict__ gam,
    float* __restrict__ dS_end, float* __restrict__ betap) {
  constexpr int64_t SS4 = static_cast<int64_t>(D) * D / 4;
  constexpr int NSW = static_cast<int>(SS4 / SCAN_THR);
  __shared__ float red[SCAN_THR / 64];
  const int li = blockIdx.x / NSW, part = blockIdx.x % NSW, h = blockIdx.y, t = threadIdx.x;
  const int64_t e4 = static_cast<int64_t>(part) * SCAN_THR + t;
  const int32_t* seq = seq_tab + li * SEQ_WORDS;
  const int b0 = seq[SEQ_BLK_OFF], nb = seq[SEQ_N_BLK];
  // The reverse-order kernel starts a sequence's last block from dS_final
  // and ends its first block with dS0; the forward-order kernel adds the last
  // block's boundary term <dS_final, S_final>.  Here: the end adjoints of
  // the other blocks, with the injections and boundary terms of requested
  // states at their ends.
  if (nb == 1) return;
  const float4* S4 = reinterpret_cast<const float4*>(S_end);
  float4 ds = reinterpret_cast<const float4*>(dS_final)[(static_cast<int64_t>(seq[SEQ_FINAL_LEAF]) * H + h) * SS4 + e4];
  for (int bg = b0 + nb - 1; bg > b0; bg -= SCAN_PF) {
    float4 u[SCAN_PF];
    float gm[SCAN_PF];
#pragma unroll
    for (int i = 0; i < SCAN_PF; ++i) {
      if (bg - i > b0) {
        const int64_t bi = static_cast<int64_t>(bg - i) * H + h;
        gm[i] = gam[bi];
        u[i] = reinterpret_cast<const float4*>(U)[bi * SS4 + e4];
      }
    }
#pragma unroll
    for (int i = 0; i < SCAN_PF; ++i) {
      const int b = bg - i;
      if (b <= b0) break;
      // ds: the adjoint at the end of block b -> at its start = the end of b - 1
      const float dec = __expf(gm[i]);
      ds.x = dec * ds.x + u[i].x;
      ds.y = dec * ds.y + u[i].y;
      ds.z = dec * ds.z + u[i].z;
      ds.w = dec * ds.w + u[i].w;
      const int64_t pi = static_cast<int64_t>(b - 1) * H + h;
      const int eb = blk_tab[(b - 1) * BLK_WORDS + BLK_END_BANK];
      float bsum = 0.f;
      if (eb >= 0) {  // uniform over the workgroup
        const float4 inj = reinterpret_cast<const float4*>(dbank)[(static_cast<int64_t>(eb) * H + h) * SS4 + e4];
        const float4 s = S4[pi * SS4 + e4];
        bsum = scan_block_sum(inj.x * s.x + inj.y * s.y + inj.z * s.z + inj.w * s.w, red, t);
        ds.x += inj.x;
        ds.y += inj.y;
        ds.z += inj.z;
        ds.w += inj.w;
      }
      if (t == 0) betap[pi * NSW + part] = bsum;
      reinterpret_cast<float4*>(dS_end)[pi * SS4 + e4] = ds;
    }
  }
}

// ---------------------------------------------------------------------------
// forward: outputs of the own rows of a block
// ---------------------------------------------------------------------------
template <typename T, int D>
struct FwdSmem {
  T Q[Tile<T, D>::SIZE];
  T K[Tile<T, D>::SIZE];
  T V[Tile<T, D>::SIZE];
  T A[Tile<T, CB>::SIZE];    // masked Q K^T
  ChunkMeta meta;  // x = exp(G_last - G), y = exp(G)
};

template <typename T, int D>
__global__ __launch_bounds__((Cfg<T, D>::NTHR), (Cfg<T, D>::WPE)) void k_fwd_block(
    const int32_t* __restrict__ seq_tab, const int32_t* __restrict__ blk_tab,
    const int32_t* __restrict__ blk_launch,
    const int32_t* __restrict__ replay_row, int H, float scale, const T* __restrict__ q,
    const T* __restrict__ k, const T* __restrict__ v, const float* __restrict__ g,
    const InitSrc is, const float* __restrict__ S_end, T* __restrict__ o, float* __restrict__ S_final) {
  using C = Cfg<T, D>;
  constexpr int NS = C::CPW * C::NT;
  __shared__ FwdSmem<T, D> sm;
  const BlkInfo bl = blk_info(blk_launch, blockIdx.x / H);
  const int b = bl.b, h = blockIdx.x % H, t = threadIdx.x, lane = t & 63;
  const int w = wave_id(t);
  const int col0 = C::CPW * w * 16;
  const SeqInfo sq = bl.sq;
  const int c0 = bl.c0, c_end = c0 + bl.nc;
  const int64_t DD = static_cast<int64_t>(D) * D;
  // the first chunk's rows are requested before the start state
  ChunkSrc<T, D> cs;
  Vec16 pq[C::NV], pk[C::NV], pv[C::NV];
  cs.resolve(sq, c0, replay_row, g, H, h, t, t < CB ? t : -1);
  fetch<T, D>(pq, q, cs, H, h, t, ROW_OWN);
  fetch<T, D>(pk, k, cs, H, h, t, ROW_REPLAY);
  fetch<T, D>(pv, v, cs, H, h, t, ROW_REPLAY);
  f32x4 S[NS];  // S : rows (dk), columns (dv) of the wave's strips
  // the start state, staged through the (still unused) tiles in two halves
  static_assert(D / 2 * (D + 4) * 4 <= static_cast<int>(sizeof(FwdSmem<T, D>) - sizeof(ChunkMeta)),
                "half a state fits the tiles");
  state_via_lds<D, C::CPW, C::NTHR, 2>(S, reinterpret_cast<float*>(&sm.Q[0]),
                                       bl.idx == 0 ? init_state(is, bl, H, h, DD)
                                                   : S_end + (static_cast<int64_t>(b - 1) * H + h) * DD,
                                       false, w, lane, t);
  for (int c = c0; c < c_end; ++c) {
    if (t < CB) {
      float Gt, GLw;
      meta_publish(sm.meta, cs, t, Gt, GLw);
      sm.meta.x[t] = __expf(GLw - Gt);
      sm.meta.y[t] = __expf(Gt);
    }
    const ChunkRows cur = cs.cr;
    put<T, D>(sm.Q, pq, nullptr, t);
    put<T, D>(sm.K, pk, nullptr, t);
    put<T, D>(sm.V, pv, nullptr, t);
    __syncthreads();
    const float GL = sm.meta.G[CB - 1];
    // the next chunk's rows are loaded one tile at a time between the phases
    // of this chunk, so that the loads do not queue up behind each other
    const bool more = c + 1 < c_end;
    if (more) {
      cs.resolve(sq, c + 1, replay_row, g, H, h, t, t < CB ? t : -1);
      fetch<T, D>(pq, q, cs, H, h, t, ROW_OWN);
    }
    // A = (Q K^T) * exp(G_i - G_j) [j <= i]; wave w computes row block w
    if (w < 3) score_block<T, D>(sm.A, sm.Q, sm.K, sm.meta.G, 1.f, w, lane);
    if (more) fetch<T, D>(pk, k, cs, H, h, t, ROW_REPLAY);
    __syncthreads();
    // O[:, wave columns] = scale * (diag(exp(G)) Q S_c + A V), products with
    // swapped operands: lane (g, i) holds row 16 it + i, columns
    // col0 + 16 j + 4g .. + 3
    PackedState<T, C::NT, C::CPW> ps;
    ps.pack(S);
#pragma unroll 1
    for (int it = 0; it < CB / 16; ++it) {
      if (it == 1 && more) fetch<T, D>(pv, v, cs, H, h, t, ROW_REPLAY);
      f32x4 acc[C::CPW];
#pragma unroll
      for (int j = 0; j < C::CPW; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
      regb_rows_packed<T, typename C::TD, C::NT, C::CPW, true, true>(acc, sm.Q, it * 16, ps, lane);
      const int m = it * 16 + (lane & 15);
      {
        const float e = sm.meta.y[m];
#pragma unroll
        for (int j = 0; j < C::CPW; ++j) acc[j] *= e;
      }
      tile_cols<T, typename C::TA, false, typename C::TD, C::CPW, true, true>(
          acc, sm.A, it * 16, sm.V, col0, 0, (it + 1) * 16, lane);
      const int rk = cur.fast ? 0 : sm.meta.rowk[m];
      if (cur.fast || (rk & 3) == ROW_OWN) {
        const int64_t row = cur.fast ? static_cast<int64_t>(cur.row0) + m : (rk >> 2);
        T* dst = o + (row * H + h) * D + col0 + 4 * (lane >> 4);
#pragma unroll
        for (int j = 0; j < C::CPW; ++j) Vec4<T>::store(dst + 16 * j, acc[j] * scale);
      }
    }
    // S_{c+1} = exp(G_last) S_c + K^T diag(exp(G_last - G)) V
    const float dec = __expf(GL);
#pragma unroll
    for (int i = 0; i < NS; ++i) S[i] *= dec;
    state_update<T, typename C::TD, typename C::TD, C::NT, C::CPW>(S, sm.K, sm.V, col0, sm.meta.x, lane);
    __syncthreads();
  }
  // the last block of a sequence: its end state is the final state
  if (S_final && bl.idx == bl.n_blk - 1)
    state_store<D, C::CPW>(S_final + (static_cast<int64_t>(bl.final_leaf) * H + h) * DD, S, w, lane);
}

// ---------------------------------------------------------------------------
// backward, forward order (needs S_c: chunks forward).  One workgroup of two
// halves per (block, head), sharing double-buffered chunk tiles in LDS:
//   waves 0..3 (side 0): dq = scale diag(exp(G)) dO S_c^T + dA K and q.dq
//                        per row, holding S^T (rows dv, columns dk);
//   waves 4..7 (side 1): every load and LDS write of the chunk tiles and of
//                        the row table; the masked score
//                        dA = scale (dO V^T) exp(G_i - G_j) [j <= i]
//                        (waves 4..6; wave 7 sums the previous chunk's q.dq);
//                        and the block's adjoint summary
//                        U_b = sum_t exp(G_t^blk) scale q_t dO_t^T, with
//                        G_t^blk the inclusive log-decay from the block start
//                        to row t, which the adjoint chain over blocks needs
//                        (never for a sequence's first block).
// Per chunk c, between two workgroup barriers each: (1) side 0 converts
// S_c^T once to MFMA operands and advances S^T, side 1 forms dA; (2) side 0
// forms the dq rows from the converted S_c^T, side 1 advances U_b, writes
// chunk c + 1 (loaded during chunk c - 1) to the other buffer and requests
// chunk c + 2.
// ---------------------------------------------------------------------------
template <typename T, int D>
struct BfMeta {
  ChunkMeta m;              // x = exp(G_last - G), y = exp(G) * scale
  alignas(16) float u[CB];  // exp(G_t^blk) * scale
};
template <typename T, int D>
struct BfSmem {
  using C = Cfg<T, D>;
  T dO[2][Tile<T, D>::SIZE];
  T V[2][Tile<T, D>::SIZE];
  T K[2][Tile<T, D>::SIZE];
  T Q[2][Tile<T, D>::SIZE];  // own rows
  T dA[Tile<T, CB>::SIZE];   // scale * (dO V^T) masked
  BfMeta<T, D> meta[2];
  float rq[C::NW][CB];
  float red[2 * C::NW];
};

template <typename T, int D>
__global__ __launch_bounds__((2 * Cfg<T, D>::NTHR), (Cfg<T, D>::WPE)) void k_bwd_fwdorder(
    const int32_t* __restrict__ seq_tab, const int32_t* __restrict__ blk_tab,
    const int32_t* __restrict__ blk_launch,
    const int32_t* __restrict__ replay_row, int H, float scale, const T* __restrict__ q,
    const T* __restrict__ k, const T* __restrict__ v, const float* __restrict__ g,
    const T* __restrict__ dO, const InitSrc is, const float* __restrict__ S_end,
    T* __restrict__ dq, float* __restrict__ rq_out, const float* __restrict__ dS_final,
    float* __restrict__ betap, float* __restrict__ U) {
  using C = Cfg<T, D>;
  constexpr int NTH = 2 * C::NTHR;
  constexpr int NS = C::CPW * C::NT;
  constexpr int NIT = CB / 16;
  __shared__ BfSmem<T, D> sm;
  const BlkInfo bl = blk_info(blk_launch, blockIdx.x / H);
  const int b = bl.b, h = blockIdx.x % H, t = threadIdx.x, lane = t & 63;
  const int w = wave_id(t);
  const int side = w >= C::NW;
  const int ws = w - side * C::NW;       // wave within its half
  const int t1 = t - side * C::NTHR;     // thread within its half
  const int col0 = C::CPW * ws * 16;
  const SeqInfo sq = bl.sq;
  const int c0 = bl.c0, c_end = c0 + bl.nc;
  const int64_t DD = static_cast<int64_t>(D) * D;
  const bool want_u = bl.idx > 0;
  // side 1: the first chunk's rows are requested before the start state
  ChunkSrc<T, D> cs;
  Vec16 pq[C::NV], pk[C::NV], pv[C::NV], pd[C::NV];
  if (side) {
    cs.resolve(sq, c0, replay_row, g, H, h, t1, t1 < CB ? t1 : -1);
    fetch<T, D>(pq, q, cs, H, h, t1, ROW_OWN);
    fetch<T, D>(pk, k, cs, H, h, t1, ROW_REPLAY);
    fetch<T, D>(pv, v, cs, H, h, t1, ROW_REPLAY);
    fetch<T, D>(pd, dO, cs, H, h, t1, ROW_OWN);
  }
  f32x4 S[NS];  // side 0: S^T in its column strips; side 1: U_b in its column strips
  // the start state, staged through the (still unused) tiles
  using BfS = BfSmem<T, D>;
  static_assert(D * (D + 4) * 4 <= static_cast<int>(offsetof(BfS, dA)), "state fits the tiles");
  float* stage = reinterpret_cast<float*>(&sm.dO[0][0]);
  state_via_lds<D, C::CPW, NTH, 1>(S, stage,
                                   bl.idx == 0 ? init_state(is, bl, H, h, DD)
                                               : S_end + (static_cast<int64_t>(b - 1) * H + h) * DD,
                                   true, ws, lane, t, !side);
  float Gs = 0.f;  // wave 4, lane = row: log-decay from the block start to the chunk start
  // side 1 writes a chunk (its row table and tiles) to buffer nb
  auto put_chunk = [&](int nb) {
    if (t1 < CB) {
      float Gt, GLw;
      meta_publish(sm.meta[nb].m, cs, t1, Gt, GLw);
      sm.meta[nb].m.x[t1] = __expf(GLw - Gt);
      sm.meta[nb].m.y[t1] = __expf(Gt) * scale;
      sm.meta[nb].u[t1] = __expf(Gs + Gt) * scale;
      Gs += GLw;
    }
    put<T, D>(sm.dO[nb], pd, nullptr, t1);
    put<T, D>(sm.V[nb], pv, nullptr, t1);
    put<T, D>(sm.K[nb], pk, nullptr, t1);
    put<T, D>(sm.Q[nb], pq, nullptr, t1);
  };
  if (side) {
#pragma unroll
    for (int i = 0; i < NS; ++i) S[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    put_chunk(0);
    if (c0 + 1 < c_end) {
      cs.resolve(sq, c0 + 1, replay_row, g, H, h, t1, t1 < CB ? t1 : -1);
      fetch<T, D>(pq, q, cs, H, h, t1, ROW_OWN);
      fetch<T, D>(pk, k, cs, H, h, t1, ROW_REPLAY);
      fetch<T, D>(pv, v, cs, H, h, t1, ROW_REPLAY);
      fetch<T, D>(pd, dO, cs, H, h, t1, ROW_OWN);
    }
  }
  __syncthreads();
  // The halves run loops of their own (the branch is uniform per wave), each
  // with two workgroup barriers per chunk, so that neither half's registers
  // are held across the other's code.  The lane index is hidden from the
  // optimiser inside the loops: LDS addresses are formed per chunk instead
  // of being held across the loop.
  if (!side) {
    for (int c = c0; c < c_end; ++c) {
      const int bf = (c - c0) & 1;
      const ChunkMeta& mt = sm.meta[bf].m;
      int ln = lane;
      asm volatile("" : "+v"(ln));
      // (1) S_c^T packed once into MFMA operands for the rows below, then
      // S^T <- exp(G_last) S^T + V^T diag(exp(G_last - G)) K
      PackedState<T, C::NT, C::CPW> ps;
      ps.pack(S);
      const float dec = __expf(mt.G[CB - 1]);
#pragma unroll
      for (int i = 0; i < NS; ++i) S[i] *= dec;
      state_update<T, typename C::TD, typename C::TD, C::NT, C::CPW>(S, sm.V[bf], sm.K[bf], col0, mt.x, ln);
      __syncthreads();
      // (2) dq[:, wave columns] = scale diag(exp(G)) dO S_c^T + dA K ; partial
      // q.dq.  Products with swapped operands: lane (g, i) holds row
      // 16 it + i, columns col0 + 16 j + 4g .. + 3
      const ChunkRows cur = chunk_rows(sq, c);
      const int g4 = 4 * (ln >> 4);
#pragma unroll 1
      for (int it = 0; it < NIT; ++it) {
        f32x4 acc[C::CPW];
#pragma unroll
        for (int j = 0; j < C::CPW; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
        regb_rows_packed<T, typename C::TD, C::NT, C::CPW, true>(acc, sm.dO[bf], it * 16, ps, ln);
        const int m = it * 16 + (ln & 15);
        {
          const float e = mt.y[m];
#pragma unroll
          for (int j = 0; j < C::CPW; ++j) acc[j] *= e;
        }
        tile_cols<T, typename C::TA, false, typename C::TD, C::CPW, true>(acc, sm.dA, it * 16, sm.K[bf],
                                                                         col0, 0, (it + 1) * 16, ln);
        float qd = 0.f;
#pragma unroll
        for (int j = 0; j < C::CPW; ++j) {
          const f32x4 qv = Vec4<T>::load(sm.Q[bf] + C::TD::at(m, col0 + 16 * j + g4));
#pragma unroll
          for (int r = 0; r < 4; ++r) qd += qv[r] * acc[j][r];
        }
        qd = group_sum4(qd);
        if (ln < 16) sm.rq[ws][m] = qd;
        const int rk = cur.fast ? 0 : mt.rowk[m];
        if (cur.fast || (rk & 3) == ROW_OWN) {
          const int64_t row = cur.fast ? static_cast<int64_t>(cur.row0) + m : (rk >> 2);
          T* dst = dq + (row * H + h) * D + col0 + g4;
#pragma unroll
          for (int j = 0; j < C::CPW; ++j) Vec4<T>::store(dst + 16 * j, acc[j]);
        }
      }
      __syncthreads();
    }
    // The last block of a sequence ends with S_final (S^T is held here):
    // <dS_final, S_final> is its boundary term of dg, the first of the
    // block's NSW partial sums (threads t < NSW are in this half).
    if (bl.idx == bl.n_blk - 1) {
      constexpr int NSW = D * D / 4 / SCAN_THR;
      static_assert(NSW <= 64 * C::NW, "partial sums written by side 0");
      const float dot = state_dot_via_lds<D, C::CPW, NTH>(
          S, stage, dS_final + (static_cast<int64_t>(bl.final_leaf) * H + h) * DD, true, ws, lane, t,
          sm.red, true);
      if (t < NSW) betap[(static_cast<int64_t>(b) * H + h) * NSW + t] = t == 0 ? dot : 0.f;
    }
  } else {
    for (int c = c0; c < c_end; ++c) {
      const int bf = (c - c0) & 1;
      int ln = lane;
      asm volatile("" : "+v"(ln));
      // (1) the masked score dA (waves 4..6); wave 7: q.dq of the previous
      // chunk's rows (lane = row)
      if (ws < 3) {
        score_block<T, D>(sm.dA, sm.dO[bf], sm.V[bf], sm.meta[bf].m.G, scale, ws, ln);
      } else if (c > c0) {
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < C::NW; ++i) s += sm.rq[i][ln];
        rq_out[((static_cast<int64_t>(sq.chunk_off) + c - 1) * CB + ln) * H + h] = s;
      }
      __syncthreads();
      // (2) U_b += Q^T diag(exp(G^blk) scale) dO; then the next chunk to the
      // other buffer, and the one after it requested
      if (want_u)
        state_update<T, typename C::TD, typename C::TD, C::NT, C::CPW>(S, sm.Q[bf], sm.dO[bf], col0,
                                                                       sm.meta[bf].u, ln);
      if (c + 1 < c_end) {
        put_chunk(bf ^ 1);
        if (c + 2 < c_end) {
          int tt = t1;
          asm volatile("" : "+v"(tt));
          cs.resolve(sq, c + 2, replay_row, g, H, h, tt, tt < CB ? tt : -1);
          fetch<T, D>(pq, q, cs, H, h, tt, ROW_OWN);
          fetch<T, D>(pk, k, cs, H, h, tt, ROW_REPLAY);
          fetch<T, D>(pv, v, cs, H, h, tt, ROW_REPLAY);
          fetch<T, D>(pd, dO, cs, H, h, tt, ROW_OWN);
        }
      }
      __syncthreads();
    }
    if (ws == C::NW - 1) {
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < C::NW; ++i) s += sm.rq[i][lane];
      rq_out[((static_cast<int64_t>(sq.chunk_off) + c_end - 1) * CB + lane) * H + h] = s;
    }
    if (want_u) state_store<D, C::CPW>(U + (static_cast<int64_t>(b) * H + h) * DD, S, ws, lane);
    // (this half joins the staging and the sum of side 0's boundary term)
    if (bl.idx == bl.n_blk - 1)
      state_dot_via_lds<D, C::CPW, NTH>(S, stage, dS_final + (static_cast<int64_t>(bl.final_leaf) * H + h) * DD,
                                        true, ws, lane, t, sm.red, false);
  }
}

// ---------------------------------------------------------------------------
// backward, reverse order (needs dS_{c+1}: chunks backward).  One workgroup of
// two halves per (block, head), sharing the chunk tiles in LDS:
//   waves 0..3 (side 0): dv = diag(exp(G_last - G)) K dS + scale A^T dO,
//                        holding dS;
//   waves 4..7 (side 1): dk = diag(exp(G_last - G)) V dS^T + dA^T Q, plus
//                        k.dk per row and the local suffix sums of dg.
// The adjoint recurrence
//   dS_c = exp(G_last) dS_{c+1} + Q^T diag(exp(G) scale) dO
// runs in side 0 only (bf16): after each update side 0 converts dS once to
// bf16 MFMA operands and writes them, transposed, to LDS, from where side 1
// reads its operands of V dS^T with the transpose read during the next
// score phase.  In fp32 each half runs the recurrence in its own layout.
// ---------------------------------------------------------------------------
// Chunk tiles.  bf16: Q and K are double-buffered (the next chunk's are
// written during the score phase), V and dO single-buffered (written after
// every wave is done with the current ones); the packed transposed adjoint
// takes the room of the second V, dO pair, next to two score tiles.  fp32:
// all four double-buffered, the halves taking turns with one score tile
// (score A, dv rows, score dA, dk rows).
enum { TQ = 0, TK = 1, TV = 2, TDO = 3 };

// [D][D] bf16 tile of the adjoint's transpose (rows dv, columns dk), each
// row padded by 16 bytes like the chunk tiles.
template <int D>
struct AdjT {
  static constexpr int LD = D + 8;
  static constexpr int SIZE = D * LD;
  __device__ static inline int at(int r, int c) { return r * LD + c; }
  __device__ static inline int base(int r0, int c0) { return r0 * LD + c0; }
  __device__ static inline int lane(int ri, int ci) { return ri * LD + ci; }
};

// Q and dO are read transposed (state update, the products with the score
// tiles) and take the swizzled layout where it exists; K and V are read
// k-contiguous only.
template <typename T, int D, bool SH = (sizeof(T) == 2)>
struct BrTiles;
template <typename T, int D>
struct BrTiles<T, D, false> {
  using LQ = Tile<T, D>;
  using LK = Tile<T, D>;
  T tile[2][4][Tile<T, D>::SIZE];
  static constexpr int STAGE_BYTES = 4 * Tile<T, D>::SIZE * static_cast<int>(sizeof(T));
  __device__ inline T* at(int bf, int which) { return tile[bf][which]; }
  __device__ inline float* stage() { return reinterpret_cast<float*>(&tile[1][0][0]); }
};
template <typename T, int D>
struct BrTiles<T, D, true> {
  using LQ = TileX<T, D>;  // Q and dO
  using LK = Tile<T, D>;   // K and V
  T q0[LQ::SIZE];
  T k0[LK::SIZE];
  T q1[LQ::SIZE];          // q1, k1 and dt form the staging area
  T k1[LK::SIZE];
  T dt[AdjT<D>::SIZE];
  T v[LK::SIZE];
  T dO[LQ::SIZE];
  static constexpr int STAGE_BYTES = (LQ::SIZE + LK::SIZE + AdjT<D>::SIZE) * static_cast<int>(sizeof(T));
  __device__ inline T* at(int bf, int which) {
    return which == TQ ? (bf ? q1 : q0) : which == TK ? (bf ? k1 : k0) : which == TV ? v : dO;
  }
  __device__ inline float* stage() { return reinterpret_cast<float*>(q1); }
};

template <typename T, int D>
struct BrSmem {
  using C = Cfg<T, D>;
  static constexpr bool SH = sizeof(T) == 2;  // one adjoint, shared through LDS
  static constexpr int NP = SH ? 2 : 1;
  // score tiles: rows padded by 8 bytes in bf16 (fragment reads stay
  // conflict-free, and the workgroup's LDS fits 160 KiB)
  using TP = Tile<T, CB, false, SH ? 8 : 16>;
  BrTiles<T, D> tl;
  T P[NP][TP::SIZE];               // A = Q K^T masked; dA = scale (dO V^T) masked
  ChunkMeta meta[2];               // x = exp(G_last - G), y = exp(G) * scale
  float rk[C::NW][CB];             // partial k.dk of each row, per wave
  float rqb[2][CB];                // q.dq of the rows of a chunk (buffer as meta)
};

// Side 1's B operands of V dS^T from the transposed adjoint in LDS: the same
// values as PackedState::pack of dS^T held in side 1's accumulator layout.
template <int D, int NT, int CPW>
__device__ inline void adj_load(PackedState<bf16, NT, CPW>& ps, const bf16* dt, int w, int lane) {
#pragma unroll
  for (int j = 0; j < CPW; ++j)
#pragma unroll
    for (int kt = 0; kt < NT; kt += 2)
      ps.p[j][kt / 2] = Frag<bf16>::km<AdjT<D>>(dt, 16 * kt, 16 * (CPW * w + j), lane);
}

// Side 0's packed adjoint written transposed: lane (g, i) of strip j holds
// dS[16 kt + 4g + 0..3][16 (CPW w + j) + i] (and the next 16 rows), four
// consecutive elements of row dv = 16 (CPW w + j) + i of the transpose.
template <int D, int NT, int CPW>
__device__ inline void adj_store(bf16* dt, const PackedState<bf16, NT, CPW>& ps, int w, int lane) {
  const int r = 16 * CPW * w + (lane & 15), c = 4 * (lane >> 4);
#pragma unroll
  for (int j = 0; j < CPW; ++j)
#pragma unroll
    for (int kt = 0; kt < NT; kt += 2) {
      const bf16x8 v = ps.p[j][kt / 2];
      bf16x4 lo, hi;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[e] = v[e];
        hi[e] = v[4 + e];
      }
      *reinterpret_cast<bf16x4*>(dt + AdjT<D>::at(r + 16 * j, 16 * kt + c)) = lo;
      *reinterpret_cast<bf16x4*>(dt + AdjT<D>::at(r + 16 * j, 16 * kt + 16 + c)) = hi;
    }
}

// Output rows of one chunk (tiles of buffer bf) for one half of the
// workgroup, from the adjoint's B operands ps.  The products run with their
// operands swapped, so that lane (g, i) of a wave holds row 16 jt + i of the
// output at columns col0 + 16 j + 4g .. + 3: one 8-byte (bf16) or 16-byte
// (float) store per strip, one row per lane.  Then the adjoint update: in
// bf16 by side 0 only, which also converts the new adjoint for the next
// chunk (ps) and publishes it (when `more`); in fp32 by each half.
template <typename T, int D, int SIDE>
__device__ __forceinline__ void bwd_revorder_rows(
    BrSmem<T, D>& sm, int bf, f32x4* dS, PackedState<T, Cfg<T, D>::NT, Cfg<T, D>::CPW>& ps,
    const ChunkRows& cur, const SeqInfo& sq, int c, bool more, int H, int h, float scale, float GL,
    int w, int lane, T* __restrict__ dk, T* __restrict__ dv, float* __restrict__ rep_grad) {
  using C = Cfg<T, D>;
  constexpr bool SH = BrSmem<T, D>::SH;
  constexpr int NS = C::CPW * C::NT;
  constexpr int RG = 2 * D + 1;
  constexpr bool side = SIDE == 1;
  const int col0 = C::CPW * w * 16;
  const T* PT = sm.P[BrSmem<T, D>::NP == 2 ? SIDE : 0];  // transposed score tile
  using LQ = typename BrTiles<T, D>::LQ;  // Q and dO
  using LK = typename BrTiles<T, D>::LK;  // K and V
  const T* Q = sm.tl.at(bf, TQ);
  const T* K = sm.tl.at(bf, TK);
  const T* V = sm.tl.at(bf, TV);
  const T* dOt = sm.tl.at(bf, TDO);
  const ChunkMeta& mt = sm.meta[bf];
  const int g4 = 4 * (lane >> 4);
  // the chunk's 64 rows of the output (row0 may precede the sequence's own
  // rows when the chunk starts with replay rows; only own rows are stored)
  const __amdgpu_buffer_rsrc_t out_rsrc =
      buffer_rsrc((side ? dk : dv) + static_cast<int64_t>(cur.row0) * H * D,
                  static_cast<uint32_t>(CB * H * D * sizeof(T)));
  if constexpr (!SH) ps.pack(dS);
  // the row factors of the lane's four rows, read before the loop
  float xr[CB / 16];
#pragma unroll
  for (int jt = 0; jt < CB / 16; ++jt) xr[jt] = mt.x[jt * 16 + (lane & 15)];
#pragma unroll 1
  for (int jt = 0; jt < CB / 16; ++jt) {
    const int m = jt * 16 + (lane & 15);
    // side 1: the K values of the lane's row and columns, requested first
    typename Vec4Raw<T>::V kraw[C::CPW];
    if (side) {
#pragma unroll
      for (int j = 0; j < C::CPW; ++j) kraw[j] = Vec4Raw<T>::load(K + LK::at(m, col0 + 16 * j + g4));
    }
    // side 0: dv = diag(x) K dS + scale A^T dO ; side 1: dk = diag(x) V dS^T + dA^T Q
    // (A and dA vanish above the diagonal, so the transposed products start at row block jt)
    f32x4 acc[C::CPW], ad[C::CPW];
#pragma unroll
    for (int j = 0; j < C::CPW; ++j) {
      acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
      ad[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    regb_rows_packed<T, LK, C::NT, C::CPW, true, true>(acc, side ? V : K, jt * 16, ps, lane);
    const int k0 = (jt * 16 / Frag<T>::KSTEP) * Frag<T>::KSTEP;
    tile_cols<T, typename BrSmem<T, D>::TP, false, LQ, C::CPW, true, true>(
        ad, PT, jt * 16, side ? Q : dOt, col0, k0, CB, lane);
    float e = xr[0];
#pragma unroll
    for (int i = 1; i < CB / 16; ++i) e = jt == i ? xr[i] : e;
    const float f = side ? 1.f : scale;
#pragma unroll
    for (int j = 0; j < C::CPW; ++j) acc[j] = acc[j] * e + f * ad[j];
    if (side) {
      // k.dk of row m over the wave's columns (the waves' partial sums are
      // added by the suffix step)
      float kd = 0.f;
#pragma unroll
      for (int j = 0; j < C::CPW; ++j) {
        const f32x4 kv = Vec4Raw<T>::widen(kraw[j]);
#pragma unroll
        for (int r = 0; r < 4; ++r) kd += kv[r] * acc[j][r];
      }
      kd = group_sum4(kd);
      if (lane < 16) sm.rk[w][m] = kd;
    }
    // Own rows: an own row at position m of the chunk is physical row
    // row0 + m, so every lane stores at its offset from row0 (through a
    // resource over the chunk's 64 rows) and a lane whose row is not own
    // stores nothing.  The stores are thus the same on every path, which lets
    // the wait for the next chunk's loads skip them.
    const int kind = cur.fast ? static_cast<int>(ROW_OWN) : (mt.rowk[m] & 3);
    {
      const uint32_t off = kind == ROW_OWN
                               ? static_cast<uint32_t>(((m * H + h) * D + col0 + g4) * static_cast<int>(sizeof(T)))
                               : BUF_DROP;
#pragma unroll
      for (int j = 0; j < C::CPW; ++j)
        BufVec4<T>::store(out_rsrc, off + static_cast<uint32_t>(16 * j * sizeof(T)), acc[j]);
    }
    if (kind == ROW_REPLAY) {
      // rows of 2D + 1 floats: no vector alignment
      float* dst = rep_grad + ((static_cast<int64_t>(sq.replay_off) + c * CB + m) * H + h) * RG +
                   (side ? 0 : D) + col0 + g4;
#pragma unroll
      for (int j = 0; j < C::CPW; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[16 * j + r] = acc[j][r];
    }
  }
  if constexpr (SH) {
    if (side) return;
  }
  // side 0: dS   <- exp(G_last) dS   + Q^T  diag(exp(G) scale) dO
  // side 1: dS^T <- exp(G_last) dS^T + dO^T diag(exp(G) scale) Q   (fp32)
  const float dec = __expf(GL);
#pragma unroll
  for (int i = 0; i < NS; ++i) dS[i] *= dec;
  if (!side)
    state_update<T, LQ, LQ, C::NT, C::CPW, true>(dS, Q, dOt, col0, mt.y, lane);
  else
    state_update<T, LQ, LQ, C::NT, C::CPW, true>(dS, dOt, Q, col0, mt.y, lane);
  if constexpr (SH) {
    if (more) {
      ps.pack(dS);
      adj_store<D, C::NT, C::CPW>(sm.tl.dt, ps, w, lane);
    }
  }
}

template <typename T, int D>
__global__ __launch_bounds__((2 * Cfg<T, D>::NTHR), (Cfg<T, D>::WPE)) void k_bwd_revorder(
    const int32_t* __restrict__ seq_tab, const int32_t* __restrict__ blk_tab,
    const int32_t* __restrict__ blk_launch, const int32_t* __restrict__ replay_row, int H,
    float scale, const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
    const float* __restrict__ g, const T* __restrict__ dO, const float* __restrict__ dS_end,
    const float* __restrict__ rq, T* __restrict__ dk, T* __restrict__ dv,
    float* __restrict__ dg, float* __restrict__ rep_grad, float* __restrict__ Rb,
    const float* __restrict__ dS_final, float* __restrict__ dS0) {
  using C = Cfg<T, D>;
  constexpr int NTH = 2 * C::NTHR;
  constexpr bool SH = BrSmem<T, D>::SH;
  using SG = Stg<T, D, NTH>;
  using LQ = typename BrTiles<T, D>::LQ;  // Q and dO
  using LK = typename BrTiles<T, D>::LK;  // K and V
  constexpr int RG = 2 * D + 1;
  __shared__ BrSmem<T, D> sm;
  const BlkInfo bl = blk_info(blk_launch, blockIdx.x / H);
  const int b = bl.b, h = blockIdx.x % H, tid = threadIdx.x;
  const int side = tid >= C::NTHR ? 1 : 0;  // uniform over a wave
  const int t = tid - side * C::NTHR, lane = tid & 63, w = wave_id(t);
  const int li = bl.li;
  const SeqInfo sq = bl.sq;
  const int c0 = bl.c0, c_last = c0 + bl.nc - 1;
  const int64_t DD = static_cast<int64_t>(D) * D;
  // a sequence's last block starts from dS_final, its first block ends with dS0
  const bool last = bl.idx == bl.n_blk - 1;
  const float* dS_in = last ? dS_final + (static_cast<int64_t>(bl.final_leaf) * H + h) * DD
                            : dS_end + (static_cast<int64_t>(b) * H + h) * DD;
  static_assert(StateStage<D>::BYTES <= BrTiles<T, D>::STAGE_BYTES,
                "state staging fits the tiles that are free before the loop");
  float* stg = sm.tl.stage();
  // Side 0, wave 3 (lane = row of the chunk) publishes each chunk's row table
  // and decay factors during the score phase of the chunk before it, in which
  // it computes no score block.
  const bool pw = side == 0 && w == 3;
  const int mrow = pw ? lane : -1;
  const auto publish = [&](const ChunkSrc<T, D, NTH>& src, int bf) {
    float Gt, GLw;
    meta_publish(sm.meta[bf], src, lane, Gt, GLw);
    sm.meta[bf].x[lane] = __expf(GLw - Gt);
    sm.meta[bf].y[lane] = __expf(Gt) * scale;
  };
  // The last chunk of the block goes into buffer 0, two tiles at a time.
  ChunkSrc<T, D, NTH> cs;
  Vec16 pa[SG::NV], pb[SG::NV];
  // The first chunk's four tiles and dS_end (read once into the staging
  // area, free until the first chunk's score) are requested together: one
  // memory round trip before the loop.
  cs.resolve(sq, c_last, replay_row, g, H, h, tid, mrow);
  {
    Vec16 pc[SG::NV], pd[SG::NV];
    fetch<T, D, NTH>(pa, q, cs, H, h, tid, ROW_OWN);
    fetch<T, D, NTH>(pb, k, cs, H, h, tid, ROW_REPLAY);
    fetch<T, D, NTH>(pc, v, cs, H, h, tid, ROW_REPLAY);
    fetch<T, D, NTH>(pd, dO, cs, H, h, tid, ROW_OWN);
    state_to_lds<D, NTH>(stg, dS_in, tid);
    put<T, D, NTH, LQ>(sm.tl.at(0, TQ), pa, nullptr, tid);
    put<T, D, NTH, LK>(sm.tl.at(0, TK), pb, nullptr, tid);
    put<T, D, NTH, LK>(sm.tl.at(0, TV), pc, nullptr, tid);
    put<T, D, NTH, LQ>(sm.tl.at(0, TDO), pd, nullptr, tid);
  }
  if (pw) publish(cs, 0);
  ChunkRows cur_next = cs.cr;
  __syncthreads();
  // side 0: dS   rows (dk), columns (dv) of the wave's strips
  // side 1: dS^T rows (dv), columns (dk) of the wave's strips (bf16: only
  // to form the first chunk's operands)
  f32x4 dS[C::CPW * C::NT];
  state_from_lds<D, C::CPW>(dS, stg, side == 1, w, lane);
  PackedState<T, C::NT, C::CPW> ps;
  if constexpr (SH) ps.pack(dS);
  // the first two tiles of the chunk before it
  if (c_last > c0) {
    cs.resolve(sq, c_last - 1, replay_row, g, H, h, tid, mrow);
    fetch<T, D, NTH>(pa, q, cs, H, h, tid, ROW_OWN);
    fetch<T, D, NTH>(pb, k, cs, H, h, tid, ROW_REPLAY);
  }
  // Side 1, wave 3 (lane = row of the chunk) takes the local suffix sums of
  // q.dq - k.dk of each chunk during the next chunk's score phase, in which
  // it computes no score block.  It loads q.dq one chunk ahead and keeps it
  // in LDS (rqb, buffered as the chunk metadata): a loaded value carried in
  // registers from one chunk to the next would make every wave wait, at the
  // loop's back edge, for the tile loads issued after it.
  const bool sw = side == 1 && w == 3;
  const float* rq_h = rq + (static_cast<int64_t>(sq.chunk_off) * CB + lane) * H + h;
  if (sw) sm.rqb[0][lane] = rq_h[static_cast<int64_t>(c_last) * CB * H];
  int rowk_prev = 0;    // row table entry of chunk cp, the one after the current chunk
  float carry = 0.f;    // sum of (q.dq - k.dk) over the later chunks of the block
  const auto suffix = [&](int cp, int buf) {
    const int kind = rowk_prev & 3;
    float x = 0.f;
    if (kind != ROW_PAD) {
      float rks = 0.f;
#pragma unroll
      for (int i = 0; i < C::NW; ++i) rks += sm.rk[i][lane];
      x = sm.rqb[buf][lane] - rks;
    }
    x = wave_suffix_sum(x, lane);
    const float val = x + carry;
    if (kind == ROW_OWN) dg[static_cast<int64_t>(rowk_prev >> 2) * H + h] = val;
    else if (kind == ROW_REPLAY)
      rep_grad[((static_cast<int64_t>(sq.replay_off) + cp * CB + lane) * H + h) * RG + 2 * D] = val;
    carry += lane_value(x, 0);
  };
  __syncthreads();
  for (int c = c_last; c >= c0; --c) {
    const int bf = (c_last - c) & 1, nb = bf ^ 1;
    const bool more = c > c0;
    const ChunkRows cur = cur_next;
    const float GL = sm.meta[bf].G[CB - 1];
    // side 0: A = (Q K^T) * M ; side 1: dA = scale (dO V^T) * M,
    // M = exp(G_i - G_j) [j <= i], in three 32 x 32 blocks per half
    if constexpr (SH) {
      // side 1: the adjoint's operands as side 0 left them after the chunk before
      if (side && c < c_last) {
        if constexpr (sizeof(T) == 2) adj_load<D, C::NT, C::CPW>(ps, sm.tl.dt, w, lane);
      }
      if (w < 3) {
        if (side) score_block<T, D, true, LQ, LK, typename BrSmem<T, D>::TP>(sm.P[1], sm.tl.at(bf, TDO), sm.tl.at(bf, TV), sm.meta[bf].G, scale, w, lane);
        else score_block<T, D, true, LQ, LK, typename BrSmem<T, D>::TP>(sm.P[0], sm.tl.at(bf, TQ), sm.tl.at(bf, TK), sm.meta[bf].G, 1.f, w, lane);
      } else if (sw) {
        // the suffix of the chunk after, then the chunk before's q.dq into
        // the buffer it has read (loaded here, so that no other path of the
        // loop sees the load outstanding)
        const float rq_ld = more ? rq_h[static_cast<int64_t>(c - 1) * CB * H] : 0.f;
        if (c < c_last) suffix(c + 1, nb);
        if (more) sm.rqb[nb][lane] = rq_ld;
      } else if (pw && more) {
        publish(cs, nb);
      }
    } else {
      if (pw && more) publish(cs, nb);
      if (!side && w < 3) score_block<T, D, true, LQ, LK, typename BrSmem<T, D>::TP>(sm.P[0], sm.tl.at(bf, TQ), sm.tl.at(bf, TK), sm.meta[bf].G, 1.f, w, lane);
    }
    // next chunk: Q, K into the other buffer; V, dO requested
    if (more) {
      put<T, D, NTH, LQ>(sm.tl.at(nb, TQ), pa, nullptr, tid);
      put<T, D, NTH, LK>(sm.tl.at(nb, TK), pb, nullptr, tid);
      fetch<T, D, NTH>(pa, v, cs, H, h, tid, ROW_REPLAY);
      fetch<T, D, NTH>(pb, dO, cs, H, h, tid, ROW_OWN);
    }
    __syncthreads();
    if constexpr (SH) {
      if (side) bwd_revorder_rows<T, D, 1>(sm, bf, dS, ps, cur, sq, c, more, H, h, scale, GL, w, lane, dk, dv, rep_grad);
      else bwd_revorder_rows<T, D, 0>(sm, bf, dS, ps, cur, sq, c, more, H, h, scale, GL, w, lane, dk, dv, rep_grad);
      // every wave is done with this chunk's V and dO before the next ones
      // replace them
      if (more) __syncthreads();
    } else {
      if (!side) bwd_revorder_rows<T, D, 0>(sm, bf, dS, ps, cur, sq, c, more, H, h, scale, GL, w, lane, dk, dv, rep_grad);
      __syncthreads();
      if (side && w < 3) score_block<T, D, true, LQ, LK, typename BrSmem<T, D>::TP>(sm.P[0], sm.tl.at(bf, TDO), sm.tl.at(bf, TV), sm.meta[bf].G, scale, w, lane);
      else if (sw) {
        const float rq_ld = more ? rq_h[static_cast<int64_t>(c - 1) * CB * H] : 0.f;
        if (c < c_last) suffix(c + 1, nb);
        if (more) sm.rqb[nb][lane] = rq_ld;
      }
      __syncthreads();
      if (side) bwd_revorder_rows<T, D, 1>(sm, bf, dS, ps, cur, sq, c, more, H, h, scale, GL, w, lane, dk, dv, rep_grad);
    }
    // next chunk: V, dO into their buffer; the chunk after it resolved and
    // its Q, K requested
    if (more) {
      put<T, D, NTH, LK>(sm.tl.at(nb, TV), pa, nullptr, tid);
      put<T, D, NTH, LQ>(sm.tl.at(nb, TDO), pb, nullptr, tid);
      cur_next = cs.cr;
      if (c - 1 > c0)
        resolve_fetch2<T, D, NTH>(cs, sq, c - 2, replay_row, g, H, h, tid, mrow, pa, q, ROW_OWN, pb, k,
                                  ROW_REPLAY);
    }
    if (sw) rowk_prev = sm.meta[bf].rowk[lane];
    __syncthreads();
  }
  if (sw) {
    suffix(c0, (c_last - c0) & 1);
    if (lane == 0) Rb[static_cast<int64_t>(b) * H + h] = carry;
  }
  // side 0 holds dS at the start of the block: the first block's is dS0
  if (bl.idx == 0 && side == 0) state_store<D, C::CPW>(dS0 + (static_cast<int64_t>(li) * H + h) * DD, dS, w, lane);
}

// ---------------------------------------------------------------------------
// dg: add the contributions of later blocks and of the boundary terms
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(SCAN_THR) void k_dg_carry(
    const int32_t* __restrict__ seq_tab, const int32_t* __restrict__ blk_tab, int H,
    const float* __restrict__ betap, const float* __restrict__ Rb, float* __restrict__ dg,
    float* __restrict__ rep_grad) {
  // One workgroup per (block, chunk of the block, group of DG_HEADS heads):
  // lane hl = t % DG_HEADS is a head, part = t / DG_HEADS a slice of the
  // terms summed into its carry; the chunk's rows are then updated for all
  // heads of the group at once (dg rows are [rows, H], so a row's heads are
  // contiguous).
  constexpr int NSW = D * D / 4 / SCAN_THR;
  constexpr int RG = 2 * D + 1;
  constexpr int NPART = SCAN_THR / DG_HEADS;
  __shared__ float red[SCAN_THR];
  __shared__ float carry_s[DG_HEADS];
  const int b = blockIdx.x, cc = blockIdx.y, h0 = blockIdx.z * DG_HEADS, t = threadIdx.x;
  const int hl = t % DG_HEADS, part = t / DG_HEADS, h = h0 + hl;
  const int32_t* bk = blk_tab + b * BLK_WORDS;
  if (cc >= bk[BLK_NC]) return;  // uniform: blocks have up to block_chunks chunks
  const int32_t* seq = seq_tab + bk[BLK_SEQ] * SEQ_WORDS;
  const int b_end = seq[SEQ_BLK_OFF] + seq[SEQ_N_BLK];
  float carry = 0.f;
  if (h < H) {
    for (int bb = b; bb < b_end; ++bb) {
      const int64_t bi = static_cast<int64_t>(bb) * H + h;
      for (int p = part; p < NSW; p += NPART) carry += betap[bi * NSW + p];
      if (bb > b && part == 0) carry += Rb[bi];
    }
  }
  red[t] = carry;
  __syncthreads();
  if (t < DG_HEADS) {
    float c = 0.f;
#pragma unroll
    for (int k = 0; k < NPART; ++k) c += red[t + DG_HEADS * k];
    carry_s[t] = c;
  }
  __syncthreads();
  const float ch = carry_s[hl];
  const int c = bk[BLK_C0] + cc;
  const int n_rep = seq[SEQ_N_REPLAY], n_tok = seq[SEQ_N_TOK];
  if (h >= H) return;
#pragma unroll
  for (int idx = t; idx < CB * DG_HEADS; idx += SCAN_THR) {
    const int p = c * CB + idx / DG_HEADS;  // idx % DG_HEADS == hl
    if (p < n_rep) {
      const int j = seq[SEQ_REPLAY_OFF] + p;
      rep_grad[(static_cast<int64_t>(j) * H + h) * RG + 2 * D] += ch;
    } else if (p < n_tok) {
      dg[(static_cast<int64_t>(seq[SEQ_OWN_ROW]) + (p - n_rep)) * H + h] += ch;
    }
  }
}

// state handoff and replay reduction
// ---------------------------------------------------------------------------
__global__ void k_gather(const float4* __restrict__ src, const int32_t* __restrict__ idx,
                         int64_t e4, float4* __restrict__ dst) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int i = blockIdx.y;
  if (e >= e4) return;
  const int s = idx[i];
  dst[static_cast<int64_t>(i) * e4 + e] =
      s < 0 ? make_float4(0.f, 0.f, 0.f, 0.f) : src[static_cast<int64_t>(s) * e4 + e];
}

__global__ void k_scatter_add(const float4* __restrict__ src, const int32_t* __restrict__ idx,
                              int n, int64_t e4, float4* __restrict__ dst) {
  const int64_t e = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  if (e >= e4) return;
  for (int i = 0; i < n; ++i) {  // one thread per element: sources in order
    const int s = idx[i];
    if (s < 0) continue;
    float4 a = dst[static_cast<int64_t>(s) * e4 + e];
    const float4 b = src[static_cast<int64_t>(i) * e4 + e];
    a.x += b.x;
    a.y += b.y;
    a.z += b.z;
    a.w += b.w;
    dst[static_cast<int64_t>(s) * e4 + e] = a;
  }
}

// One wave per (compact row, head): lane l owns elements 4l .. 4l + 3 of the
// row's 2D gradient values (dk then dv), lane 0 also its dg; each sums the
// row's replay instances in order and adds the sum to the own-row gradient.
constexpr int RED_WAVES = 4;
template <typename T, int D>
__global__ __launch_bounds__(64 * RED_WAVES) void k_replay_reduce(
    const int32_t* __restrict__ red_rows, const int32_t* __restrict__ red_off,
    const int32_t* __restrict__ red_idx, int H, const float* __restrict__ rep_grad,
    T* __restrict__ dk, T* __restrict__ dv, float* __restrict__ dg) {
  constexpr int RG = 2 * D + 1;
  static_assert(2 * D / 4 <= 64, "a wave covers the row");
  const int u = blockIdx.x, lane = threadIdx.x & 63;
  const int h = blockIdx.y * RED_WAVES + wave_id(threadIdx.x);
  if (h >= H) return;
  const int64_t row = red_rows[u];
  const int b = red_off[u], e = red_off[u + 1];
  if (lane < 2 * D / 4) {
    f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int j = b; j < e; ++j) {
      const float* r = rep_grad + (static_cast<int64_t>(red_idx[j]) * H + h) * RG + 4 * lane;
#pragma unroll
      for (int i = 0; i < 4; ++i) s[i] += r[i];
    }
    const int x = 4 * lane;
    T* p = x < D ? dk + (row * H + h) * D + x : dv + (row * H + h) * D + (x - D);
    Vec4<T>::store(p, Vec4<T>::load(p) + s);
  }
  if (lane == 0) {
    float s = 0.f;
    for (int j = b; j < e; ++j) s += rep_grad[(static_cast<int64_t>(red_idx[j]) * H + h) * RG + 2 * D];
    dg[row * H + h] += s;
  }
}

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------
namespace {

// Optional per-launch timing: a pair of events recorded on the launch stream
// around every kernel while profiling is on (harts_profile_begin/end).
struct ProfRecord {
  const char* name;
  hipEvent_t start, stop;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<ProfRecord> g_prof;
std::vector<hipEvent_t> g_event_pool;

hipEvent_t pooled_event() {
  if (!g_event_pool.empty()) {
    hipEvent_t e = g_event_pool.back();
    g_event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

struct ProfScope {
  ProfRecord rec{nullptr, nullptr, nullptr};
  hipStream_t stream;
  ProfScope(const char* name, hipStream_t s) : stream(s) {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (!g_prof_on) return;
    rec.name = name;
    rec.start = pooled_event();
    rec.stop = pooled_event();
    if (rec.start) (void)hipEventRecord(rec.start, stream);
  }
  ~ProfScope() {
    if (!rec.name) return;
    std::lock_guard<std::mutex> lk(g_prof_mu);
    if (rec.stop) (void)hipEventRecord(rec.stop, stream);
    if (rec.start && rec.stop) g_prof.push_back(rec);
  }
};

int hip_check(const char* where) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error(std::string(where) + ": " + hipGetErrorString(e));
    return HARTS_EHIP;
  }
  return HARTS_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_shape(const harts_plan_t* p, int32_t round, int32_t dtype, int32_t H, int32_t dk,
                int32_t dv, const char* where) {
  const std::string w(where);
  if (!p) { set_error(w + ": plan is NULL"); return HARTS_EINVAL; }
  if (round < 0 || round >= p->K) { set_error(w + ": round out of range"); return HARTS_EINVAL; }
  if (H < 1 || H > 65535) { set_error(w + ": H must be in [1, 65535]"); return HARTS_EINVAL; }
  if (p->chunk != CB) { set_error(w + ": device calls need chunk size 64"); return HARTS_EUNSUPPORTED; }
  if (dtype != HARTS_F32 && dtype != HARTS_BF16) { set_error(w + ": unknown dtype"); return HARTS_EUNSUPPORTED; }
  if (dk != dv || (dk != 64 && dk != 128)) { set_error(w + ": need dk == dv in {64, 128}"); return HARTS_EUNSUPPORTED; }
  if (dtype == HARTS_F32 && dk != 64) { set_error(w + ": float32 path supports d = 64"); return HARTS_EUNSUPPORTED; }
  // the kernels' row tables pack (physical row, kind) as row * 4 + kind in
  // an int32, so packed rows must stay below 2^29
  if (p->C + p->R >= (int64_t{1} << 29)) {
    set_error(w + ": more than 2^29 packed rows (C + R) per plan");
    return HARTS_EUNSUPPORTED;
  }
  return HARTS_OK;
}

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Buffer sizes of one round.
struct Sizes {
  size_t blk_state;  // [n_blk, H, D, D] float32
  size_t gam;        // [n_blk, H] float32
  size_t rq;         // [n_chunks * 64, H] float32
  size_t rb;         // [n_blk, H] float32
  size_t betap;      // [n_blk, H, NSW] float32
  size_t saved;      // S_end + Gamma
  size_t ws_fwd;     // block summaries
  size_t ws_bwd;     // U + dS_end + rq + Rb + betap
  size_t ws_rec;     // extra for the recompute path: summaries + saved
};

Sizes sizes(const harts_plan_t* p, int32_t round, int32_t H, int32_t D) {
  const RoundLayout& L = p->rounds[round];
  Sizes s{};
  const size_t nsw = static_cast<size_t>(D) * D / 4 / SCAN_THR;
  s.blk_state = align256(static_cast<size_t>(L.n_blk) * H * D * D * sizeof(float));
  s.gam = align256(static_cast<size_t>(L.n_blk) * H * sizeof(float));
  s.rq = align256(static_cast<size_t>(L.n_chunks) * CB * H * sizeof(float));
  s.rb = align256(static_cast<size_t>(L.n_blk) * H * sizeof(float));
  s.betap = align256(static_cast<size_t>(L.n_blk) * H * nsw * sizeof(float));
  s.saved = s.blk_state + s.gam;
  s.ws_fwd = s.blk_state;
  s.ws_bwd = 2 * s.blk_state + s.rq + s.rb + s.betap;
  s.ws_rec = s.blk_state + s.saved;
  return s;
}

struct Blob {
  const int32_t* seq_tab;
  const int32_t* blk_tab;
  const int32_t* blk_launch;
  const int32_t* replay_row;
  const int32_t* init_idx;
};

Blob blob_ptrs(const harts_plan_t* p, int32_t round, const void* d_blob) {
  const int32_t* b = static_cast<const int32_t*>(d_blob);
  const RoundLayout& L = p->rounds[round];
  return Blob{b + L.seq_tab, b + L.blk_tab, b + L.blk_launch, b + p->off_replay_row, b + L.init_idx};
}

// Forward block summaries dS_b and Gamma_b; skip1: none for sequences of one
// block.
template <typename T, int D>
int launch_blocksum(const harts_plan_t* p, int32_t round, const Blob& B, int H, const void* k,
                    const void* v, const float* g, float* dSb, float* gam, int skip1, hipStream_t s) {
  const RoundLayout& L = p->rounds[round];
  ProfScope ps("k_blocksum", s);
  hipLaunchKernelGGL((k_blocksum<T, D>), dim3(L.n_blk * H), dim3(Cfg<T, D>::NTHR), 0, s, B.seq_tab,
                     B.blk_tab, B.blk_launch, B.replay_row, H, static_cast<const T*>(k),
                     static_cast<const T*>(v), g, dSb, gam, skip1);
  return hip_check("k_blocksum");
}

// Chain of block summaries: S_end per block, requested boundary states, final
// states; skip1: not for sequences of one block.
template <int D>
int launch_fwd_scan(const harts_plan_t* p, int32_t round, const Blob& B, int H, const InitSrc& is,
                    const float* dSb, const float* gam, float* S_end, float* bank, float* S_final,
                    int skip1, hipStream_t s) {
  const RoundLayout& L = p->rounds[round];
  constexpr int NSW = D * D / 4 / SCAN_THR;
  ProfScope ps("k_fwd_blockscan", s);
  hipLaunchKernelGGL((k_fwd_blockscan<D>), dim3(L.n_seq * NSW, H), dim3(SCAN_THR), 0, s,
                     B.seq_tab, B.blk_tab, H, is, dSb, gam, S_end, bank, S_final, skip1);
  return hip_check("k_fwd_blockscan");
}

template <typename T, int D>
int run_fwd(const harts_plan_t* p, int32_t round, const void* d_blob, int H, float scale,
            const void* q, const void* k, const void* v, const float* g, const float* S0, void* o,
            float* S_final, float* bank, char* saved, char* ws, hipStream_t s) {
  const RoundLayout& L = p->rounds[round];
  const Sizes z = sizes(p, round, H, D);
  const Blob B = blob_ptrs(p, round, d_blob);
  float* dSb = reinterpret_cast<float*>(ws);
  float* S_end = reinterpret_cast<float*>(saved);
  float* gam = reinterpret_cast<float*>(saved + z.blk_state);
  const InitSrc is{S0, bank, B.init_idx};
  // Sequences of one block need no summary or chain: the block kernel starts
  // from the initial state and writes the final state itself (with outputs),
  // and the backward kernels start and end such sequences themselves.
  const int skip1 = o || !S_final;
  if (int rc = launch_blocksum<T, D>(p, round, B, H, k, v, g, dSb, gam, skip1, s))
    return rc;
  if (int rc = launch_fwd_scan<D>(p, round, B, H, is, dSb, gam, S_end, bank, S_final, skip1, s))
    return rc;
  if (!o) return HARTS_OK;  // state pass only (recompute-forward)
  {
    ProfScope ps("k_fwd_block", s);
    hipLaunchKernelGGL((k_fwd_block<T, D>), dim3(L.n_blk * H), dim3(Cfg<T, D>::NTHR), 0, s, B.seq_tab,
                       B.blk_tab, B.blk_launch, B.replay_row, H, scale, static_cast<const T*>(q),
                       static_cast<const T*>(k), static_cast<const T*>(v), g, is, S_end,
                       static_cast<T*>(o), S_final);
  }
  return hip_check("k_fwd_block");
}

template <typename T, int D>
int run_bwd(const harts_plan_t* p, int32_t round, const void* d_blob, int H, float scale,
            const void* q, const void* k, const void* v, const float* g, const float* S0,
            const float* bank, const void* dO, const float* dS_final, const float* dbank, const char* saved,
            char* ws, void* dq, void* dk, void* dv, float* dg, float* rep_grad, float* dS0,
            hipStream_t s) {
  const RoundLayout& L = p->rounds[round];
  const Sizes z = sizes(p, round, H, D);
  const Blob B = blob_ptrs(p, round, d_blob);
  const InitSrc is{S0, bank, B.init_idx};
  char* w = ws;
  float* U = reinterpret_cast<float*>(w);
  w += z.blk_state;
  float* dS_end = reinterpret_cast<float*>(w);
  w += z.blk_state;
  float* rq = reinterpret_cast<float*>(w);
  w += z.rq;
  float* Rb = reinterpret_cast<float*>(w);
  w += z.rb;
  float* betap = reinterpret_cast<float*>(w);
  w += z.betap;
  if (!saved) {
    // recompute-forward: forward summaries, chained from S0 below
    float* dSb = reinterpret_cast<float*>(w);
    char* sv = w + z.blk_state;
    float* S_end_w = reinterpret_cast<float*>(sv);
    float* gam_w = reinterpret_cast<float*>(sv + z.blk_state);
    if (int rc = launch_blocksum<T, D>(p, round, B, H, k, v, g, dSb, gam_w, 1, s))
      return rc;
    if (int rc = launch_fwd_scan<D>(p, round, B, H, is, dSb, gam_w, S_end_w, nullptr, nullptr, 1, s))
      return rc;
    saved = sv;
  }
  const float* S_end = reinterpret_cast<const float*>(saved);
  const float* gam = reinterpret_cast<const float*>(saved + z.blk_state);
  {
    ProfScope ps("k_bwd_fwdorder", s);
    hipLaunchKernelGGL((k_bwd_fwdorder<T, D>), dim3(L.n_blk * H), dim3(2 * Cfg<T, D>::NTHR), 0, s,
                       B.seq_tab, B.blk_tab, B.blk_launch, B.replay_row, H, scale,
                       static_cast<const T*>(q), static_cast<const T*>(k),
                       static_cast<const T*>(v), g, static_cast<const T*>(dO), is, S_end,
                       static_cast<T*>(dq), rq, dS_final, betap, U);
  }
  if (int rc = hip_check("k_bwd_fwdorder")) return rc;
  {
    constexpr int NSW = D * D / 4 / SCAN_THR;
    ProfScope ps("k_bwd_blockscan", s);
    hipLaunchKernelGGL((k_bwd_blockscan<D>), dim3(L.n_seq * NSW, H), dim3(SCAN_THR), 0, s,
                       B.seq_tab, B.blk_tab, H, dS_final, dbank, S_end, U, gam, dS_end, betap);
  }
  if (int rc = hip_check("k_bwd_blockscan")) return rc;
  {
    ProfScope ps("k_bwd_revorder", s);
    hipLaunchKernelGGL((k_bwd_revorder<T, D>), dim3(L.n_blk * H), dim3(2 * Cfg<T, D>::NTHR), 0, s,
                       B.seq_tab, B.blk_tab, B.blk_launch, B.replay_row, H, scale,
                       static_cast<const T*>(q), static_cast<const T*>(k),
                       static_cast<const T*>(v), g, static_cast<const T*>(dO), dS_end, rq,
                       static_cast<T*>(dk), static_cast<T*>(dv), dg, rep_grad, Rb, dS_final, dS0);
  }
  if (int rc = hip_check("k_bwd_revorder")) return rc;
  {
    ProfScope ps("k_dg_carry", s);
    hipLaunchKernelGGL((k_dg_carry<D>), dim3(L.n_blk, L.block_chunks, (H + DG_HEADS - 1) / DG_HEADS),
                       dim3(SCAN_THR), 0, s, B.seq_tab, B.blk_tab, H, betap, Rb, dg, rep_grad);
  }
  return hip_check("k_dg_carry");
}

}  // namespace
}  // namespace harts

using namespace harts;

extern "C" int harts_la_saved_size(const harts_plan_t* p, int32_t round, int32_t dtype, int32_t H,
                                   int32_t dk, int32_t dv, size_t* bytes) {
  if (int rc = check_shape(p, round, dtype, H, dk, dv, "harts_la_saved_size")) return rc;
  if (!bytes) { set_error("harts_la_saved_size: bytes is NULL"); return HARTS_EINVAL; }
  *bytes = sizes(p, round, H, dk).saved;
  return HARTS_OK;
}

extern "C" int harts_la_workspace_size(const harts_plan_t* p, int32_t round, int32_t pass,
                                       int32_t dtype, int32_t H, int32_t dk, int32_t dv,
                                       int32_t has_saved, size_t* bytes) {
  if (int rc = check_shape(p, round, dtype, H, dk, dv, "harts_la_workspace_size")) return rc;
  if (!bytes || (pass != 0 && pass != 1)) {
    set_error("harts_la_workspace_size: bad pass or NULL bytes");
    return HARTS_EINVAL;
  }
  const Sizes z = sizes(p, round, H, dk);
  if (pass == 0) *bytes = z.ws_fwd + (has_saved ? 0 : z.saved);
  else *bytes = z.ws_bwd + (has_saved ? 0 : z.ws_rec);
  return HARTS_OK;
}

namespace harts {
namespace {

int la_fwd_impl(const harts_plan_t* p, int32_t round, const void* d_blob, int32_t dtype, int32_t H,
                int32_t dk, int32_t dv, float scale, const void* q, const void* k, const void* v,
                const float* g, const float* S0, void* o, float* S_final, float* bank, void* saved,
                void* ws, size_t ws_bytes, void* stream, const char* where) {
  const std::string w0(where);
  if (int rc = check_shape(p, round, dtype, H, dk, dv, where)) return rc;
  if (!d_blob || !q || !k || !v || !g || !ws || (!bank && (p->n_slots > 0 || !S0))) {
    set_error(w0 + ": NULL required pointer");
    return HARTS_EINVAL;
  }
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(S0) || !aligned16(o) ||
      !aligned16(S_final) || !aligned16(bank) || !aligned16(saved) || !aligned16(ws)) {
    set_error(w0 + ": pointers must be 16-byte aligned");
    return HARTS_EINVAL;
  }
  const Sizes z = sizes(p, round, H, dk);
  if (ws_bytes < z.ws_fwd + (saved ? 0 : z.saved)) {
    set_error(w0 + ": workspace too small (see harts_la_workspace_size)");
    return HARTS_EINVAL;
  }
  char* w = static_cast<char*>(ws);
  char* sv = saved ? static_cast<char*>(saved) : w + z.ws_fwd;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == HARTS_BF16) {
    if (dk == 128)
      return run_fwd<bf16, 128>(p, round, d_blob, H, scale, q, k, v, g, S0, o, S_final, bank, sv, w, s);
    return run_fwd<bf16, 64>(p, round, d_blob, H, scale, q, k, v, g, S0, o, S_final, bank, sv, w, s);
  }
  return run_fwd<float, 64>(p, round, d_blob, H, scale, q, k, v, g, S0, o, S_final, bank, sv, w, s);
}

// Scratch of harts_la_fwd_noalloc: the round's block summaries, block-end
// states and block log-decays, in a file-scope device array that each GPU
// holds from the library's load until the process ends.  Host code never
// passes the array's name to a kernel (on the host it is only a stand-in
// for the symbol): the device address comes from hipGetSymbolAddress, taken
// once per device with that device current.
constexpr size_t kScratchBytes = size_t{64} << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) char scratch[kScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_ptr(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    set_error("harts_la_fwd_noalloc: no current HIP device (or device id >= 64)");
    return HARTS_EHIP;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      set_error(std::string("harts_la_fwd_noalloc: hipGetSymbolAddress: ") + hipGetErrorString(e));
      return HARTS_EHIP;
    }
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return HARTS_OK;
}

}  // namespace
}  // namespace harts

extern "C" int harts_la_fwd(const harts_plan_t* p, int32_t round, const void* d_blob,
                            int32_t dtype, int32_t H, int32_t dk, int32_t dv, float scale,
                            const void* q, const void* k, const void* v, const float* g,
                            const float* S0, void* o, float* S_final, float* bank, void* saved,
                            void* ws, size_t ws_bytes, void* stream) {
  return la_fwd_impl(p, round, d_blob, dtype, H, dk, dv, scale, q, k, v, g, S0, o, S_final, bank,
                     saved, ws, ws_bytes, stream, "harts_la_fwd");
}

extern "C" int harts_la_fwd_noalloc(const harts_plan_t* p, int32_t round, const void* d_blob,
                                    int32_t dtype, int32_t H, int32_t dk, int32_t dv, float scale,
                                    const void* q, const void* k, const void* v, const float* g,
                                    const float* S0, void* o, float* S_final, float* bank,
                                    void* stream) {
  if (int rc = check_shape(p, round, dtype, H, dk, dv, "harts_la_fwd_noalloc")) return rc;
  const Sizes z = sizes(p, round, H, dk);
  const size_t need = z.ws_fwd + z.saved;
  if (need > kScratchBytes) {
    set_error("harts_la_fwd_noalloc: the round needs " + std::to_string(need) +
              " bytes of scratch, above the library's fixed " + std::to_string(kScratchBytes) +
              " (use harts_la_fwd with a workspace)");
    return HARTS_ENOMEM;
  }
  void* ws = nullptr;
  if (int rc = scratch_ptr(&ws)) return rc;
  return la_fwd_impl(p, round, d_blob, dtype, H, dk, dv, scale, q, k, v, g, S0, o, S_final, bank,
                     nullptr, ws, kScratchBytes, stream, "harts_la_fwd_noalloc");
}

extern "C" int harts_la_bwd(const harts_plan_t* p, int32_t round, const void* d_blob,
                            int32_t dtype, int32_t H, int32_t dk, int32_t dv, float scale,
                            const void* q, const void* k, const void* v, const float* g,
                            const float* S0, const float* bank, const void* dO,
                            const float* dS_final, const float* dbank, const void* saved, void* dq,
                            void* dk_, void* dv_, float* dg, float* replay_grad, float* dS0,
                            void* ws, size_t ws_bytes, void* stream) {
  if (int rc = check_shape(p, round, dtype, H, dk, dv, "harts_la_bwd")) return rc;
  if (!d_blob || !q || !k || !v || !g || (!S0 && !bank) || !dO || !dS_final || !dq || !dk_ || !dv_ || !dg ||
      !dS0 || (!dbank && p->n_slots > 0) || (!replay_grad && p->R > 0) || !ws) {
    set_error("harts_la_bwd: NULL required pointer");
    return HARTS_EINVAL;
  }
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dO) || !aligned16(dq) ||
      !aligned16(dk_) || !aligned16(dv_) || !aligned16(saved) || !aligned16(ws) ||
      !aligned16(dS0) || !aligned16(dS_final) || !aligned16(S0) || !aligned16(bank) ||
      !aligned16(dbank)) {
    set_error("harts_la_bwd: pointers must be 16-byte aligned");
    return HARTS_EINVAL;
  }
  const Sizes z = sizes(p, round, H, dk);
  if (ws_bytes < z.ws_bwd + (saved ? 0 : z.ws_rec)) {
    set_error("harts_la_bwd: workspace too small (see harts_la_workspace_size)");
    return HARTS_EINVAL;
  }
  const char* sv = static_cast<const char*>(saved);
  char* w = static_cast<char*>(ws);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dtype == HARTS_BF16) {
    if (dk == 128)
      return run_bwd<bf16, 128>(p, round, d_blob, H, scale, q, k, v, g, S0, bank, dO, dS_final, dbank,
                                sv, w, dq, dk_, dv_, dg, replay_grad, dS0, s);
    return run_bwd<bf16, 64>(p, round, d_blob, H, scale, q, k, v, g, S0, bank, dO, dS_final, dbank, sv,
                             w, dq, dk_, dv_, dg, replay_grad, dS0, s);
  }
  return run_bwd<float, 64>(p, round, d_blob, H, scale, q, k, v, g, S0, bank, dO, dS_final, dbank, sv,
                            w, dq, dk_, dv_, dg, replay_grad, dS0, s);
}
extern "C" int harts_state_gather(const float* src, const int32_t* idx, int32_t n,
                                  int64_t elems_per_state, float* dst, int32_t mode,
                                  void* stream) {
  if (n < 0 || elems_per_state <= 0 || elems_per_state % 4 != 0 || (mode != 0 && mode != 1)) {
    set_error("harts_state_gather: bad n, elems_per_state or mode");
    return HARTS_EINVAL;
  }
  if (n == 0) return HARTS_OK;
  if (!src || !idx || !dst || !aligned16(src) || !aligned16(dst)) {
    set_error("harts_state_gather: NULL or misaligned pointer");
    return HARTS_EINVAL;
  }
  if (mode == 0 && n > 65535) {
    set_error("harts_state_gather: at most 65535 states per gather");
    return HARTS_EINVAL;
  }
  const int64_t e4 = elems_per_state / 4;
  const unsigned blocks = static_cast<unsigned>((e4 + 255) / 256);
  hipStream_t s = static_cast<hipStream_t>(stream);
  ProfScope ps(mode == 0 ? "k_gather" : "k_scatter_add", s);
  if (mode == 0)
    hipLaunchKernelGGL(k_gather, dim3(blocks, n), dim3(256), 0, s,
                       reinterpret_cast<const float4*>(src), idx, e4,
                       reinterpret_cast<float4*>(dst));
  else
    hipLaunchKernelGGL(k_scatter_add, dim3(blocks), dim3(256), 0, s,
                       reinterpret_cast<const float4*>(src), idx, n, e4,
                       reinterpret_cast<float4*>(dst));
  return hip_check("harts_state_gather");
}

extern "C" int harts_replay_reduce(const harts_plan_t* p, const void* d_blob, int32_t dtype,
                                   int32_t H, int32_t dk, int32_t dv, const float* replay_grad,
                                   void* dk_, void* dv_, float* dg, void* stream) {
  if (int rc = check_shape(p, 0, dtype, H, dk, dv, "harts_replay_reduce")) return rc;
  if (p->n_red == 0) return HARTS_OK;
  if (!d_blob || !replay_grad || !dk_ || !dv_ || !dg) {
    set_error("harts_replay_reduce: NULL required pointer");
    return HARTS_EINVAL;
  }
  const int32_t* b = static_cast<const int32_t*>(d_blob);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid(static_cast<unsigned>(p->n_red), (H + RED_WAVES - 1) / RED_WAVES);
  ProfScope ps("k_replay_reduce", s);
  if (dtype == HARTS_BF16) {
    if (dk == 128)
      hipLaunchKernelGGL((k_replay_reduce<bf16, 128>), grid, dim3(64 * RED_WAVES), 0, s, b + p->off_red_rows,
                         b + p->off_red_off, b + p->off_red_idx, H, replay_grad,
                         static_cast<bf16*>(dk_), static_cast<bf16*>(dv_), dg);
    else
      hipLaunchKernelGGL((k_replay_reduce<bf16, 64>), grid, dim3(64 * RED_WAVES), 0, s, b + p->off_red_rows,
                         b + p->off_red_off, b + p->off_red_idx, H, replay_grad,
                         static_cast<bf16*>(dk_), static_cast<bf16*>(dv_), dg);
  } else {
    hipLaunchKernelGGL((k_replay_reduce<float, 64>), grid, dim3(64 * RED_WAVES), 0, s, b + p->off_red_rows,
                       b + p->off_red_off, b + p->off_red_idx, H, replay_grad,
                       static_cast<float*>(dk_), static_cast<float*>(dv_), dg);
  }
  return hip_check("harts_replay_reduce");
}

extern "C" int harts_profile_begin(void) {
  std::lock_guard<std::mutex> lk(g_prof_mu);
  g_prof_on = true;
  return HARTS_OK;
}

extern "C" int harts_profile_end(harts_kernel_time* out, int32_t cap, int32_t* n_out) {
  std::vector<ProfRecord> recs;
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    g_prof_on = false;
    recs.swap(g_prof);
  }
  std::vector<harts_kernel_time> agg;
  int rc = HARTS_OK;
  for (const ProfRecord& r : recs) {
    float ms = 0.f;
    if (hipEventSynchronize(r.stop) != hipSuccess || hipEventElapsedTime(&ms, r.start, r.stop) != hipSuccess) {
      set_error("harts_profile_end: event query failed");
      rc = HARTS_EHIP;
    }
    size_t j = 0;
    while (j < agg.size() && std::strcmp(agg[j].name, r.name) != 0) ++j;
    if (j == agg.size()) {
      harts_kernel_time k{};
      std::strncpy(k.name, r.name, sizeof(k.name) - 1);
      agg.push_back(k);
    }
    agg[j].launches += 1;
    agg[j].total_ms += ms;
  }
  {
    std::lock_guard<std::mutex> lk(g_prof_mu);
    for (const ProfRecord& r : recs) {
      g_event_pool.push_back(r.start);
      g_event_pool.push_back(r.stop);
    }
  }
  const int32_t n = static_cast<int32_t>(agg.size());
  if (n_out) *n_out = n;
  if (out)
    for (int32_t i = 0; i < n && i < cap; ++i) out[i] = agg[i];
  return rc;
}
