// Full attention over compact rows through asymmetric packed Q/KV views
// (HARTS, Sec. 4.2, eqs. asymmetric-qkv and bottom-right), bf16 on gfx950.
//
// A view is one input sequence of the plan: its query row holds its l own
// rows (contiguous physical compact rows), its key/value row the h ancestor
// positions of its trajectory followed by the same l rows, gathered into a
// packed KV buffer.  Query i sees keys j <= h + i (bottom-right alignment).
// Outputs go straight back to the queries' compact rows (a row is an own row
// of exactly one view); key/value gradients of the views are summed into
// the compact rows they were gathered from, in a fixed order.
//
// Flash-style kernels: a workgroup of 4 waves owns 128 rows of one view and
// head (queries in the forward and dq, keys in dk/dv), a wave 32 of them as
// two 16-row halves, and steps over the other side 64 rows at a time; bf16
// MFMA 16x16x32 with float32 accumulation.  Each step's tiles are staged in
// LDS and the next step's are loaded into registers meanwhile; every
// fragment read from LDS feeds both halves of the wave.  Every product is
// issued with the operand roles chosen so that the row the wave owns is the
// accumulator column (lane % 16): per-row softmax statistics, rescales and
// outputs then stay in one lane, and a score tile in accumulators is already
// the B operand of the next product (two 16-key tiles form one 32-deep
// operand).  Steps that no row of a wave can see are skipped by that wave;
// masks are evaluated only on steps that cross the causal diagonal.
//   k_attn_fwd   per (query tile, head): S = Q K^T, online softmax, O = P V;
//                writes o and the row log-sum-exp;
//   k_attn_delta per (row, head): delta = dO . O;
//   k_attn_dq    per (query tile, head): P from the stored log-sum-exp,
//                dP = dO V^T, dS = P (dP - delta), dQ = scale dS K;
//   k_attn_dkdv  per (key tile, head): over the query tiles that see it,
//                dV = P^T dO and dK = scale dS^T Q (float32 view rows);
//   k_attn_gather / k_attn_scatter: compact rows to view rows and back.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <new>
#include <string>
#include <vector>

#include "harts.h"
#include "la_common.hpp"
#include "plan.hpp"

namespace harts {
namespace {

constexpr int AT_THR = 256;          // 4 waves
constexpr int AT_T = 64;             // rows of an LDS tile (keys per step, queries per step in dk/dv)
constexpr int AT_WT = 128;           // rows of a table tile (queries in fwd/dq, keys in dk/dv)
// 16-row halves a wave owns, per kernel (measured choices)
constexpr int AT_FWD_NH = 2, AT_DQ_NH = 2, AT_DKDV_NH = 1;
constexpr float AT_LOG2E = 1.4426950408889634f;
constexpr float AT_NEG = -1.0e30f;   // masked score (finite: no inf - inf)
// The forward keeps a row's reference maximum until a score exceeds it by
// more than this (base 2): weights then stay below 2^8, and the rescale of
// the accumulators is skipped on most steps.
constexpr float AT_SLACK = 8.f;

// view table: 4 int32 per view
enum { V_QROW = 0, V_L = 1, V_KVOFF = 2, V_H = 3 };

// LDS tile of 64 rows x D: the swizzled layout at D = 128 (both the
// k-contiguous and the transposed fragment reads conflict-free), else the
// padded one.
template <int D>
using AT_Tile = TileX<bf16, D>;

// One 64-row tile of a [rows, H, D] bf16 tensor (head h) held in registers
// between its global load and its LDS store, so that the next tile's load is
// in flight while the current one is used.  The loads go through a buffer
// resource covering rows row0 .. row0 + n - 1 only: rows at or past n read
// as zero without touching memory.
template <int D>
struct RowsReg {
  static constexpr int VPR = D / 8;                  // 16-byte vectors per row
  static constexpr int NV = AT_T * VPR / AT_THR;     // vectors per thread
  uint4 v[NV];
  __device__ inline void load(const bf16* __restrict__ src, int64_t row0, int n, int H, int h, int t) {
    const int64_t rowel = static_cast<int64_t>(H) * D;
    const uint32_t bytes = n > 0 ? static_cast<uint32_t>(n * rowel * 2) : 0u;   // n <= 64, H <= 65535
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>(src + row0 * rowel + static_cast<int64_t>(h) * D), static_cast<short>(0),
        static_cast<int>(bytes), 0x00020000);
#pragma unroll
    for (int e = 0; e < NV; ++e) {
      const int idx = t + AT_THR * e, r = idx / VPR, c = (idx % VPR) * 8;
      const uint32_t off = static_cast<uint32_t>((r * rowel + c) * 2);
      v[e] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rs, static_cast<int>(off), 0, 0));
    }
  }
  __device__ inline void store(bf16* tile, int t) const {
#pragma unroll
    for (int e = 0; e < NV; ++e) {
      const int idx = t + AT_THR * e, r = idx / VPR, c = (idx % VPR) * 8;
      *reinterpret_cast<uint4*>(tile + AT_Tile<D>::at(r, c)) = v[e];
    }
  }
};

// 2^x with the hardware instruction (results below 2^-126 flush to zero,
// which a softmax weight can afford).
__device__ inline float at_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ inline float row_max4(float x) {  // over the 4 lane groups (same lane % 16)
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}
__device__ inline float row_sum4(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}

// Rows of a workgroup and of a wave: NH halves of 16 rows a wave, 4 waves.
// A table tile (AT_WT rows) is split over AT_WT / (64 NH) workgroups.
template <int NH>
struct AtRows {
  static constexpr int WR = 16 * NH;        // rows a wave owns
  static constexpr int WG = 4 * WR;         // rows a workgroup owns
  static constexpr int SUB = AT_WT / WG;    // workgroups per table tile
  static_assert(NH == 1 || NH == 2, "one or two 16-row halves a wave");
};

// Decode blockIdx.x = (table tile * SUB + sub) * H + h.
template <int NH>
__device__ inline void at_block(int H, int& tile, int& sub, int& h) {
  const int b = blockIdx.x / H;
  h = blockIdx.x % H;
  tile = b / AtRows<NH>::SUB;
  sub = b % AtRows<NH>::SUB;
}

// Stage rows row0 .. row0 + n - 1 (n <= 64 NH) of [rows, H, D] into the
// first NH LDS tiles of {ta, tb} (zero past n).
template <int D, int NH>
__device__ inline void stage_rows(bf16* ta, bf16* tb, const bf16* __restrict__ src, int64_t row0, int n, int H,
                                  int h, int t) {
  RowsReg<D> x;
  x.load(src, row0, min(n, AT_T), H, h, t);
  x.store(ta, t);
  if (NH == 2) {
    x.load(src, row0 + AT_T, n - AT_T, H, h, t);
    x.store(tb, t);
  }
}

// The k-contiguous fragments (32-deep steps s) of the 16 rows 16 a .. of
// wave w, from rows staged by stage_rows.
template <int D, int NH>
__device__ inline void wave_frags(typename Frag<bf16>::V (&f)[NH][D / 32], const bf16* ta, const bf16* tb, int w,
                                  int lane) {
#pragma unroll
  for (int a = 0; a < NH; ++a) {
    const int r = AtRows<NH>::WR * w + 16 * a;
#pragma unroll
    for (int s = 0; s < D / 32; ++s) f[a][s] = Frag<bf16>::kc<AT_Tile<D>>(r < AT_T ? ta : tb, r & (AT_T - 1), 32 * s, lane);
  }
}

// ---------------------------------------------------------------------------
// forward: workgroup = 64 NH queries of one view and head; wave w owns
// 16 NH of them (halves a).  Per 64-key step, every K fragment read from
// LDS feeds all halves, and so does every V fragment.
// ---------------------------------------------------------------------------
template <int D, int NH>
__global__ __launch_bounds__(AT_THR, 2) void k_attn_fwd(const int32_t* __restrict__ views,
                                                        const int32_t* __restrict__ qtiles, int H, float scale,
                                                        const bf16* __restrict__ q, const bf16* __restrict__ kv_k,
                                                        const bf16* __restrict__ kv_v, bf16* __restrict__ o,
                                                        float* __restrict__ lse) {
  using F = Frag<bf16>;
  using L = AT_Tile<D>;
  using R = AtRows<NH>;
  constexpr int NS = D / 32;  // 32-deep steps over d
  constexpr int NJ = D / 16;  // 16-column output tiles
  __shared__ bf16 sK[L::SIZE], sV[L::SIZE];
  int tile, sub, h;
  at_block<NH>(H, tile, sub, h);
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int v = qtiles[2 * tile], t0 = qtiles[2 * tile + 1] + R::WG * sub;
  const int32_t* vw = views + 4 * v;
  const int64_t qrow0 = vw[V_QROW];
  const int l = vw[V_L], hh = vw[V_H];
  const int64_t kvoff = vw[V_KVOFF];
  const int nq = min(R::WG, l - t0);
  if (nq <= 0) return;                      // the view ends in an earlier workgroup of the tile
  const int kv_end = hh + t0 + nq;          // keys the workgroup's last query sees
  stage_rows<D, NH>(sK, sV, q, qrow0 + t0, nq, H, h, t);
  RowsReg<D> pk, pv;                        // first key/value step in flight
  pk.load(kv_k, kvoff, min(AT_T, kv_end), H, h, t);
  pv.load(kv_v, kvoff, min(AT_T, kv_end), H, h, t);
  __syncthreads();
  const int i = lane & 15, g = lane >> 4;
  const int wq0 = t0 + R::WR * w;           // the wave's first query (within the view)
  typename F::V qf[NH][NS];
  wave_frags<D, NH>(qf, sK, sV, w, lane);
  const bool wave_live = R::WR * w < nq;
  const int wave_end = min(kv_end, hh + wq0 + R::WR);   // keys the wave's last query sees
  const float c2 = scale * AT_LOG2E;        // scores in base 2
  float m[NH], lsum[NH];
  f32x4 acc[NH][NJ];
#pragma unroll
  for (int a = 0; a < NH; ++a) {
    m[a] = AT_NEG;
    lsum[a] = 0.f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[a][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int k0 = 0; k0 < kv_end; k0 += AT_T) {
    __syncthreads();                        // readers of the previous step (and of Q) are done
    pk.store(sK, t);
    pv.store(sV, t);
    __syncthreads();
    if (k0 + AT_T < kv_end) {
      pk.load(kv_k, kvoff + k0 + AT_T, min(AT_T, kv_end - k0 - AT_T), H, h, t);
      pv.load(kv_v, kvoff + k0 + AT_T, min(AT_T, kv_end - k0 - AT_T), H, h, t);
    }
    if (!wave_live || k0 >= wave_end) continue;      // wave-uniform
    // S^T tiles: lane (g, i) of half a gets S[q = wq0 + 16 a + i][key = k0 + 16 j + 4 g + r]
    f32x4 sc[NH][4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int a = 0; a < NH; ++a) sc[a][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the product blocks run at raised wave priority, so that the other
    // wave of the SIMD issues its softmax work while this one feeds the
    // matrix core
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const typename F::V kf = F::kc<L>(sK, 16 * j, 32 * s, lane);
#pragma unroll
        for (int a = 0; a < NH; ++a) F::mma(sc[a][j], kf, qf[a][s]);
      }
    __builtin_amdgcn_s_setprio(0);
    // steps that cross the diagonal: keys past a query's last visible key
    if (k0 + AT_T > hh + wq0 + 1) {
#pragma unroll
      for (int a = 0; a < NH; ++a) {
        const int lim = hh + wq0 + 16 * a + i - k0 - 4 * g;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (16 * j + r > lim) sc[a][j][r] = AT_NEG;
      }
    }
    // online softmax in base 2 against a reference maximum m per row: it is
    // raised (and the accumulators rescaled) only when some score of the
    // wave exceeds its row's m by more than the slack
    float tmx[NH];
    bool raise = false;
#pragma unroll
    for (int a = 0; a < NH; ++a) {
      float x = sc[a][0][0];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) x = fmaxf(x, sc[a][j][r]);
      tmx[a] = x * c2;
      raise |= tmx[a] > m[a] + AT_SLACK;
    }
    if (__ballot(raise) != 0ull) {
#pragma unroll
      for (int a = 0; a < NH; ++a) {
        const float mn = fmaxf(m[a], row_max4(tmx[a]));
        const float corr = at_exp2(m[a] - mn);
        m[a] = mn;
        lsum[a] *= corr;
#pragma unroll
        for (int j = 0; j < NJ; ++j) acc[a][j] *= corr;
      }
    }
#pragma unroll
    for (int a = 0; a < NH; ++a) {
      const float nm = -m[a];
#pragma unroll
      for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = at_exp2(fmaf(sc[a][j][r], c2, nm));
          sc[a][j][r] = p;
          lsum[a] += p;          // this lane's share of the row sum
        }
    }
    // O^T += V^T P^T: lane (g, i) of half a gets O[q = wq0 + 16 a + i][d = 16 jn + 4 g + r]
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      bf16x8 pf[NH];
#pragma unroll
      for (int a = 0; a < NH; ++a) pf[a] = RegB<bf16>::pack(sc[a] + 2 * s2);
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int jn = 0; jn < NJ; ++jn) {
        const typename F::V vf = F::km<L>(sV, 32 * s2, 16 * jn, lane);
#pragma unroll
        for (int a = 0; a < NH; ++a) F::mma(acc[a][jn], vf, pf[a]);
      }
      __builtin_amdgcn_s_setprio(0);
    }
  }
#pragma unroll
  for (int a = 0; a < NH; ++a) lsum[a] = row_sum4(lsum[a]);
#pragma unroll
  for (int a = 0; a < NH; ++a) {
    if (R::WR * w + 16 * a + i < nq) {
      const float inv = lsum[a] > 0.f ? 1.f / lsum[a] : 0.f;
      const int64_t row = qrow0 + wq0 + 16 * a + i;
#pragma unroll
      for (int jn = 0; jn < NJ; ++jn)
        Vec4<bf16>::store(o + (row * H + h) * D + 16 * jn + 4 * g, acc[a][jn] * inv);
      if (g == 0) lse[row * H + h] = (m[a] + log2f(lsum[a])) / AT_LOG2E;   // natural log of sum exp(scale s)
    }
  }
}

// ---------------------------------------------------------------------------
// backward
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(AT_THR) void k_attn_delta(int64_t n, const bf16* __restrict__ o,
                                                       const bf16* __restrict__ dO, float* __restrict__ delta) {
  const int64_t rh = static_cast<int64_t>(blockIdx.x) * AT_THR + threadIdx.x;  // row * H + h
  if (rh >= n) return;
  float s = 0.f;
  for (int c = 0; c < D; c += 4) {
    const f32x4 a = Vec4<bf16>::load(o + rh * D + c), b = Vec4<bf16>::load(dO + rh * D + c);
    s += a[0] * b[0] + a[1] * b[1] + a[2] * b[2] + a[3] * b[3];
  }
  delta[rh] = s;
}

// dq: workgroup = 64 NH queries of one view and head, wave w owns 16 NH of
// them; per 64-key step S and dP from the K and V tiles (each fragment
// feeding all halves), dS = P (dP - delta), dQ += dS K.
template <int D, int NH>
__global__ __launch_bounds__(AT_THR, 2) void k_attn_dq(
    const int32_t* __restrict__ views, const int32_t* __restrict__ qtiles, int H, float scale,
    const bf16* __restrict__ q, const bf16* __restrict__ kv_k, const bf16* __restrict__ kv_v,
    const bf16* __restrict__ dO, const float* __restrict__ lse, const float* __restrict__ delta,
    bf16* __restrict__ dq) {
  using F = Frag<bf16>;
  using L = AT_Tile<D>;
  using R = AtRows<NH>;
  constexpr int NS = D / 32, NJ = D / 16;
  __shared__ bf16 sK[L::SIZE], sV[L::SIZE];
  int tile, sub, h;
  at_block<NH>(H, tile, sub, h);
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int v = qtiles[2 * tile], t0 = qtiles[2 * tile + 1] + R::WG * sub;
  const int32_t* vw = views + 4 * v;
  const int64_t qrow0 = vw[V_QROW];
  const int l = vw[V_L], hh = vw[V_H];
  const int64_t kvoff = vw[V_KVOFF];
  const int nq = min(R::WG, l - t0);
  if (nq <= 0) return;
  const int kv_end = hh + t0 + nq;
  const int i = lane & 15, g = lane >> 4;
  const int wq0 = t0 + R::WR * w;
  typename F::V qf[NH][NS], df[NH][NS];
  stage_rows<D, NH>(sK, sV, q, qrow0 + t0, nq, H, h, t);
  __syncthreads();
  wave_frags<D, NH>(qf, sK, sV, w, lane);
  __syncthreads();
  stage_rows<D, NH>(sK, sV, dO, qrow0 + t0, nq, H, h, t);
  __syncthreads();
  wave_frags<D, NH>(df, sK, sV, w, lane);
  float l2[NH], dl[NH];
#pragma unroll
  for (int a = 0; a < NH; ++a) {
    const bool live = R::WR * w + 16 * a + i < nq;
    const int64_t row = qrow0 + (live ? wq0 + 16 * a + i : t0);
    l2[a] = live ? lse[row * H + h] * AT_LOG2E : 0.f;
    dl[a] = live ? delta[row * H + h] : 0.f;
  }
  RowsReg<D> pk, pv;
  pk.load(kv_k, kvoff, min(AT_T, kv_end), H, h, t);
  pv.load(kv_v, kvoff, min(AT_T, kv_end), H, h, t);
  const bool wave_live = R::WR * w < nq;
  const int wave_end = min(kv_end, hh + wq0 + R::WR);
  const float c2 = scale * AT_LOG2E;
  f32x4 acc[NH][NJ];
#pragma unroll
  for (int a = 0; a < NH; ++a)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[a][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < kv_end; k0 += AT_T) {
    __syncthreads();
    pk.store(sK, t);
    pv.store(sV, t);
    __syncthreads();
    if (k0 + AT_T < kv_end) {
      pk.load(kv_k, kvoff + k0 + AT_T, min(AT_T, kv_end - k0 - AT_T), H, h, t);
      pv.load(kv_v, kvoff + k0 + AT_T, min(AT_T, kv_end - k0 - AT_T), H, h, t);
    }
    if (!wave_live || k0 >= wave_end) continue;
    // per 16-key group j: S and dP over d, then dS = P (dP - delta) with
    // P = exp(scale s - lse), so that dP lives for one group only
    f32x4 sc[NH][4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f32x4 dp[NH];
#pragma unroll
      for (int a = 0; a < NH; ++a) {
        sc[a][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        dp[a] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const typename F::V kf = F::kc<L>(sK, 16 * j, 32 * s, lane);
#pragma unroll
        for (int a = 0; a < NH; ++a) F::mma(sc[a][j], kf, qf[a][s]);
        const typename F::V vf = F::kc<L>(sV, 16 * j, 32 * s, lane);
#pragma unroll
        for (int a = 0; a < NH; ++a) F::mma(dp[a], vf, df[a][s]);
      }
#pragma unroll
      for (int a = 0; a < NH; ++a)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = at_exp2(fmaf(sc[a][j][r], c2, -l2[a]));
          sc[a][j][r] = p * (dp[a][r] - dl[a]);
        }
    }
    // steps that cross the diagonal, or hold rows past the view: zero what
    // the row cannot see
    if (k0 + AT_T > hh + wq0 + 1 || R::WR * (w + 1) > nq) {
#pragma unroll
      for (int a = 0; a < NH; ++a) {
        const int lim = R::WR * w + 16 * a + i < nq ? hh + wq0 + 16 * a + i - k0 - 4 * g : -AT_T;
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (16 * j + r > lim) sc[a][j][r] = 0.f;
      }
    }
    // dQ^T += K^T dS^T: lane (g, i) of half a gets dQ[q = wq0 + 16 a + i][d = 16 jn + 4 g + r]
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      bf16x8 sf[NH];
#pragma unroll
      for (int a = 0; a < NH; ++a) sf[a] = RegB<bf16>::pack(sc[a] + 2 * s2);
#pragma unroll
      for (int jn = 0; jn < NJ; ++jn) {
        const typename F::V kt = F::km<L>(sK, 32 * s2, 16 * jn, lane);
#pragma unroll
        for (int a = 0; a < NH; ++a) F::mma(acc[a][jn], kt, sf[a]);
      }
    }
  }
#pragma unroll
  for (int a = 0; a < NH; ++a) {
    if (R::WR * w + 16 * a + i < nq) {
      const int64_t row = qrow0 + wq0 + 16 * a + i;
#pragma unroll
      for (int jn = 0; jn < NJ; ++jn)
        Vec4<bf16>::store(dq + (row * H + h) * D + 16 * jn + 4 * g, acc[a][jn] * scale);
    }
  }
}

// dk, dv: workgroup = 64 NH keys of one view row and head, wave w owns
// 16 NH of them (halves b); per 64-query step over the queries that see
// them, P and dS from the Q and dO tiles, dV += P^T dO and dK += scale dS^T Q,
// each fragment feeding all halves.
template <int D, int NH>
__global__ __launch_bounds__(AT_THR, NH == 2 ? 1 : 2) void k_attn_dkdv(
    const int32_t* __restrict__ views, const int32_t* __restrict__ kvtiles, int H, float scale,
    const bf16* __restrict__ q, const bf16* __restrict__ kv_k, const bf16* __restrict__ kv_v,
    const bf16* __restrict__ dO, const float* __restrict__ lse, const float* __restrict__ delta,
    float* __restrict__ dk_view, float* __restrict__ dv_view) {
  using F = Frag<bf16>;
  using L = AT_Tile<D>;
  using R = AtRows<NH>;
  constexpr int NS = D / 32, NJ = D / 16;
  __shared__ bf16 sQ[L::SIZE], sD[L::SIZE];
  __shared__ __align__(16) float sL[AT_T], sDl[AT_T];
  int tile, sub, h;
  at_block<NH>(H, tile, sub, h);
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int v = kvtiles[2 * tile], k0 = kvtiles[2 * tile + 1] + R::WG * sub;
  const int32_t* vw = views + 4 * v;
  const int64_t qrow0 = vw[V_QROW];
  const int l = vw[V_L], hh = vw[V_H];
  const int64_t kvoff = vw[V_KVOFF];
  const int nk = min(R::WG, hh + l - k0);
  if (nk <= 0) return;
  const int i = lane & 15, g = lane >> 4;
  const int wk0 = k0 + R::WR * w;           // the wave's first key (within the view row)
  typename F::V kf[NH][NS], vf[NH][NS];
  // queries that see key k0 or later: qi >= k0 - hh
  const int q_first = max(0, k0 - hh);
  const int tq0 = (q_first / AT_T) * AT_T;
  stage_rows<D, NH>(sQ, sD, kv_k, kvoff + k0, nk, H, h, t);
  __syncthreads();
  wave_frags<D, NH>(kf, sQ, sD, w, lane);
  __syncthreads();
  stage_rows<D, NH>(sQ, sD, kv_v, kvoff + k0, nk, H, h, t);
  __syncthreads();
  wave_frags<D, NH>(vf, sQ, sD, w, lane);
  RowsReg<D> pq, pd;
  float pl = 0.f, pdl = 0.f;
  pq.load(q, qrow0 + tq0, min(AT_T, l - tq0), H, h, t);
  pd.load(dO, qrow0 + tq0, min(AT_T, l - tq0), H, h, t);
  if (t < AT_T && tq0 + t < l) {
    pl = lse[(qrow0 + tq0 + t) * H + h] * AT_LOG2E;
    pdl = delta[(qrow0 + tq0 + t) * H + h];
  }
  const bool wave_live = R::WR * w < nk;
  f32x4 dk[NH][NJ], dv[NH][NJ];
#pragma unroll
  for (int b = 0; b < NH; ++b)
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      dk[b][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      dv[b][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
  const float c2 = scale * AT_LOG2E;
  for (int t0 = tq0; t0 < l; t0 += AT_T) {
    const int nq = min(AT_T, l - t0);
    __syncthreads();
    pq.store(sQ, t);
    pd.store(sD, t);
    if (t < AT_T) {
      sL[t] = pl;
      sDl[t] = pdl;
    }
    __syncthreads();
    if (t0 + AT_T < l) {
      const int n2 = min(AT_T, l - t0 - AT_T);
      pq.load(q, qrow0 + t0 + AT_T, n2, H, h, t);
      pd.load(dO, qrow0 + t0 + AT_T, n2, H, h, t);
      if (t < n2) {
        pl = lse[(qrow0 + t0 + AT_T + t) * H + h] * AT_LOG2E;
        pdl = delta[(qrow0 + t0 + AT_T + t) * H + h];
      } else {
        pl = 0.f;
        pdl = 0.f;
      }
    }
    // no query of the step sees the wave's first key: skip (wave-uniform)
    if (!wave_live || wk0 > hh + t0 + nq - 1) continue;
    // the step's scores go by 32-query halves s2 (16-query groups j = 2 s2,
    // 2 s2 + 1), each half's P and dS consumed by its dV, dK products before
    // the next half is formed
    const bool full = wk0 + R::WR - 1 <= hh + t0 && nq == AT_T && R::WR * (w + 1) <= nk;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      // lane (g, i) of half b gets S[q = t0 + 16 j + 4 g + r][key = wk0 + 16 b + i]
      f32x4 sc[NH][2], dp[NH][2];
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int b = 0; b < NH; ++b) {
          sc[b][jj] = f32x4{0.f, 0.f, 0.f, 0.f};
          dp[b][jj] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const int j = 2 * s2 + jj;
          const typename F::V qa = F::kc<L>(sQ, 16 * j, 32 * s, lane);
#pragma unroll
          for (int b = 0; b < NH; ++b) F::mma(sc[b][jj], qa, kf[b][s]);
          const typename F::V da = F::kc<L>(sD, 16 * j, 32 * s, lane);
#pragma unroll
          for (int b = 0; b < NH; ++b) F::mma(dp[b][jj], da, vf[b][s]);
        }
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        const int j = 2 * s2 + jj;
        const f32x4 lq = *reinterpret_cast<const f32x4*>(sL + 16 * j + 4 * g);
        const f32x4 dq4 = *reinterpret_cast<const f32x4*>(sDl + 16 * j + 4 * g);
#pragma unroll
        for (int b = 0; b < NH; ++b)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float p = at_exp2(fmaf(sc[b][jj][r], c2, -lq[r]));
            sc[b][jj][r] = p;                             // P
            dp[b][jj][r] = p * (dp[b][jj][r] - dq4[r]);   // dS
          }
      }
      // steps where some query does not see some key of the wave (the
      // diagonal, rows past the view, keys past the view row): zero those
      if (!full) {
#pragma unroll
        for (int b = 0; b < NH; ++b) {
          const int key = wk0 + 16 * b + i;
          const int kl = key < hh + l ? key - hh - t0 : INT32_MAX;   // visible iff kl <= query row
#pragma unroll
          for (int jj = 0; jj < 2; ++jj)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int qr = 16 * (2 * s2 + jj) + 4 * g + r;   // query row within the step
              if (qr >= nq || kl > qr) {
                sc[b][jj][r] = 0.f;
                dp[b][jj][r] = 0.f;
              }
            }
        }
      }
      // dV^T += dO^T P, dK^T += Q^T dS: lane (g, i) of half b gets [key][d = 16 jn + 4 g + r]
      bf16x8 pf[NH], sf[NH];
#pragma unroll
      for (int b = 0; b < NH; ++b) {
        pf[b] = RegB<bf16>::pack(sc[b]);
        sf[b] = RegB<bf16>::pack(dp[b]);
      }
#pragma unroll
      for (int jn = 0; jn < NJ; ++jn) {
        const typename F::V dt = F::km<L>(sD, 32 * s2, 16 * jn, lane);
#pragma unroll
        for (int b = 0; b < NH; ++b) F::mma(dv[b][jn], dt, pf[b]);
        const typename F::V qt = F::km<L>(sQ, 32 * s2, 16 * jn, lane);
#pragma unroll
        for (int b = 0; b < NH; ++b) F::mma(dk[b][jn], qt, sf[b]);
      }
    }
  }
#pragma unroll
  for (int b = 0; b < NH; ++b) {
    if (R::WR * w + 16 * b + i < nk) {
      const int64_t e = (kvoff + wk0 + 16 * b + i) * H + h;
#pragma unroll
      for (int jn = 0; jn < NJ; ++jn) {
        *reinterpret_cast<f32x4*>(dk_view + e * D + 16 * jn + 4 * g) = dk[b][jn] * scale;
        *reinterpret_cast<f32x4*>(dv_view + e * D + 16 * jn + 4 * g) = dv[b][jn];
      }
    }
  }
}

// view rows <- compact rows (bf16, 16-byte pieces): a thread moves the same
// piece of AT_GR consecutive view rows, their loads in flight together
constexpr int AT_GR = 4;
__global__ __launch_bounds__(AT_THR) void k_attn_gather(const bf16* __restrict__ src,
                                                        const int32_t* __restrict__ rows, int64_t n_kv,
                                                        int64_t C, int row_elems, bf16* __restrict__ dst) {
  const int vpr = row_elems / 8;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * AT_THR + threadIdx.x;
  const int64_t e0 = (idx / vpr) * AT_GR;
  if (e0 >= n_kv) return;
  const int c = static_cast<int>(idx % vpr) * 8;
  int32_t r[AT_GR];
#pragma unroll
  for (int q = 0; q < AT_GR; ++q) r[q] = e0 + q < n_kv ? rows[e0 + q] : -1;
  uint4 v[AT_GR];
#pragma unroll
  for (int q = 0; q < AT_GR; ++q) {
    v[q] = uint4{0u, 0u, 0u, 0u};
    if (r[q] >= 0 && r[q] < C) v[q] = *reinterpret_cast<const uint4*>(src + static_cast<int64_t>(r[q]) * row_elems + c);
  }
#pragma unroll
  for (int q = 0; q < AT_GR; ++q)
    if (e0 + q < n_kv) *reinterpret_cast<uint4*>(dst + (e0 + q) * row_elems + c) = v[q];
}

// compact rows <- sum of their view rows, in the row's (fixed) entry order;
// the entries are taken AT_GR at a time, their indices and then their rows
// requested together (an entry past the row's last, or invalid, adds zero)
__global__ __launch_bounds__(AT_THR) void k_attn_scatter(const float* __restrict__ src,
                                                         const int64_t* __restrict__ row_off,
                                                         const int32_t* __restrict__ ent, int64_t C,
                                                         int64_t n_kv, int row_elems, bf16* __restrict__ dst) {
  const int vpr = row_elems / 4;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * AT_THR + threadIdx.x;
  const int64_t r = idx / vpr;
  if (r >= C) return;
  const int c = static_cast<int>(idx % vpr) * 4;
  const int64_t b = row_off[r] < 0 ? 0 : row_off[r];
  const int64_t e_end = row_off[r + 1] > n_kv ? n_kv : row_off[r + 1];
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int64_t j = b; j < e_end; j += AT_GR) {
    int32_t e[AT_GR];
#pragma unroll
    for (int q = 0; q < AT_GR; ++q) {
      e[q] = j + q < e_end ? ent[j + q] : -1;
      if (e[q] >= n_kv) e[q] = -1;
    }
    f32x4 v[AT_GR];
#pragma unroll
    for (int q = 0; q < AT_GR; ++q) {
      v[q] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (e[q] >= 0) v[q] = *reinterpret_cast<const f32x4*>(src + static_cast<int64_t>(e[q]) * row_elems + c);
    }
#pragma unroll
    for (int q = 0; q < AT_GR; ++q)
      if (e[q] >= 0) acc += v[q];
  }
  Vec4<bf16>::store(dst + r * row_elems + c, acc);
}

int at_status(const char* where) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error(std::string(where) + ": " + hipGetErrorString(e));
    return HARTS_EHIP;
  }
  return HARTS_OK;
}

bool at16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_attn(int32_t H, int32_t d, const char* where) {
  if (H < 1 || H > 65535 || (d != 64 && d != 128)) {
    set_error(std::string(where) + ": need 1 <= H <= 65535 and d in {64, 128}");
    return HARTS_EUNSUPPORTED;
  }
  return HARTS_OK;
}

}  // namespace
}  // namespace harts

using namespace harts;

extern "C" int harts_attn_fwd(const int32_t* views, const int32_t* qtiles, int64_t n_qtiles, int32_t H,
                              int32_t d, float scale, const void* q, const void* kv_k, const void* kv_v,
                              void* o, float* lse, void* stream) {
  if (int rc = check_attn(H, d, "harts_attn_fwd")) return rc;
  if (n_qtiles < 0 || n_qtiles * 2 * H > INT32_MAX) { set_error("harts_attn_fwd: bad tile count"); return HARTS_EINVAL; }
  if (n_qtiles == 0) return HARTS_OK;
  if (!views || !qtiles || !q || !kv_k || !kv_v || !o || !lse || !at16(q) || !at16(kv_k) || !at16(kv_v) ||
      !at16(o)) {
    set_error("harts_attn_fwd: NULL or misaligned pointer");
    return HARTS_EINVAL;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid(static_cast<uint32_t>(n_qtiles * AtRows<AT_FWD_NH>::SUB * H));
  if (d == 128)
    hipLaunchKernelGGL((k_attn_fwd<128, AT_FWD_NH>), grid, dim3(AT_THR), 0, s, views, qtiles, H, scale,
                       static_cast<const bf16*>(q), static_cast<const bf16*>(kv_k), static_cast<const bf16*>(kv_v),
                       static_cast<bf16*>(o), lse);
  else
    hipLaunchKernelGGL((k_attn_fwd<64, AT_FWD_NH>), grid, dim3(AT_THR), 0, s, views, qtiles, H, scale,
                       static_cast<const bf16*>(q), static_cast<const bf16*>(kv_k), static_cast<const bf16*>(kv_v),
                       static_cast<bf16*>(o), lse);
  return at_status("k_attn_fwd");
}

extern "C" int harts_attn_bwd(const int32_t* views, const int32_t* qtiles, int64_t n_qtiles,
                              const int32_t* kvtiles, int64_t n_kvtiles, int64_t C, int32_t H, int32_t d,
                              float scale, const void* q, const void* kv_k, const void* kv_v, const void* o,
                              const float* lse, const void* dO, float* delta, void* dq, float* dk_view,
                              float* dv_view, void* stream) {
  if (int rc = check_attn(H, d, "harts_attn_bwd")) return rc;
  if (n_qtiles < 0 || n_kvtiles < 0 || C < 0 || n_qtiles * 2 * H > INT32_MAX || n_kvtiles * 2 * H > INT32_MAX) {
    set_error("harts_attn_bwd: bad sizes");
    return HARTS_EINVAL;
  }
  if (C == 0) return HARTS_OK;
  if (!views || !qtiles || !kvtiles || !q || !kv_k || !kv_v || !o || !lse || !dO || !delta || !dq || !dk_view ||
      !dv_view || !at16(q) || !at16(kv_k) || !at16(kv_v) || !at16(o) || !at16(dO) || !at16(dq) ||
      !at16(dk_view) || !at16(dv_view)) {
    set_error("harts_attn_bwd: NULL or misaligned pointer");
    return HARTS_EINVAL;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t n = C * H;
  const auto* bq = static_cast<const bf16*>(q);
  const auto* bk = static_cast<const bf16*>(kv_k);
  const auto* bv = static_cast<const bf16*>(kv_v);
  const auto* bo = static_cast<const bf16*>(o);
  const auto* bd = static_cast<const bf16*>(dO);
  auto* bdq = static_cast<bf16*>(dq);
  const dim3 gd(static_cast<uint32_t>((n + AT_THR - 1) / AT_THR));
  if (d == 128) hipLaunchKernelGGL((k_attn_delta<128>), gd, dim3(AT_THR), 0, s, n, bo, bd, delta);
  else hipLaunchKernelGGL((k_attn_delta<64>), gd, dim3(AT_THR), 0, s, n, bo, bd, delta);
  if (int rc = at_status("k_attn_delta")) return rc;
  if (n_qtiles > 0) {
    const dim3 g(static_cast<uint32_t>(n_qtiles * AtRows<AT_DQ_NH>::SUB * H));
    if (d == 128)
      hipLaunchKernelGGL((k_attn_dq<128, AT_DQ_NH>), g, dim3(AT_THR), 0, s, views, qtiles, H, scale, bq, bk, bv, bd, lse,
                         delta, bdq);
    else
      hipLaunchKernelGGL((k_attn_dq<64, AT_DQ_NH>), g, dim3(AT_THR), 0, s, views, qtiles, H, scale, bq, bk, bv, bd, lse,
                         delta, bdq);
    if (int rc = at_status("k_attn_dq")) return rc;
  }
  if (n_kvtiles > 0) {
    const dim3 g(static_cast<uint32_t>(n_kvtiles * AtRows<AT_DKDV_NH>::SUB * H));
    if (d == 128)
      hipLaunchKernelGGL((k_attn_dkdv<128, AT_DKDV_NH>), g, dim3(AT_THR), 0, s, views, kvtiles, H, scale, bq, bk, bv, bd, lse,
                         delta, dk_view, dv_view);
    else
      hipLaunchKernelGGL((k_attn_dkdv<64, AT_DKDV_NH>), g, dim3(AT_THR), 0, s, views, kvtiles, H, scale, bq, bk, bv, bd, lse,
                         delta, dk_view, dv_view);
    if (int rc = at_status("k_attn_dkdv")) return rc;
  }
  return HARTS_OK;
}

extern "C" int harts_attn_gather(const void* src, const int32_t* kv_rows, int64_t n_kv, int64_t C, int32_t H,
                                 int32_t d, void* dst, void* stream) {
  if (int rc = check_attn(H, d, "harts_attn_gather")) return rc;
  if (n_kv < 0 || C < 0) { set_error("harts_attn_gather: bad sizes"); return HARTS_EINVAL; }
  if (n_kv == 0) return HARTS_OK;
  if (!src || !kv_rows || !dst || !at16(src) || !at16(dst)) {
    set_error("harts_attn_gather: NULL or misaligned pointer");
    return HARTS_EINVAL;
  }
  const int row_elems = H * d;
  const int64_t threads = (n_kv + AT_GR - 1) / AT_GR * (row_elems / 8);
  hipLaunchKernelGGL(k_attn_gather, dim3(static_cast<uint32_t>((threads + AT_THR - 1) / AT_THR)), dim3(AT_THR),
                     0, static_cast<hipStream_t>(stream), static_cast<const bf16*>(src), kv_rows, n_kv, C,
                     row_elems, static_cast<bf16*>(dst));
  return at_status("k_attn_gather");
}

extern "C" int harts_attn_scatter(const float* src, const int64_t* row_off, const int32_t* ent, int64_t C,
                                  int64_t n_kv, int32_t H, int32_t d, void* dst, void* stream) {
  if (int rc = check_attn(H, d, "harts_attn_scatter")) return rc;
  if (n_kv < 0 || C < 0) { set_error("harts_attn_scatter: bad sizes"); return HARTS_EINVAL; }
  if (C == 0) return HARTS_OK;
  if (!src || !row_off || (!ent && n_kv > 0) || !dst || !at16(src) || !at16(dst)) {
    set_error("harts_attn_scatter: NULL or misaligned pointer");
    return HARTS_EINVAL;
  }
  const int row_elems = H * d;
  const int64_t threads = C * (row_elems / 4);
  hipLaunchKernelGGL(k_attn_scatter, dim3(static_cast<uint32_t>((threads + AT_THR - 1) / AT_THR)), dim3(AT_THR),
                     0, static_cast<hipStream_t>(stream), src, row_off, ent, C, n_kv, row_elems,
                     static_cast<bf16*>(dst));
  return at_status("k_attn_scatter");
}
