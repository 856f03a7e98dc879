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
// Flash-style kernels, one 64-row tile per workgroup of 4 waves (a wave owns
// 16 rows), bf16 MFMA 16x16x32 with float32 accumulation, tiles staged in
// LDS.  Every product is issued with the operand roles chosen so that the
// row the wave owns is the accumulator column (lane % 16): per-row softmax
// statistics, rescales and outputs then stay in one lane, and a score tile
// in accumulators is already the B operand of the next product (two 16-key
// tiles form one 32-deep operand).
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
constexpr int AT_T = 64;             // rows per tile
constexpr float AT_LOG2E = 1.4426950408889634f;
constexpr float AT_NEG = -1.0e30f;   // masked score (finite: no inf - inf)

// view table: 4 int32 per view
enum { V_QROW = 0, V_L = 1, V_KVOFF = 2, V_H = 3 };

template <int D>
using AT_Tile = Tile<bf16, D>;
using AT_PT = Tile<bf16, AT_T>;

// Copy rows [row0, row0 + n) (n <= 64, zero beyond) of a [rows, H, D] bf16
// tensor, head h, into an LDS tile.
template <int D>
__device__ inline void load_rows(bf16* tile, const bf16* __restrict__ src, int64_t row0, int n, int H, int h,
                                 int t) {
  constexpr int VPR = D / 8;  // 16-byte vectors per row
  for (int idx = t; idx < AT_T * VPR; idx += AT_THR) {
    const int r = idx / VPR, c = (idx % VPR) * 8;
    uint4 v = {0u, 0u, 0u, 0u};
    if (r < n) v = *reinterpret_cast<const uint4*>(src + ((row0 + r) * H + h) * D + c);
    *reinterpret_cast<uint4*>(tile + AT_Tile<D>::at(r, c)) = v;
  }
}

__device__ inline float row_max4(float x) {  // over the 4 lane groups (same lane % 16)
  x = fmaxf(x, __shfl_xor(x, 16));
  return fmaxf(x, __shfl_xor(x, 32));
}
__device__ inline float row_sum4(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}

// ---------------------------------------------------------------------------
// forward
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(AT_THR) void k_attn_fwd(const int32_t* __restrict__ views,
                                                     const int32_t* __restrict__ qtiles, int H, float scale,
                                                     const bf16* __restrict__ q, const bf16* __restrict__ kv_k,
                                                     const bf16* __restrict__ kv_v, bf16* __restrict__ o,
                                                     float* __restrict__ lse) {
  using F = Frag<bf16>;
  using L = AT_Tile<D>;
  constexpr int NS = D / 32;  // 32-deep steps over d
  constexpr int NJ = D / 16;  // 16-column output tiles
  __shared__ bf16 sQ[L::SIZE], sK[L::SIZE], sV[L::SIZE];
  const int tile = blockIdx.x / H, h = blockIdx.x % H;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int v = qtiles[2 * tile], t0 = qtiles[2 * tile + 1];
  const int32_t* vw = views + 4 * v;
  const int64_t qrow0 = vw[V_QROW];
  const int l = vw[V_L], hh = vw[V_H];
  const int64_t kvoff = vw[V_KVOFF];
  const int nq = min(AT_T, l - t0);
  load_rows<D>(sQ, q, qrow0 + t0, nq, H, h, t);
  __syncthreads();
  typename F::V qf[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) qf[s] = F::kc<L>(sQ, 16 * w, 32 * s, lane);
  const int i = lane & 15, g = lane >> 4;
  const int qi = t0 + 16 * w + i;           // this lane's query, within the view
  const float c2 = scale * AT_LOG2E;        // scores in base 2
  float m = AT_NEG, lsum = 0.f;
  f32x4 acc[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int kv_end = hh + t0 + nq;          // keys the tile's last query sees
  for (int k0 = 0; k0 < kv_end; k0 += AT_T) {
    const int nk = min(AT_T, kv_end - k0);
    __syncthreads();                        // previous tile's readers are done
    load_rows<D>(sK, kv_k, kvoff + k0, nk, H, h, t);
    load_rows<D>(sV, kv_v, kvoff + k0, nk, H, h, t);
    __syncthreads();
    // S^T tiles: lane (g, i) gets S[q = 16w + i][key = k0 + 16 j + 4 g + r]
    f32x4 sc[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      sc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) F::mma(sc[j], F::kc<L>(sK, 16 * j, 32 * s, lane), qf[s]);
    }
    float tmax = AT_NEG;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + 16 * j + 4 * g + r;
        const float x = key <= hh + qi && key < kv_end ? sc[j][r] * c2 : AT_NEG;
        sc[j][r] = x;
        tmax = fmaxf(tmax, x);
      }
    const float mn = fmaxf(m, row_max4(tmax));
    const float corr = exp2f(m - mn);
    float ps = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float p = sc[j][r] <= AT_NEG ? 0.f : exp2f(sc[j][r] - mn);
        sc[j][r] = p;
        ps += p;
      }
    lsum = lsum * corr + row_sum4(ps);
    m = mn;
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[j] *= corr;
    // O^T += V^T P^T: lane (g, i) gets O[q = 16w + i][d = 16 jn + 4 g + r]
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const bf16x8 pf = RegB<bf16>::pack(sc + 2 * s2);
#pragma unroll
      for (int jn = 0; jn < NJ; ++jn) F::mma(acc[jn], F::km<L>(sV, 32 * s2, 16 * jn, lane), pf);
    }
  }
  if (16 * w + i < nq) {
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    const int64_t row = qrow0 + qi;
#pragma unroll
    for (int jn = 0; jn < NJ; ++jn)
      Vec4<bf16>::store(o + (row * H + h) * D + 16 * jn + 4 * g, acc[jn] * inv);
    if (g == 0) lse[row * H + h] = (m + log2f(lsum)) / AT_LOG2E;   // natural log of sum exp(scale s)
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

template <int D>
__global__ __launch_bounds__(AT_THR) void k_attn_dq(const int32_t* __restrict__ views,
                                                    const int32_t* __restrict__ qtiles, int H, float scale,
                                                    const bf16* __restrict__ q, const bf16* __restrict__ kv_k,
                                                    const bf16* __restrict__ kv_v, const bf16* __restrict__ dO,
                                                    const float* __restrict__ lse,
                                                    const float* __restrict__ delta, bf16* __restrict__ dq) {
  using F = Frag<bf16>;
  using L = AT_Tile<D>;
  constexpr int NS = D / 32, NJ = D / 16;
  __shared__ bf16 sQ[L::SIZE], sK[L::SIZE], sV[L::SIZE];
  const int tile = blockIdx.x / H, h = blockIdx.x % H;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int v = qtiles[2 * tile], t0 = qtiles[2 * tile + 1];
  const int32_t* vw = views + 4 * v;
  const int64_t qrow0 = vw[V_QROW];
  const int l = vw[V_L], hh = vw[V_H];
  const int64_t kvoff = vw[V_KVOFF];
  const int nq = min(AT_T, l - t0);
  const int i = lane & 15, g = lane >> 4;
  const int qi = t0 + 16 * w + i;
  const bool live = 16 * w + i < nq;
  const int64_t qrow = qrow0 + (live ? qi : t0);
  const float l2 = live ? lse[qrow * H + h] * AT_LOG2E : 0.f;
  const float dl = live ? delta[qrow * H + h] : 0.f;
  const float c2 = scale * AT_LOG2E;
  load_rows<D>(sQ, q, qrow0 + t0, nq, H, h, t);
  load_rows<D>(sK, dO, qrow0 + t0, nq, H, h, t);   // dO tile staged through sK
  __syncthreads();
  typename F::V qf[NS], df[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    qf[s] = F::kc<L>(sQ, 16 * w, 32 * s, lane);
    df[s] = F::kc<L>(sK, 16 * w, 32 * s, lane);
  }
  f32x4 acc[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int kv_end = hh + t0 + nq;
  for (int k0 = 0; k0 < kv_end; k0 += AT_T) {
    const int nk = min(AT_T, kv_end - k0);
    __syncthreads();
    load_rows<D>(sK, kv_k, kvoff + k0, nk, H, h, t);
    load_rows<D>(sV, kv_v, kvoff + k0, nk, H, h, t);
    __syncthreads();
    f32x4 sc[4], dp[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      sc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
      dp[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        F::mma(sc[j], F::kc<L>(sK, 16 * j, 32 * s, lane), qf[s]);
        F::mma(dp[j], F::kc<L>(sV, 16 * j, 32 * s, lane), df[s]);
      }
    }
    // dS = P (dP - delta), P = exp(scale s - lse)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = k0 + 16 * j + 4 * g + r;
        const float p = live && key <= hh + qi ? exp2f(sc[j][r] * c2 - l2) : 0.f;
        sc[j][r] = p * (dp[j][r] - dl);
      }
    // dQ^T += K^T dS^T: lane (g, i) gets dQ[q = 16w + i][d = 16 jn + 4 g + r]
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const bf16x8 sf = RegB<bf16>::pack(sc + 2 * s2);
#pragma unroll
      for (int jn = 0; jn < NJ; ++jn) F::mma(acc[jn], F::km<L>(sK, 32 * s2, 16 * jn, lane), sf);
    }
  }
  if (live) {
#pragma unroll
    for (int jn = 0; jn < NJ; ++jn) Vec4<bf16>::store(dq + (qrow * H + h) * D + 16 * jn + 4 * g, acc[jn] * scale);
  }
}

template <int D>
__global__ __launch_bounds__(AT_THR) void k_attn_dkdv(const int32_t* __restrict__ views,
                                                      const int32_t* __restrict__ kvtiles, int H, float scale,
                                                      const bf16* __restrict__ q, const bf16* __restrict__ kv_k,
                                                      const bf16* __restrict__ kv_v, const bf16* __restrict__ dO,
                                                      const float* __restrict__ lse,
                                                      const float* __restrict__ delta, float* __restrict__ dk_view,
                                                      float* __restrict__ dv_view) {
  using F = Frag<bf16>;
  using L = AT_Tile<D>;
  constexpr int NS = D / 32, NJ = D / 16;
  __shared__ bf16 sQ[L::SIZE], sD[L::SIZE];
  __shared__ float sL[AT_T], sDl[AT_T];
  const int tile = blockIdx.x / H, h = blockIdx.x % H;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int v = kvtiles[2 * tile], k0 = kvtiles[2 * tile + 1];
  const int32_t* vw = views + 4 * v;
  const int64_t qrow0 = vw[V_QROW];
  const int l = vw[V_L], hh = vw[V_H];
  const int64_t kvoff = vw[V_KVOFF];
  const int nk = min(AT_T, hh + l - k0);
  const int i = lane & 15, g = lane >> 4;
  const int key = k0 + 16 * w + i;          // this lane's key, within the view row
  // K and V rows of the wave's 16 keys, as B operands (staged through sQ, sD)
  load_rows<D>(sQ, kv_k, kvoff + k0, nk, H, h, t);
  load_rows<D>(sD, kv_v, kvoff + k0, nk, H, h, t);
  __syncthreads();
  typename F::V kf[NS], vf[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    kf[s] = F::kc<L>(sQ, 16 * w, 32 * s, lane);
    vf[s] = F::kc<L>(sD, 16 * w, 32 * s, lane);
  }
  f32x4 dk[NJ], dv[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    dk[j] = f32x4{0.f, 0.f, 0.f, 0.f};
    dv[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const float c2 = scale * AT_LOG2E;
  // queries that see key k0 or later: qi >= k0 - hh
  const int q_first = max(0, k0 - hh);
  for (int t0 = (q_first / AT_T) * AT_T; t0 < l; t0 += AT_T) {
    const int nq = min(AT_T, l - t0);
    __syncthreads();
    load_rows<D>(sQ, q, qrow0 + t0, nq, H, h, t);
    load_rows<D>(sD, dO, qrow0 + t0, nq, H, h, t);
    if (t < AT_T) {
      const bool ok = t < nq;
      const int64_t row = qrow0 + t0 + t;
      sL[t] = ok ? lse[row * H + h] * AT_LOG2E : 0.f;
      sDl[t] = ok ? delta[row * H + h] : 0.f;
    }
    __syncthreads();
    // lane (g, i) gets S[q = t0 + 16 j + 4 g + r][key]
    f32x4 sc[4], dp[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      sc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
      dp[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        F::mma(sc[j], F::kc<L>(sQ, 16 * j, 32 * s, lane), kf[s]);
        F::mma(dp[j], F::kc<L>(sD, 16 * j, 32 * s, lane), vf[s]);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int qr = 16 * j + 4 * g + r;          // query row within the tile
        const bool vis = qr < nq && key < hh + l && key <= hh + t0 + qr;
        const float p = vis ? exp2f(sc[j][r] * c2 - sL[qr]) : 0.f;
        sc[j][r] = p;                                // P
        dp[j][r] = p * (dp[j][r] - sDl[qr]);         // dS
      }
    // dV^T += dO^T P, dK^T += Q^T dS: lane (g, i) gets [key][d = 16 jn + 4 g + r]
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      const bf16x8 pf = RegB<bf16>::pack(sc + 2 * s2);
      const bf16x8 sf = RegB<bf16>::pack(dp + 2 * s2);
#pragma unroll
      for (int jn = 0; jn < NJ; ++jn) {
        F::mma(dv[jn], F::km<L>(sD, 32 * s2, 16 * jn, lane), pf);
        F::mma(dk[jn], F::km<L>(sQ, 32 * s2, 16 * jn, lane), sf);
      }
    }
  }
  if (16 * w + i < nk) {
    const int64_t e = (kvoff + key) * H + h;
#pragma unroll
    for (int jn = 0; jn < NJ; ++jn) {
      *reinterpret_cast<f32x4*>(dk_view + e * D + 16 * jn + 4 * g) = dk[jn] * scale;
      *reinterpret_cast<f32x4*>(dv_view + e * D + 16 * jn + 4 * g) = dv[jn];
    }
  }
}

// view rows <- compact rows (bf16, 16-byte pieces)
__global__ __launch_bounds__(AT_THR) void k_attn_gather(const bf16* __restrict__ src,
                                                        const int32_t* __restrict__ rows, int64_t n_kv,
                                                        int64_t C, int row_elems, bf16* __restrict__ dst) {
  const int vpr = row_elems / 8;
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * AT_THR + threadIdx.x;
  const int64_t e = idx / vpr;
  if (e >= n_kv) return;
  const int c = static_cast<int>(idx % vpr) * 8;
  const int32_t r = rows[e];
  uint4 v = {0u, 0u, 0u, 0u};
  if (r >= 0 && r < C) v = *reinterpret_cast<const uint4*>(src + static_cast<int64_t>(r) * row_elems + c);
  *reinterpret_cast<uint4*>(dst + e * row_elems + c) = v;
}

// compact rows <- sum of their view rows, in the row's (fixed) entry order
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
  for (int64_t j = b; j < e_end; ++j) {
    const int32_t e = ent[j];
    if (e < 0 || e >= n_kv) continue;
    acc += *reinterpret_cast<const f32x4*>(src + static_cast<int64_t>(e) * row_elems + c);
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
  if (n_qtiles < 0 || n_qtiles * H > INT32_MAX) { set_error("harts_attn_fwd: bad tile count"); return HARTS_EINVAL; }
  if (n_qtiles == 0) return HARTS_OK;
  if (!views || !qtiles || !q || !kv_k || !kv_v || !o || !lse || !at16(q) || !at16(kv_k) || !at16(kv_v) ||
      !at16(o)) {
    set_error("harts_attn_fwd: NULL or misaligned pointer");
    return HARTS_EINVAL;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  const dim3 grid(static_cast<uint32_t>(n_qtiles * H));
  if (d == 128)
    hipLaunchKernelGGL((k_attn_fwd<128>), grid, dim3(AT_THR), 0, s, views, qtiles, H, scale,
                       static_cast<const bf16*>(q), static_cast<const bf16*>(kv_k), static_cast<const bf16*>(kv_v),
                       static_cast<bf16*>(o), lse);
  else
    hipLaunchKernelGGL((k_attn_fwd<64>), grid, dim3(AT_THR), 0, s, views, qtiles, H, scale,
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
  if (n_qtiles < 0 || n_kvtiles < 0 || C < 0 || n_qtiles * H > INT32_MAX || n_kvtiles * H > INT32_MAX) {
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
    const dim3 g(static_cast<uint32_t>(n_qtiles * H));
    if (d == 128)
      hipLaunchKernelGGL((k_attn_dq<128>), g, dim3(AT_THR), 0, s, views, qtiles, H, scale, bq, bk, bv, bd, lse,
                         delta, bdq);
    else
      hipLaunchKernelGGL((k_attn_dq<64>), g, dim3(AT_THR), 0, s, views, qtiles, H, scale, bq, bk, bv, bd, lse,
                         delta, bdq);
    if (int rc = at_status("k_attn_dq")) return rc;
  }
  if (n_kvtiles > 0) {
    const dim3 g(static_cast<uint32_t>(n_kvtiles * H));
    if (d == 128)
      hipLaunchKernelGGL((k_attn_dkdv<128>), g, dim3(AT_THR), 0, s, views, kvtiles, H, scale, bq, bk, bv, bd, lse,
                         delta, dk_view, dv_view);
    else
      hipLaunchKernelGGL((k_attn_dkdv<64>), g, dim3(AT_THR), 0, s, views, kvtiles, H, scale, bq, bk, bv, bd, lse,
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
  const int64_t threads = n_kv * (row_elems / 8);
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
